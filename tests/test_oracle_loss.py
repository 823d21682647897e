"""Pins for the oracle's LM-head + PPO loss and its gradients.

Independent anchors: float64 torch autograd of the plain formula, scipy's
logsumexp, central finite differences, softmax invariants, closed forms of the
special cases (A = 0, rho = 1, W = 0), and brute-force enumeration of every
cutoff (App. B: the cutoff-weighted mean of the truncated update equals the
full update).
"""
import numpy as np
import pytest
import torch
from scipy import special

from oracle import cutoffs, ppo_head


def _small_case(seed=0, N=37, d=24, V=53, R=5, sigma=0.08):
    rng = np.random.default_rng(seed)
    h = rng.standard_normal((N, d))
    W = 0.3 * rng.standard_normal((V, d))
    target = rng.integers(0, V, N)
    seq_id = np.sort(rng.integers(0, R, N))
    adv = rng.standard_normal(R)
    weight = rng.uniform(1.0, 3.0, N).astype(np.float32)
    lp_new = ppo_head.target_logprob(h, W, target)
    lp_old = lp_new + sigma * rng.standard_normal(N)
    return h, W, target, lp_old, weight, seq_id, adv


def _torch_reference(h, W, target, lp_old, weight, seq_id, adv, el, eh, scale):
    th = torch.tensor(h, dtype=torch.float64, requires_grad=True)
    tW = torch.tensor(W, dtype=torch.float64, requires_grad=True)
    z = th @ tW.T
    logp = torch.log_softmax(z, dim=1)[torch.arange(len(target)), torch.tensor(target)]
    rho = torch.exp(logp - torch.tensor(lp_old, dtype=torch.float64))
    A = torch.tensor(adv, dtype=torch.float64)[torch.tensor(seq_id)]
    s = torch.minimum(rho * A, torch.clamp(rho, 1 - el, 1 + eh) * A)
    loss = -scale * (torch.tensor(weight, dtype=torch.float64) * s).sum()
    loss.backward()
    return loss.item(), th.grad.numpy(), tW.grad.numpy(), logp.detach().numpy()


@pytest.mark.parametrize("seed,el,eh", [(0, 0.1, 0.1), (1, 0.2, 0.28), (2, 0.05, 0.1)])
def test_matches_float64_autograd(seed, el, eh):
    args = _small_case(seed, sigma=0.25)
    out = ppo_head.loss_fwd_bwd(*args, eps_low=el, eps_high=eh, loss_scale=0.125, chunk=8)
    L, dh, dw, logp = _torch_reference(*args, el, eh, 0.125)
    assert out["loss"] == pytest.approx(L, rel=1e-12, abs=1e-14)
    np.testing.assert_allclose(out["d_hidden"], dh, rtol=1e-10, atol=1e-13)
    np.testing.assert_allclose(out["d_w"], dw, rtol=1e-10, atol=1e-13)
    np.testing.assert_allclose(out["logp_new"], logp, rtol=1e-13, atol=1e-13)
    assert 0 < out["mu"].sum() < len(out["mu"])   # both branches exercised


def test_lse_matches_scipy():
    h, W, target, *_ = _small_case(3)
    z = h @ W.T
    lp = ppo_head.target_logprob(h, W, target, chunk=5)
    np.testing.assert_allclose(lp, z[np.arange(len(target)), target] - special.logsumexp(z, axis=1), rtol=0, atol=1e-12)


def test_finite_differences():
    h, W, target, lp_old, weight, seq_id, adv = _small_case(4, N=12, d=6, V=9, R=3, sigma=0.02)
    kw = dict(eps_low=0.1, eps_high=0.1, loss_scale=0.5)
    out = ppo_head.loss_fwd_bwd(h, W, target, lp_old, weight, seq_id, adv, **kw)
    # keep away from the clip boundaries so the loss is smooth at the probe points
    assert np.min(np.abs(out["rho"] - 1.1)) > 1e-3 and np.min(np.abs(out["rho"] - 0.9)) > 1e-3
    eps = 1e-6
    rng = np.random.default_rng(9)
    for _ in range(6):
        i, k = rng.integers(0, h.shape[0]), rng.integers(0, h.shape[1])
        hp, hm = h.copy(), h.copy()
        hp[i, k] += eps
        hm[i, k] -= eps
        fd = (ppo_head.loss_fwd_bwd(hp, W, target, lp_old, weight, seq_id, adv, **kw)["loss"]
              - ppo_head.loss_fwd_bwd(hm, W, target, lp_old, weight, seq_id, adv, **kw)["loss"]) / (2 * eps)
        assert fd == pytest.approx(out["d_hidden"][i, k], rel=1e-6, abs=1e-9)
        v, k = rng.integers(0, W.shape[0]), rng.integers(0, W.shape[1])
        Wp, Wm = W.copy(), W.copy()
        Wp[v, k] += eps
        Wm[v, k] -= eps
        fd = (ppo_head.loss_fwd_bwd(h, Wp, target, lp_old, weight, seq_id, adv, **kw)["loss"]
              - ppo_head.loss_fwd_bwd(h, Wm, target, lp_old, weight, seq_id, adv, **kw)["loss"]) / (2 * eps)
        assert fd == pytest.approx(out["d_w"][v, k], rel=1e-6, abs=1e-9)


def test_invariants():
    args = _small_case(5)
    h, W = args[0], args[1]
    out = ppo_head.loss_fwd_bwd(*args, eps_low=0.1, eps_high=0.1, loss_scale=1.0)
    # softmax rows sum to one, so every token's logit gradient sums to zero over V
    np.testing.assert_allclose(out["d_w"].sum(axis=0), 0.0, atol=1e-12)
    # <dW, W> and <dH, H> are both sum_{i,v} G_iv z_iv
    assert np.sum(out["d_w"] * W) == pytest.approx(np.sum(out["d_hidden"] * h), rel=1e-11)
    # App. D: dH_i = delta_i (W_{o_i} - sum_v p_iv W_v)
    z = h @ W.T
    p = np.exp(z - special.logsumexp(z, axis=1, keepdims=True))
    expect = out["delta"][:, None] * (W[args[2]] - p @ W)
    np.testing.assert_allclose(out["d_hidden"], expect, rtol=1e-10, atol=1e-13)


def test_special_cases():
    h, W, target, lp_old, weight, seq_id, adv = _small_case(6)
    kw = dict(eps_low=0.1, eps_high=0.1, loss_scale=0.25)
    z0 = ppo_head.loss_fwd_bwd(h, W, target, lp_old, weight, seq_id, np.zeros_like(adv), **kw)
    assert z0["loss"] == 0.0 and not z0["d_hidden"].any() and not z0["d_w"].any()
    # rho == 1: the objective is the weighted policy-gradient surrogate sum c_i A_i
    lp = ppo_head.target_logprob(h, W, target)
    r1 = ppo_head.loss_fwd_bwd(h, W, target, lp, weight, seq_id, adv, **kw)
    np.testing.assert_allclose(r1["rho"], 1.0, rtol=0, atol=1e-14)
    assert r1["loss"] == pytest.approx(-0.25 * np.sum(weight.astype(np.float64) * adv[seq_id]), rel=1e-12)
    np.testing.assert_allclose(r1["delta"], -0.25 * weight * adv[seq_id], rtol=1e-12)
    # W = 0: uniform softmax, lse = log V
    w0 = ppo_head.loss_fwd_bwd(h, np.zeros_like(W), target, lp_old, weight, seq_id, adv, **kw)
    np.testing.assert_allclose(w0["lse"], np.log(W.shape[0]), rtol=1e-15)
    np.testing.assert_allclose(w0["logp_new"], -np.log(W.shape[0]), rtol=1e-15)


def test_bf16_widening_is_exact():
    bits = np.array([0x3F80, 0xBF80, 0x0000, 0x7F7F, 0x0001, 0x4049], dtype=np.uint16)
    got = ppo_head.bf16_bits_to_f64(bits)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(got, ref)


def test_brute_force_unbiasedness():
    """App. B: sum over every cutoff h of Pr(H_r = h) x (truncated, reweighted update of
    completion r cut at h) equals the completion's full update, for loss, dH and dW."""
    rng = np.random.default_rng(11)
    P, K, d, V = 2, 3, 10, 17
    lengths = rng.integers(3, 12, P * K).astype(np.int32)
    horizon = lengths.reshape(P, K).max(axis=1)
    xi_off = np.concatenate([[0], np.cumsum(horizon)]).astype(np.int64)
    xi = np.concatenate([np.minimum.accumulate(np.sort(rng.uniform(0.05, 1.0, T))[::-1]) for T in horizon])
    S = int(lengths.sum())
    h_full = rng.standard_normal((S, d))
    W = 0.4 * rng.standard_normal((V, d))
    tgt = rng.integers(0, V, S)
    lp_old = ppo_head.target_logprob(h_full, W, tgt) + 0.08 * rng.standard_normal(S)
    adv = ppo_head.advantages(rng.integers(0, 2, P * K).astype(float), K)
    kw = dict(eps_low=0.1, eps_high=0.1, loss_scale=1.0 / (P * K))

    def run(H, xi_tab):
        pk = cutoffs.pack_prefixes(H, lengths, xi_tab, xi_off, P, K, tgt, lp_old)
        src = pk["src_row"]
        hid = h_full[src]
        out = ppo_head.loss_fwd_bwd(hid, W, pk["target"], lp_old[src], pk["weight"], pk["seq_id"], adv, **kw)
        dfull = np.zeros_like(h_full)
        dfull[src] = out["d_hidden"]
        return out["loss"], dfull, out["d_w"]

    full = run(lengths.copy(), np.ones_like(xi))
    acc = [0.0, np.zeros_like(h_full), np.zeros_like(W)]
    for r in range(P * K):
        p = r // K
        pmf = cutoffs.cutoff_pmf(xi[xi_off[p]:xi_off[p + 1]], int(lengths[r]))
        for hcut, pr in enumerate(pmf):
            if pr == 0.0:
                continue
            H = np.zeros(P * K, dtype=np.int32)
            H[r] = hcut
            L, dh, dw = run(H, xi)
            acc[0] += pr * L
            acc[1] += pr * dh
            acc[2] += pr * dw
    # weights are float32(2^32/q): exact up to float32 rounding, relative 2^-24
    assert acc[0] == pytest.approx(full[0], rel=1e-6)
    # (elementwise with an absolute floor: single entries of dW are sums that cancel)
    np.testing.assert_allclose(acc[1], full[1], rtol=1e-6, atol=1e-6 * np.abs(full[1]).max())
    np.testing.assert_allclose(acc[2], full[2], rtol=1e-6, atol=1e-6 * np.abs(full[2]).max())
    # and a deliberately wrong weight (1 instead of 1/xi) is detectably biased
    L_unweighted = 0.0
    for r in range(P * K):
        p = r // K
        pmf = cutoffs.cutoff_pmf(xi[xi_off[p]:xi_off[p + 1]], int(lengths[r]))
        for hcut, pr in enumerate(pmf):
            H = np.zeros(P * K, dtype=np.int32)
            H[r] = hcut
            L_unweighted += pr * run(H, np.ones_like(xi))[0]
    assert abs(L_unweighted - full[0]) > 1e-3 * abs(full[0])


@pytest.mark.parametrize("seed,el,eh", [(5, 0.1, 0.1), (6, 0.2, 0.28)])
def test_loss_terms_and_grad_w_rows_match_autograd(seed, el, eh):
    """The large-batch helpers: the loss from given log-probs, and selected dW rows from each
    token's lse and delta, against float64 autograd of the plain formula (independent of
    loss_fwd_bwd).  Rows: targets of one token, of several tokens, of none, first and last."""
    h, W, target, lp_old, weight, seq_id, adv = _small_case(seed, N=41, V=29, sigma=0.25)
    target[:6] = 3                      # a row that is the target of several tokens
    lp_old = ppo_head.target_logprob(h, W, target) + 0.25 * np.random.default_rng(seed).standard_normal(len(target))
    L, dh, dw, logp = _torch_reference(h, W, target, lp_old, weight, seq_id, adv, el, eh, 0.125)
    t = ppo_head.loss_terms(logp, lp_old, weight, seq_id, adv, el, eh, 0.125)
    assert t["loss"] == pytest.approx(L, rel=1e-12, abs=1e-14)
    assert 0 < t["mu"].sum() < len(target)
    # delta = dL/dl: autograd through the ratio and clip alone
    tl = torch.tensor(logp, dtype=torch.float64, requires_grad=True)
    rho = torch.exp(tl - torch.tensor(lp_old, dtype=torch.float64))
    A = torch.tensor(adv, dtype=torch.float64)[torch.tensor(seq_id)]
    (-0.125 * (torch.tensor(weight, dtype=torch.float64)
               * torch.minimum(rho * A, torch.clamp(rho, 1 - el, 1 + eh) * A)).sum()).backward()
    np.testing.assert_allclose(t["delta"], tl.grad.numpy(), rtol=1e-12, atol=1e-15)
    lse = ppo_head.target_logits(h, W, target) - logp
    np.testing.assert_allclose(lse, special.logsumexp(h @ W.T, axis=1), rtol=1e-13)
    empty = next(v for v in range(W.shape[0]) if not np.any(target == v))   # no token targets it
    rows = np.array([0, 3, int(target[10]), W.shape[0] - 1, empty])
    got = ppo_head.grad_w_rows(h, W, target, lse, t["delta"], rows, chunk=7)
    np.testing.assert_allclose(got, dw[rows], rtol=1e-10, atol=1e-13)
    # and the full oracle agrees
    full = ppo_head.loss_fwd_bwd(h, W, target, lp_old, weight, seq_id, adv, el, eh, 0.125)
    np.testing.assert_allclose(got, full["d_w"][rows], rtol=1e-10, atol=1e-13)
