"""GPU parity of the cutoff design ("Computing xi": proxy weights and the budgeted monotone
solve) through the C ABI, against the float64 oracle.

Bar: the weights and the tables are float64 on both sides with the same operations except
summation order, so they agree to relative 1e-12; the designed tables are valid survival
tables (non-increasing, in (0, 1], spending the budget exactly); and a designed table drives
the sampler bit-exactly like any other table.
"""
import numpy as np
import pytest
import torch

from oracle import cutoff_design as cd
from oracle import cutoffs as ocut
from oracle import score_proxy as osp
from paper_2606_29758_amd import pspo, synth

pytestmark = pytest.mark.gpu

MINI7B = synth.custom("mini7b", "qwen7b", P=2, K=2, length_law=("uniform", 150, 420), data_seed=31)


def _cuda(a, dtype):
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda").to(dtype)


def _layout(wl):
    full_off = np.concatenate([[0], np.cumsum(wl.lengths)]).astype(np.int32)
    return full_off, np.asarray(wl.xi_off, dtype=np.int64), int(wl.xi_off[-1])


def _weights(wl, gamma, ids, logp, want_parts=True):
    cfg = wl.cfg
    full_off, xi_off, total = _layout(wl)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    out = pspo.design_weights(_cuda(gamma, torch.float32), _cuda(ids, torch.int32), _cuda(logp, torch.float32),
                              _cuda(wl.lengths, torch.int32), _cuda(full_off, torch.int32),
                              _cuda(wl.rewards, torch.float32), _cuda(xi_off, torch.int64), cfg.P, cfg.K, total,
                              want_parts=want_parts, err_flag=err)
    torch.cuda.synchronize()
    return out, int(err.item())


@pytest.mark.parametrize("name", ["tiny", "mini7b", "qwen7b"])
def test_design_weights_parity(name):
    wl = synth.make_workload(MINI7B if name == "mini7b" else name, with_matrices=False)
    rng = np.random.default_rng(4)
    gamma = rng.gamma(2.0, 500.0, wl.total_tokens).astype(np.float32)
    ids, logp = synth.make_topk(wl)
    out, err = _weights(wl, gamma, ids, logp)
    assert err == 0
    ref = cd.proxy_weights(gamma, ids, logp, wl.lengths, wl.rewards, wl.cfg.P, wl.cfg.K)
    np.testing.assert_allclose(out["gamma_bar"].cpu().numpy(), ref["gbar"], rtol=1e-12)
    np.testing.assert_allclose(out["u"].cpu().numpy(), ref["u"], rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(out["w"].cpu().numpy(), ref["w"], rtol=1e-12, atol=1e-12)
    u = out["u"].cpu().numpy()
    assert np.all(u >= 0) and np.all(u <= 0.5)
    # equal-reward prompts: the outcome is known, u = 0 exactly
    R = wl.rewards.reshape(wl.cfg.P, wl.cfg.K)
    for p in np.flatnonzero((R == R[:, :1]).all(axis=1)):
        assert not u[wl.xi_off[p]:wl.xi_off[p + 1]].any()


def _random_weights(xi_off, seed):
    """Heavy-tailed weights with increasing runs (pooling), zero runs and tails."""
    rng = np.random.default_rng(seed)
    w = rng.gamma(0.6, 1.0, xi_off[-1]) * np.exp(rng.normal(0, 2.0, xi_off[-1]))
    for p in range(len(xi_off) - 1):
        a, b = xi_off[p], xi_off[p + 1]
        n = b - a
        w[a + n // 5: a + n // 5 + n // 10] = np.linspace(0.1, 30.0, n // 10)   # increasing run
        if p % 2 == 1:
            w[b - n // 8: b] = 0.0                                                 # zero tail
    return w


@pytest.mark.parametrize("variant,budget,lam", [(cd.OPTIMIZED, 128.0, 0.0), (cd.OPTIMIZED, 700.0, 0.0),
                                                (cd.OPTIMIZED, 3.5, 0.0), (cd.HEURISTIC, 128.0, 0.0),
                                                (cd.UNIFORM, 128.0, 0.0), (cd.TIME_PRIOR, 128.0, 0.004)])
@pytest.mark.parametrize("name", ["mini7b", "qwen7b"])
def test_design_cutoffs_parity(name, variant, budget, lam):
    wl = synth.make_workload(MINI7B if name == "mini7b" else name, with_matrices=False)
    _, xi_off, total = _layout(wl)
    w = _random_weights(xi_off, 9)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    xi = pspo.design_cutoffs(_cuda(w, torch.float64), _cuda(xi_off, torch.int64), wl.cfg.P, total, budget,
                             variant, lam, err_flag=err).cpu().numpy()
    assert int(err.item()) == 0
    ref = cd.design_tables(w, xi_off, budget, variant, lam)
    np.testing.assert_allclose(xi, ref, rtol=1e-12)
    for p in range(wl.cfg.P):
        x = xi[xi_off[p]:xi_off[p + 1]]
        assert np.all(np.diff(x) <= 0) and x[0] <= 1.0 and x[-1] >= cd.XI_FLOOR
        if variant in (cd.OPTIMIZED, cd.HEURISTIC) and budget < len(x):
            if variant == cd.OPTIMIZED:
                assert x.sum() == pytest.approx(budget, rel=1e-9, abs=len(x) * cd.XI_FLOOR)
            else:
                assert x.sum() <= budget * (1 + 1e-12) + len(x) * cd.XI_FLOOR
        if budget >= len(x) and variant in (cd.OPTIMIZED, cd.HEURISTIC):
            assert np.all(x == 1.0)


def test_design_cutoffs_edge_cases():
    xi_off = np.array([0, 10, 14, 20], dtype=np.int64)
    w = np.concatenate([np.zeros(10), [4.0, 1.0, 0.0, 0.0], np.full(6, 2.0)])
    xi = pspo.design_cutoffs(_cuda(w, torch.float64), _cuda(xi_off, torch.int64), 3, 20, 3.0).cpu().numpy()
    np.testing.assert_allclose(xi, cd.design_tables(w, xi_off, 3.0), rtol=1e-15)
    np.testing.assert_allclose(xi[:10], 0.3)                        # all-zero weights: B / T
    # a negative weight is rejected on the device
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    w[12] = -1.0
    xi = pspo.design_cutoffs(_cuda(w, torch.float64), _cuda(xi_off, torch.int64), 3, 20, 3.0, err_flag=err)
    assert int(err.item()) == pspo.DEVERR_BAD_XI
    assert torch.isnan(xi[10:14]).all() and not torch.isnan(xi[:10]).any()


def test_computing_xi_end_to_end():
    """Score proxy on the matrix cores -> weights -> designed tables -> sampled cutoffs, on the
    7B-width mini workload, each stage against the oracle fed the same inputs."""
    wl = synth.make_workload(MINI7B)
    cfg = wl.cfg
    h = torch.from_numpy(wl.hidden_bits.view(np.int16)).cuda().view(torch.bfloat16)
    W = torch.from_numpy(wl.w_bits.view(np.int16)).cuda().view(torch.bfloat16)
    prox = pspo.score_proxy(h, W, _cuda(wl.target_full, torch.int32), wl.total_tokens, want_logp=False)
    gamma = prox["gamma"].cpu().numpy()
    ref_g = osp.score_proxy(wl.hidden_bits, wl.w_bits, wl.target_full)["gamma"]
    np.testing.assert_allclose(gamma, ref_g, rtol=1e-4)
    ids, logp = synth.make_topk(wl)
    wts, err = _weights(wl, gamma, ids, logp, want_parts=False)
    assert err == 0
    w_ref = cd.proxy_weights(gamma, ids, logp, wl.lengths, wl.rewards, cfg.P, cfg.K)["w"]
    np.testing.assert_allclose(wts["w"].cpu().numpy(), w_ref, rtol=1e-12, atol=1e-12)
    _, xi_off, total = _layout(wl)
    budget = 128.0
    xi = pspo.design_cutoffs(wts["w"], _cuda(xi_off, torch.int64), cfg.P, total, budget)
    xi_np = xi.cpu().numpy()
    np.testing.assert_allclose(xi_np, cd.design_tables(w_ref, xi_off, budget), rtol=1e-10)
    # the designed tables drive the sampler like any other table
    H = pspo.sample_cutoffs(xi, _cuda(xi_off, torch.int64), _cuda(wl.lengths, torch.int32), cfg.P, cfg.K, seed=3)
    H_ref = ocut.sample_cutoffs(xi_np, xi_off, wl.lengths, cfg.P, cfg.K, 3, 0)
    assert np.array_equal(H.cpu().numpy(), H_ref)
    for p in range(cfg.P):
        assert xi_np[xi_off[p]:xi_off[p + 1]].sum() == pytest.approx(budget, rel=1e-9)


@pytest.mark.parametrize("variant", [cd.OPTIMIZED, cd.HEURISTIC])
def test_design_cutoffs_lds_and_global_paths(variant):
    """Prompt horizons on both sides of the solve's two LDS limits (its weights and block
    stack in the 160 KB of LDS up to T = 8192, the weights alone up to T = 20480, both in
    device memory beyond), in one call, against the oracle; the no-allocation entry point
    gives the same bits."""
    T = np.array([100, 8191, 8192, 8193, 20480, 20481, 30000], dtype=np.int64)
    xi_off = np.concatenate([[0], np.cumsum(T)]).astype(np.int64)
    P, total = len(T), int(xi_off[-1])
    w = _random_weights(xi_off, 17)
    budget = 600.0
    print(f"[design paths] T = {T.tolist()} variant={variant}", flush=True)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    tw, toff = _cuda(w, torch.float64), _cuda(xi_off, torch.int64)
    xi = pspo.design_cutoffs(tw, toff, P, total, budget, variant, err_flag=err)
    out = torch.full((total,), float("nan"), dtype=torch.float64, device="cuda")
    xi_na = pspo.design_cutoffs_noalloc(tw, toff, P, total, budget, out, variant=variant, err_flag=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    assert torch.equal(xi, xi_na)
    np.testing.assert_allclose(xi.cpu().numpy(), cd.design_tables(w, xi_off, budget, variant), rtol=1e-12)
