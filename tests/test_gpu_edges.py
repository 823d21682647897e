"""GPU: token counts on and around the tile edges, against the float64 oracle
(loss call and score proxy).

The products tile the tokens by 256 (forward, logit gradient), 384 (dH) and
pad them to 768; the forward and backward token sets are compacted on the
device.  Each case calls pspo_loss_fwd_bwd directly on seeded packed inputs
with N at such an edge (and the clip range wide enough that every token
reaches the backward, so the backward token count sits on the same edge), at
a vocabulary that is a whole number of 384-row tiles and one that is not, and
a width that is no multiple of 64.  Loss, per-token log-probs, both gradients
and the backward-token count are compared with the oracle.
"""
import numpy as np
import pytest
import torch

from oracle import ppo_head as ohead
from paper_2606_29758_amd import pspo, synth

from parity_util import GRAD_REL_L2, LOGP_ATOL, LOSS_RTOL, f32, rel_l2

pytestmark = pytest.mark.gpu

EDGES = [1, 2, 255, 256, 257, 383, 384, 385, 767, 768, 769, 1537]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    pspo.load()


def _bits_tensor(bits):
    return torch.from_numpy(bits.view(np.int16)).to("cuda").view(torch.bfloat16)


@pytest.mark.parametrize("V,d", [(1152, 128), (1000, 200)])
@pytest.mark.parametrize("N", EDGES)
def test_token_count_edges(N, V, d):
    rng = np.random.default_rng(7919 * N + V + d)
    R = 5
    h = synth.round_to_bf16_bits(rng.normal(0.0, 1.0, (N, d)).astype(np.float32))
    W = synth.round_to_bf16_bits(rng.normal(0.0, 0.05, (V, d)).astype(np.float32))
    tgt = rng.integers(0, V, N).astype(np.int32)
    seq = np.sort(rng.integers(0, R, N)).astype(np.int32)
    adv = rng.choice([-1.0, 1.0], R).astype(np.float32)
    weight = (1.0 + rng.random(N)).astype(np.float32)
    lp_old = (ohead.target_logprob(h, W, tgt) + rng.normal(0.0, 0.05, N)).astype(np.float32)
    eps, scale = 0.9, 1.0 / R
    ref = ohead.loss_fwd_bwd(h, W, tgt, lp_old, weight, seq, adv, f32(eps), f32(eps), f32(scale))
    assert np.all(ref["delta"] != 0)   # every token reaches the backward

    t = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a)).to(device="cuda", dtype=dt)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    out = pspo.loss_fwd_bwd(_bits_tensor(h), _bits_tensor(W), t(tgt, torch.int32), t(lp_old, torch.float32),
                            t(weight, torch.float32), t(seq, torch.int32), t(adv, torch.float32), N, eps, eps, scale,
                            err_flag=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    loss = float(out["loss"].item())
    assert abs(loss - ref["loss"]) <= LOSS_RTOL * abs(ref["loss"]), (loss, ref["loss"])
    np.testing.assert_allclose(out["logp_new"].cpu().numpy(), ref["logp_new"], rtol=0, atol=LOGP_ATOL)
    assert int(out["stats"][4].item()) == N
    assert rel_l2(out["d_hidden"].cpu().numpy(), ref["d_hidden"]) <= GRAD_REL_L2
    assert rel_l2(out["d_w_head"].cpu().numpy(), ref["d_w"]) <= GRAD_REL_L2


@pytest.mark.parametrize("V,d", [(1152, 128), (1000, 200)])
@pytest.mark.parametrize("N", EDGES)
def test_score_proxy_token_count_edges(N, V, d):
    from oracle import score_proxy as osp
    rng = np.random.default_rng(104729 * N + V + d)
    h = synth.round_to_bf16_bits(rng.normal(0.0, 1.0, (N, d)).astype(np.float32))
    W = synth.round_to_bf16_bits(rng.normal(0.0, 0.05, (V, d)).astype(np.float32))
    tgt = rng.integers(0, V, N).astype(np.int32)
    ref = osp.score_proxy(h, W, tgt)
    out = pspo.score_proxy(_bits_tensor(h), _bits_tensor(W), torch.from_numpy(tgt).to("cuda"), N, want_p_sq=True)
    torch.cuda.synchronize()
    np.testing.assert_allclose(out["gamma"].cpu().numpy().astype(np.float64), ref["gamma"], rtol=1e-4, atol=0)
    np.testing.assert_allclose(out["p_sq"].cpu().numpy().astype(np.float64), ref["p_sq"], rtol=1e-4, atol=0)
    assert np.max(np.abs(out["logp"].cpu().numpy().astype(np.float64) - ref["logp"])) <= LOGP_ATOL


# vocabularies around the 384-row tile (down to a single entry) and widths that are no
# multiple of 32 or 64 (down to one 16-byte piece per row), for the loss call and the
# score proxy; a single-entry vocabulary has p = 1 and every gradient exactly zero
SHAPES = [(1, 128, 300), (2, 8, 769), (383, 24, 300), (384, 40, 257), (385, 264, 300), (767, 520, 200),
          (769, 136, 385), (3001, 8, 1), (3001, 200, 1537)]


@pytest.mark.parametrize("V,d,N", SHAPES)
def test_vocabulary_and_width_edges(V, d, N):
    from oracle import score_proxy as osp
    print(f"[edges] V={V} d={d} N={N}", flush=True)
    rng = np.random.default_rng(31 * V + 7 * d + N)
    R = 5
    h = synth.round_to_bf16_bits(rng.normal(0.0, 1.0, (N, d)).astype(np.float32))
    W = synth.round_to_bf16_bits(rng.normal(0.0, 0.3 / np.sqrt(d) * 4, (V, d)).astype(np.float32))
    tgt = rng.integers(0, V, N).astype(np.int32)
    seq = np.sort(rng.integers(0, R, N)).astype(np.int32)
    adv = rng.choice([-1.0, 0.0, 1.0], R).astype(np.float32)
    weight = (1.0 + rng.random(N)).astype(np.float32)
    lp_old = (ohead.target_logprob(h, W, tgt) + rng.normal(0.0, 0.2, N)).astype(np.float32)
    el, eh, scale = 0.2, 0.28, 1.0 / R
    ref = ohead.loss_fwd_bwd(h, W, tgt, lp_old, weight, seq, adv, f32(el), f32(eh), f32(scale))

    t = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a)).to(device="cuda", dtype=dt)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    out = pspo.loss_fwd_bwd(_bits_tensor(h), _bits_tensor(W), t(tgt, torch.int32), t(lp_old, torch.float32),
                            t(weight, torch.float32), t(seq, torch.int32), t(adv, torch.float32), N, el, eh, scale,
                            err_flag=err)
    prox = pspo.score_proxy(_bits_tensor(h), _bits_tensor(W), t(tgt, torch.int32), N, want_p_sq=True)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    loss = float(out["loss"].item())
    assert abs(loss - ref["loss"]) <= LOSS_RTOL * max(abs(ref["loss"]), 1e-3 * ref["abs_mass"]), (loss, ref["loss"])
    np.testing.assert_allclose(out["logp_new"].cpu().numpy(), ref["logp_new"], rtol=0, atol=LOGP_ATOL)
    st = out["stats"].cpu().numpy()
    A = adv.astype(np.float64)[seq]
    assert st[2] == np.count_nonzero(A == 0) and st[4] == np.count_nonzero(ref["delta"])
    dh, dw = out["d_hidden"].cpu().numpy(), out["d_w_head"].cpu().numpy()
    if V == 1:   # p = 1: every logit-gradient row is zero (up to the log-prob's rounding)
        assert np.abs(dh).max() <= 1e-5 and np.abs(dw).max() <= 1e-5
    else:
        assert rel_l2(dh, ref["d_hidden"]) <= GRAD_REL_L2
        assert rel_l2(dw, ref["d_w"]) <= GRAD_REL_L2
    pref = osp.score_proxy(h, W, tgt)
    assert np.max(np.abs(prox["logp"].cpu().numpy().astype(np.float64) - pref["logp"])) <= LOGP_ATOL
    np.testing.assert_allclose(prox["p_sq"].cpu().numpy().astype(np.float64), pref["p_sq"], rtol=1e-4, atol=0)
    np.testing.assert_allclose(prox["gamma"].cpu().numpy().astype(np.float64), pref["gamma"], rtol=1e-4,
                               atol=1e-6 * float(np.max(pref["gamma"], initial=0.0)) if V > 1 else 1e-5)
