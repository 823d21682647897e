"""GPU parity of the output-head score proxy (App. D) through the C ABI, against the
float64 oracle.

Bar: gamma and ||p||^2 within relative 1e-4 per token, log p(o) within 2e-4, on
every completion token of the small workloads (several tiles in every dimension,
ragged vocabulary and token tails), on a peaked head where p(o) -> 1 (the regime
where 1 - 2 p(o) + ||p||^2 cancels), and on sampled tokens plus every token's
log-prob at full size.  The 1e-4 bound: each logit carries a float32
accumulation error of about sqrt(d) 2^-24 |h||w| (under 1e-5 here), which moves
exp(z - m) and the sums built from it by the same relative amount; the norm
||h||^2 is summed in float32 from the exact bf16 values.
"""
import numpy as np
import pytest
import torch

from oracle import score_proxy as osp
from oracle.ppo_head import as_f64
from paper_2606_29758_amd import pspo, synth

from parity_util import GOLDEN, LOGP_ATOL

pytestmark = pytest.mark.gpu

GAMMA_RTOL = 1e-4

MINI = {
    "mini7b": synth.custom("mini7b", "qwen7b", P=2, K=2, length_law=("uniform", 150, 420), data_seed=31),
    "mini1p5b": synth.custom("mini1p5b", "qwen1.5b", P=2, K=3, length_law=("uniform", 60, 300), data_seed=21),
}


def _np(t):
    return t.detach().cpu().numpy()


def _run(h_bits, w_bits, target, want_p_sq=True):
    dev = "cuda"
    h = torch.from_numpy(h_bits.view(np.int16)).to(dev).view(torch.bfloat16)
    w = torch.from_numpy(w_bits.view(np.int16)).to(dev).view(torch.bfloat16)
    t = torch.from_numpy(np.ascontiguousarray(target, dtype=np.int32)).to(dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    out = pspo.score_proxy(h, w, t, h.shape[0], want_logp=True, want_p_sq=want_p_sq, err_flag=err)
    torch.cuda.synchronize()
    return out, int(err.item())


def _compare(out, ref, rtol=GAMMA_RTOL):
    g = _np(out["gamma"]).astype(np.float64)
    np.testing.assert_allclose(g, ref["gamma"], rtol=rtol, atol=0)
    np.testing.assert_allclose(_np(out["p_sq"]).astype(np.float64), ref["p_sq"], rtol=rtol, atol=0)
    assert np.max(np.abs(_np(out["logp"]).astype(np.float64) - ref["logp"])) <= LOGP_ATOL
    rel = np.max(np.abs(g - ref["gamma"]) / ref["gamma"])
    print(f"gamma max rel {rel:.2e}")


@pytest.mark.parametrize("name", ["tiny", "mini7b", "mini1p5b"])
def test_score_proxy_parity(name):
    wl = synth.make_workload(MINI.get(name) or synth.CONFIGS[name])
    out, err = _run(wl.hidden_bits, wl.w_bits, wl.target_full)
    assert err == 0
    ref = osp.score_proxy(wl.hidden_bits, wl.w_bits, wl.target_full)
    _compare(out, ref)


def test_score_proxy_peaked_head():
    """A sharp head and targets at the most likely token: p(o) close to 1, gamma tiny."""
    rng = np.random.default_rng(11)
    wl = synth.make_workload("tiny")
    h_bits = wl.hidden_bits
    w = rng.standard_normal(wl.w_bits.shape) * 1.5
    w_bits = synth.round_to_bf16_bits(w)
    z = as_f64(h_bits) @ as_f64(w_bits).T
    target = z.argmax(axis=1).astype(np.int32)
    ref = osp.score_proxy(h_bits, w_bits, target)
    po = np.exp(ref["logp"])
    assert np.median(po) > 0.9 and ref["gamma"].min() < 1e-3 * (as_f64(h_bits) ** 2).sum(axis=1).max()
    out, err = _run(h_bits, w_bits, target)
    assert err == 0
    # large logits: the float32 error of each logit is about sqrt(d) 2^-24 max|z|, and
    # gamma picks it up at most four times (two exp ratios, squared)
    rtol = 4 * 2 * np.sqrt(wl.cfg.d) * 2.0 ** -24 * np.abs(z).max()
    _compare(out, ref, rtol=max(GAMMA_RTOL, rtol))


def test_score_proxy_bad_target():
    wl = synth.make_workload("tiny")
    target = wl.target_full.copy()
    target[5] = wl.cfg.V            # out of range
    out, err = _run(wl.hidden_bits, wl.w_bits, target)
    assert err == pspo.DEVERR_TARGET
    g = _np(out["gamma"])
    assert np.isnan(g[5]) and np.isfinite(np.delete(g, 5)).all()


@pytest.mark.parametrize("name", ["qwen7b"])
def test_score_proxy_full_size(name):
    """Every completion token of the 7B-shaped batch, as the cutoff design would run it."""
    wl = synth.make_workload(name)
    print(f"[{name}] {wl.total_tokens} tokens", flush=True)
    out, err = _run(wl.hidden_bits, wl.w_bits, wl.target_full, want_p_sq=False)
    assert err == 0
    # every token's log p(o) against the stored oracle values (old log-prob = oracle + noise)
    stored = synth.load_stored_logp_old(wl, GOLDEN).astype(np.float64) - wl.lp_noise
    lp = _np(out["logp"]).astype(np.float64)
    assert np.max(np.abs(lp - stored)) <= LOGP_ATOL + 1e-5   # + float32 rounding of the stored values
    # sampled tokens against the oracle one by one
    rng = np.random.default_rng(3)
    idx = np.unique(np.concatenate([[0, wl.total_tokens - 1], rng.choice(wl.total_tokens, 46, replace=False)]))
    ref = osp.score_proxy(wl.hidden_bits[idx], wl.w_bits, wl.target_full[idx])
    np.testing.assert_allclose(_np(out["gamma"])[idx].astype(np.float64), ref["gamma"], rtol=GAMMA_RTOL)
    # bounds that hold for every token: 0 <= gamma <= 2 ||h||^2
    g = out["gamma"].double()
    h = torch.from_numpy(wl.hidden_bits.view(np.int16)).cuda().view(torch.bfloat16)
    hn = torch.cat([h[i:i + 16384].double().pow(2).sum(dim=1) for i in range(0, h.shape[0], 16384)])
    assert bool((g >= 0).all()) and bool((g <= 2 * hn * (1 + 1e-5)).all())
    print(f"[{name}] proxy checks hold", flush=True)
