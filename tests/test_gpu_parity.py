"""GPU parity: the HIP path (through the C ABI) against the float64 oracle.

Bar: bit-exact cutoffs, packing and weights; loss relative error <= 1e-4;
d_hidden and d_w_head relative L2 error <= 1e-2 (bf16 inputs, fp32
accumulation, bf16 logit gradients away from the target entries); per-token
log-probs within 2e-4.  Small workloads are compared element by element.  The
full-size workloads, in the launch configuration the benchmark times, are
compared on every token's log-prob (against the oracle's, stored with the
old log-probs), on the loss (the oracle's, from those log-probs), on 64 rows of
d_w_head and 48 rows of d_hidden that the oracle computes one by one, and on
identities that hold at any size.
"""
import dataclasses

import numpy as np
import pytest
import torch

from oracle import ppo_head as ohead
from paper_2606_29758_amd import pipeline, pspo, synth

from parity_util import (GRAD_REL_L2, LOGP_ATOL, LOSS_RTOL, ambiguous_clip, f32, logp_old_for,
                         oracle_logp_old, oracle_loss, oracle_sample_pack, rel_l2)

pytestmark = pytest.mark.gpu

MINI = {
    "tiny": synth.CONFIGS["tiny"],
    "tiny_full": synth.custom("tiny_full", "tiny", full_trajectory=True),
    # the 7B and 1.5B vocabulary and width with a few short completions: several
    # tiles in every dimension and ragged tails (V = 151936 is not a multiple of 256)
    "mini7b": synth.custom("mini7b", "qwen7b", P=2, K=2, length_law=("uniform", 150, 420), data_seed=31),
    "mini1p5b": synth.custom("mini1p5b", "qwen1.5b", P=2, K=3, length_law=("uniform", 60, 300), data_seed=21),
    # odd shapes: a vocabulary that is no multiple of 32 (2.6 tiles of 384, one chunk) with a width
    # of 6 K steps, and one of three chunks whose last ends in a partial tile (7B width)
    "odd_small": synth.custom("odd_small", "tiny", d=192, V=1000, P=2, K=3, length_law=("uniform", 20, 90),
                              data_seed=41),
    "odd_chunks": synth.custom("odd_chunks", "qwen7b", V=130003, P=2, K=3, length_law=("uniform", 60, 160),
                               data_seed=49),
    # the 7B width and vocabulary with short completions (the oracle's logp_old of a rescaled head
    # is recomputed per test)
    "short7b": synth.custom("short7b", "qwen7b", P=2, K=2, length_law=("uniform", 40, 90), data_seed=33),
    # a width that is a multiple of 8 but not of 32 or 64 (K padded with zeros in the products)
    "odd_d": synth.custom("odd_d", "tiny", d=200, V=1500, P=2, K=3, length_law=("uniform", 40, 120), data_seed=43),
}
_CACHE = {}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    pspo.load()


def _workload(name):
    if name not in _CACHE:
        cfg = MINI.get(name) or synth.CONFIGS[name]
        wl = synth.make_workload(cfg)
        _CACHE.clear()   # keep at most one (possibly multi-GB) workload alive
        _CACHE[name] = (wl, logp_old_for(wl))
    return _CACHE[name]


def _to_np(t):
    return t.detach().cpu().numpy()


def _check_pack(out, H, pk):
    N = pk["n_tokens"]
    assert np.array_equal(_to_np(out["cutoffs"]), H)
    got = out["pack"]
    assert int(_to_np(got["n_tokens"])[0]) == N
    for key in ("cu_seqlens", "full_off"):
        assert np.array_equal(_to_np(got[key]), pk[key]), key
    for key in ("src_row", "seq_id", "weight", "target", "logp_old"):
        assert np.array_equal(_to_np(got[key])[:N], pk[key]), key


# ---------------------------------------------------------------- sampler + packer


@pytest.mark.parametrize("name", ["tiny", "qwen1.5b", "qwen7b", "qwen7b_long", "qwen7b_full"])
@pytest.mark.parametrize("seed,offset", [(0, 0), (7, 3), (2 ** 40 + 5, 2 ** 33 + 1)])
def test_sample_and_pack_bitwise(name, seed, offset):
    wl = synth.make_workload(name, with_matrices=False)
    cfg = wl.cfg
    lp = wl.lp_noise.astype(np.float32)   # any float32 per-token array exercises the gather
    dev = "cuda"
    t = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a)).to(dev, dt)
    xi, xi_off, lengths = t(wl.xi, torch.float64), t(wl.xi_off, torch.int64), t(wl.lengths, torch.int32)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    cut = pspo.sample_cutoffs(xi, xi_off, lengths, cfg.P, cfg.K, seed, offset, err_flag=err)
    got = pspo.pack_prefixes(cut, lengths, xi, xi_off, cfg.P, cfg.K, wl.total_tokens,
                             target_full=t(wl.target_full, torch.int32), logp_old_full=t(lp, torch.float32),
                             err_flag=err)
    H, pk = oracle_sample_pack(wl, lp, seed, offset)
    _check_pack(dict(cutoffs=cut, pack=got), H, pk)
    assert int(err.item()) == 0
    if cfg.full_trajectory:
        assert np.array_equal(H, wl.lengths) and np.all(pk["weight"] == 1.0)


def test_hidden_gather_bitwise():
    wl, lp = _workload("mini7b")
    dw = pipeline.upload(wl, lp)
    step = pipeline.Step(dw)
    pk_gpu = step.sample_and_pack(seed=5)
    H, pk = oracle_sample_pack(wl, lp, 5)
    N = pk["n_tokens"]
    got = _to_np(pk_gpu["hidden"].view(torch.int16))[:N].view(np.uint16)
    assert np.array_equal(got, wl.hidden_bits[pk["src_row"]])


# ---------------------------------------------------------------- loss fwd + bwd


def _compare_loss(out, ref):
    loss = float(out["loss"].item())
    assert abs(loss - ref["loss"]) <= LOSS_RTOL * abs(ref["loss"]), (loss, ref["loss"])
    lp = _to_np(out["logp_new"]).astype(np.float64)
    assert np.max(np.abs(lp - ref["logp_new"])) <= LOGP_ATOL
    assert _to_np(out["stats"])[0] == pytest.approx(ref["abs_mass"], rel=LOSS_RTOL)
    e_h = rel_l2(_to_np(out["d_hidden"]), ref["d_hidden"])
    e_w = rel_l2(_to_np(out["d_w_head"]), ref["d_w"])
    print(f"loss rel {abs(loss - ref['loss']) / abs(ref['loss']):.2e}  dH relL2 {e_h:.2e}  dW relL2 {e_w:.2e}")
    assert e_h <= GRAD_REL_L2 and e_w <= GRAD_REL_L2


@pytest.mark.parametrize("name,seed", [("tiny", 0), ("tiny", 1), ("tiny", 123456789), ("tiny_full", 0),
                                       ("mini1p5b", 0), ("mini7b", 3), ("odd_small", 0), ("odd_chunks", 2),
                                       ("odd_d", 1)])
def test_loss_parity(name, seed):
    wl, lp = _workload(name)
    cfg = wl.cfg
    dw = pipeline.upload(wl, lp)
    out = pipeline.Step(dw)(seed=seed)
    torch.cuda.synchronize()
    H, pk = oracle_sample_pack(wl, lp, seed)
    _check_pack(out, H, pk)
    ref = oracle_loss(wl, pk)
    assert not ambiguous_clip(ref, cfg.eps_low, cfg.eps_high).any()
    _compare_loss(out, ref)
    # the clip mask and degenerate groups agree exactly
    A = wl.advantage[pk["seq_id"]]
    st = _to_np(out["stats"])
    assert int(st[1]) == int(np.sum((A != 0) & (ref["mu"] == 0)))
    assert int(st[2]) == int(np.sum(A == 0))
    assert st[3] == float(pk["weight"].max())
    # the backward ran over exactly the tokens with a nonzero logit-gradient row
    assert int(st[4]) == int(np.sum(ref["delta"] != 0))
    assert int(out["pack"]["n_tokens"].item()) == pk["n_tokens"]


@pytest.mark.parametrize("name,eps_low,eps_high,adv_norm", [("mini7b", 0.2, 0.28, "mean"),
                                                            ("tiny", 0.1, 0.1, "std"),
                                                            ("mini1p5b", 0.2, 0.28, "std")])
def test_loss_variants(name, eps_low, eps_high, adv_norm):
    """Loss variants of the paper's baselines as parameters: asymmetric clip range
    (clip-higher) and std-normalised group advantages."""
    wl, lp = _workload(name)
    cfg = dataclasses.replace(wl.cfg, eps_low=eps_low, eps_high=eps_high, adv_norm=adv_norm)
    adv = synth.make_workload(cfg, with_matrices=False).advantage
    wl1 = synth.Workload(**{**wl.__dict__, "cfg": cfg, "advantage": adv})
    out = pipeline.Step(pipeline.upload(wl1, lp))(seed=5)
    torch.cuda.synchronize()
    H, pk = oracle_sample_pack(wl1, lp, 5)
    _check_pack(out, H, pk)
    ref = oracle_loss(wl1, pk)
    assert not ambiguous_clip(ref, eps_low, eps_high).any()
    _compare_loss(out, ref)
    A = adv[pk["seq_id"]]
    st = _to_np(out["stats"])
    assert int(st[1]) == int(np.sum((A != 0) & (ref["mu"] == 0)))
    assert int(st[4]) == int(np.sum(ref["delta"] != 0))


@pytest.mark.parametrize("name", ["tiny", "mini7b"])
def test_without_logp_is_identical(name):
    """Without per-token log-probs the forward skips zero-advantage tokens; every other
    output is bitwise the same, and still matches the oracle."""
    wl, lp = _workload(name)
    adv = wl.advantage.copy()
    adv[:wl.cfg.K] = 0.0      # one group with equal rewards, so that some tokens are skipped
    wl = synth.Workload(**{**wl.__dict__, "advantage": adv})
    step = pipeline.Step(pipeline.upload(wl, lp))
    a = step(seed=6)
    la, dha, dwa, sa = (a[k].clone() for k in ("loss", "d_hidden", "d_w_head", "stats"))
    b = step(seed=6, want_logp=False)
    torch.cuda.synchronize()
    assert b["logp_new"] is None
    assert torch.equal(la, b["loss"]) and torch.equal(sa, b["stats"])
    assert torch.equal(dha, b["d_hidden"]) and torch.equal(dwa, b["d_w_head"])
    A = wl.advantage[_to_np(a["pack"]["seq_id"][:a["N"]])]
    assert 0 < np.sum(A == 0) < a["N"]   # the skip is exercised
    assert int(step.err.item()) == 0
    H, pk = oracle_sample_pack(wl, lp, 6)
    ref = oracle_loss(wl, pk)
    assert abs(float(b["loss"].item()) - ref["loss"]) <= LOSS_RTOL * abs(ref["loss"])
    assert rel_l2(_to_np(b["d_hidden"]), ref["d_hidden"]) <= GRAD_REL_L2
    assert rel_l2(_to_np(b["d_w_head"]), ref["d_w"]) <= GRAD_REL_L2


@pytest.mark.parametrize("name", ["tiny", "mini7b", "mini1p5b", "odd_small", "odd_chunks"])
@pytest.mark.parametrize("want_logp", [True, False])
def test_kept_logits_match_recompute(name, want_logp):
    """With PSPO_KEEP_LOGITS the forward keeps the first vocabulary chunk's logits (as fp16
    offsets from each tile's per-column maximum) and the backward turns them into that
    chunk's logit gradient without a recomputing product.  The forward outputs (loss,
    log-probs, stats) are bitwise those of the default path, which recomputes every chunk;
    the gradients differ only by the fp16 rounding of the kept offsets, and both match the
    oracle.  tiny has one chunk (the whole padded vocabulary); the 7B and 1.5B widths have
    several."""
    wl, lp = _workload(name)
    step = pipeline.Step(pipeline.upload(wl, lp))
    pk = step.sample_and_pack(seed=11)
    N = int(pk["n_tokens"].item())
    a = step.loss(pk, N, want_logp=want_logp)
    ka = {k: a[k].clone() for k in ("loss", "d_hidden", "d_w_head", "stats")}
    ka_lp = a["logp_new"].clone() if want_logp else None
    b = step.loss(pk, N, flags=pspo.PSPO_KEEP_LOGITS, want_logp=want_logp)
    torch.cuda.synchronize()
    for k in ("loss", "stats"):
        assert torch.equal(ka[k], b[k]), k
    if want_logp:
        assert torch.equal(ka_lp, b["logp_new"])
    # kept vs recomputed chunk: the fp16 rounding of the kept offsets
    for k in ("d_hidden", "d_w_head"):
        assert rel_l2(_to_np(ka[k]), _to_np(b[k]).astype(np.float64)) <= 1e-3, k
    assert int(step.err.item()) == 0
    assert float(ka["stats"][4].item()) > 32   # several 32-token K steps of backward tokens
    H, opk = oracle_sample_pack(wl, lp, 11)
    ref = oracle_loss(wl, opk)
    for out in (ka, b):
        assert rel_l2(_to_np(out["d_hidden"]), ref["d_hidden"]) <= GRAD_REL_L2
        assert rel_l2(_to_np(out["d_w_head"]), ref["d_w"]) <= GRAD_REL_L2


def _scaled_w(wl, k):
    """The same workload with W multiplied by 2^k (exact in bf16, so the logits are exactly
    2^k times larger); logp_old recomputed by the oracle for the new head."""
    f = (wl.w_bits.astype(np.uint32) << 16).view(np.float32) * np.float32(2.0 ** k)
    wl2 = synth.Workload(**{**wl.__dict__, "w_bits": (f.view(np.uint32) >> 16).astype(np.uint16)})
    return wl2, oracle_logp_old(wl2)


@pytest.mark.parametrize("name,k,seed", [("tiny", 7, 0), ("short7b", 4, 3)])
def test_large_logits(name, k, seed):
    """Logits of standard deviation ~20-30 (W scaled by 2^k): peaked softmax rows, targets
    dozens of nats below the tile maxima, kept fp16 offsets far into their coarse range.
    The default path (every chunk recomputed) and the kept-chunk path both match the oracle,
    agree with each other to ~1e-4 on the gradients, and bitwise on loss and log-probs."""
    wl, _ = _workload(name)
    wl, lp = _scaled_w(wl, k)
    cfg = wl.cfg
    step = pipeline.Step(pipeline.upload(wl, lp))
    out = step(seed=seed)
    ka = {key: out[key].clone() for key in ("loss", "d_hidden", "d_w_head", "logp_new", "stats")}
    torch.cuda.synchronize()
    H, pk = oracle_sample_pack(wl, lp, seed)
    ref = oracle_loss(wl, pk)
    assert not ambiguous_clip(ref, cfg.eps_low, cfg.eps_high).any()
    assert np.median(ref["logp_new"]) < -10.0   # the regime this test is for
    _compare_loss(ka, ref)
    pkg = step.sample_and_pack(seed)
    N = int(pkg["n_tokens"].item())
    b = step.loss(pkg, N, flags=pspo.PSPO_KEEP_LOGITS)
    torch.cuda.synchronize()
    assert torch.equal(ka["loss"], b["loss"]) and torch.equal(ka["logp_new"], b["logp_new"])
    for key in ("d_hidden", "d_w_head"):
        assert rel_l2(_to_np(ka[key]), _to_np(b[key]).astype(np.float64)) <= 1e-3, key
    assert int(step.err.item()) == 0


def test_deterministic():
    wl, lp = _workload("tiny")
    step = pipeline.Step(pipeline.upload(wl, lp))
    a = step(seed=1)
    la, dha, dwa = a["loss"].clone(), a["d_hidden"].clone(), a["d_w_head"].clone()
    b = step(seed=1)
    assert torch.equal(la, b["loss"]) and torch.equal(dha, b["d_hidden"]) and torch.equal(dwa, b["d_w_head"])


def test_accumulate_flag():
    wl, lp = _workload("tiny")
    step = pipeline.Step(pipeline.upload(wl, lp))
    one = step(seed=2)["d_w_head"].clone()
    step.d_w.zero_()
    pk = step.sample_and_pack(seed=2)
    N = int(pk["n_tokens"].item())
    step.loss(pk, N, flags=pspo.PSPO_ACCUMULATE_DW)
    step.loss(pk, N, flags=pspo.PSPO_ACCUMULATE_DW)
    assert torch.allclose(step.d_w, 2 * one, rtol=1e-6, atol=0)


def test_empty_prefixes():
    """Every cutoff 0 (xi_1 tiny): N = 0, loss 0, d_w_head zeroed."""
    wl, lp = _workload("tiny")
    wl0 = synth.Workload(**{**wl.__dict__, "xi": np.full_like(wl.xi, 2.0 ** -40)})
    step = pipeline.Step(pipeline.upload(wl0, lp))
    step.d_w.fill_(7.0)
    out = step(seed=0)
    assert out["N"] == 0
    assert float(out["loss"].item()) == 0.0
    assert not torch.any(out["d_w_head"])


def test_zero_advantage():
    wl, lp = _workload("tiny")
    wl0 = synth.Workload(**{**wl.__dict__, "advantage": np.zeros_like(wl.advantage)})
    out = pipeline.Step(pipeline.upload(wl0, lp))(seed=0)
    assert float(out["loss"].item()) == 0.0
    assert not torch.any(out["d_hidden"]) and not torch.any(out["d_w_head"])
    assert int(out["stats"][2].item()) == out["N"]
    assert int(out["stats"][4].item()) == 0   # no token enters the backward products


def test_all_tokens_active():
    """No clipping and no zero advantage: every token enters the backward."""
    wl, lp = _workload("tiny")
    cfg = dataclasses.replace(wl.cfg, eps_low=0.9, eps_high=0.9)
    adv = np.where(wl.advantage >= 0, 1.0, -1.0).astype(wl.advantage.dtype)
    wl1 = synth.Workload(**{**wl.__dict__, "cfg": cfg, "advantage": adv})
    out = pipeline.Step(pipeline.upload(wl1, lp))(seed=4)
    torch.cuda.synchronize()
    H, pk = oracle_sample_pack(wl1, lp, 4)
    ref = oracle_loss(wl1, pk)
    assert np.all(ref["delta"] != 0)
    assert int(out["stats"][4].item()) == out["N"] == pk["n_tokens"]
    _compare_loss(out, ref)


def test_device_error_flags():
    wl, lp = _workload("tiny")
    dw = pipeline.upload(wl, lp)
    step = pipeline.Step(dw)
    pk = step.sample_and_pack(seed=0)
    N = int(pk["n_tokens"].item())
    cfg = wl.cfg
    # a target id outside [0, V): flagged, that token contributes nothing
    tgt = pk["target"].clone()
    tgt[3] = cfg.V
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    pspo.loss_fwd_bwd(pk["hidden"], dw.w_head, tgt, pk["logp_old"], pk["weight"], pk["seq_id"], dw.advantage, N,
                      cfg.eps_low, cfg.eps_high, cfg.loss_scale, err_flag=err)
    assert int(err.item()) & pspo.DEVERR_TARGET
    # a seq_id outside [0, R)
    seq = pk["seq_id"].clone()
    seq[0] = cfg.R
    err.zero_()
    pspo.loss_fwd_bwd(pk["hidden"], dw.w_head, pk["target"], pk["logp_old"], pk["weight"], seq, dw.advantage, N,
                      cfg.eps_low, cfg.eps_high, cfg.loss_scale, err_flag=err)
    assert int(err.item()) & pspo.DEVERR_SEQ_ID
    # an increasing xi table
    bad = dw.xi.clone()
    bad[5] = 1.0
    bad[4] = 0.5
    err.zero_()
    pspo.sample_cutoffs(bad, dw.xi_off, dw.lengths, cfg.P, cfg.K, 0, 0, err_flag=err)
    assert int(err.item()) & pspo.DEVERR_BAD_XI
    # capacity below the kept-token count: flagged, n_tokens clipped, nothing written past it
    err.zero_()
    cut = pspo.sample_cutoffs(dw.xi, dw.xi_off, dw.lengths, cfg.P, cfg.K, 0, 0)
    small = pspo.pack_prefixes(cut, dw.lengths, dw.xi, dw.xi_off, cfg.P, cfg.K, 10,
                               target_full=dw.target_full, logp_old_full=dw.logp_old_full,
                               hidden_full=dw.hidden_full, err_flag=err)
    assert int(err.item()) & pspo.DEVERR_CAPACITY
    assert int(small["n_tokens"].item()) == 10


# ---------------------------------------------------------------- target entries in float32


@pytest.mark.parametrize("name,seed", [("tiny", 0), ("mini7b", 3), ("mini1p5b", 0)])
def test_target_entries_exact(name, seed):
    """The target entry of each logit-gradient row, delta (1 - p(o)), is applied in float32
    (d_hidden += g W[o], d_w_head[o] += g h); only the other entries, -delta p, pass through
    bf16.  With a flat softmax the target entry carries almost all of a row's norm, so the
    gradients sit far inside the gradient tolerance of the parity tests (GRAD_REL_L2): the
    bound here is a hundredth of it
    (a path that rounded the target entries to bf16 lands at ~1.5e-3)."""
    wl, lp = _workload(name)
    out = pipeline.Step(pipeline.upload(wl, lp))(seed=seed)
    torch.cuda.synchronize()
    H, pk = oracle_sample_pack(wl, lp, seed)
    ref = oracle_loss(wl, pk)
    e_h = rel_l2(_to_np(out["d_hidden"]), ref["d_hidden"])
    e_w = rel_l2(_to_np(out["d_w_head"]), ref["d_w"])
    print(f"[{name}] dH relL2 {e_h:.2e}  dW relL2 {e_w:.2e}", flush=True)
    assert e_h <= 1e-4 and e_w <= 1e-4


def test_confident_targets():
    """Peaked rows whose target is the row maximum (p(o) near 1): the target entry
    delta (1 - p(o)) is small and is formed as -delta expm1(l) in float32, so no
    cancellation against a rounded delta p(o) occurs.  W scaled by 2^7 (exact in bf16)
    and every target set to its row's largest logit (float64 oracle logits).  Here the
    other entries carry about half of each row's norm, so their bf16 rounding (2^-9 / sqrt(3)
    relative, RMS) sets the error near 1.2e-3; a split that put delta p(o) in bf16 and
    delta in float32 would cancel to ~2^-9 / (1 - p(o)) per row, past 1e-2 here."""
    wl, _ = _workload("tiny")
    wl, _ = _scaled_w(wl, 7)
    z = ohead.as_f64(wl.hidden_bits) @ ohead.as_f64(wl.w_bits).T
    tgt = np.argmax(z, axis=1).astype(wl.target_full.dtype)
    wl = synth.Workload(**{**wl.__dict__, "target_full": tgt})
    lp = oracle_logp_old(wl)
    cfg = wl.cfg
    out = pipeline.Step(pipeline.upload(wl, lp))(seed=2)
    torch.cuda.synchronize()
    H, pk = oracle_sample_pack(wl, lp, 2)
    ref = oracle_loss(wl, pk)
    assert np.median(ref["logp_new"]) > -0.05     # the regime this test is for: p(o) > 0.95
    assert not ambiguous_clip(ref, cfg.eps_low, cfg.eps_high).any()
    _compare_loss(out, ref)
    e_h = rel_l2(_to_np(out["d_hidden"]), ref["d_hidden"])
    e_w = rel_l2(_to_np(out["d_w_head"]), ref["d_w"])
    print(f"[confident] dH relL2 {e_h:.2e}  dW relL2 {e_w:.2e}", flush=True)
    assert e_h <= 4e-3 and e_w <= 4e-3


def test_nonfinite_flag():
    """A NaN hidden row and an old log-prob of -inf (an infinite ratio) raise
    PSPO_DEVERR_NONFINITE; the clean call raises nothing."""
    wl, lp = _workload("tiny")
    dw = pipeline.upload(wl, lp)
    step = pipeline.Step(dw)
    pk = step.sample_and_pack(seed=0)
    N = int(pk["n_tokens"].item())
    cfg = wl.cfg
    err = torch.zeros(1, dtype=torch.int32, device="cuda")

    def call(hidden, logp_old):
        err.zero_()
        pspo.loss_fwd_bwd(hidden, dw.w_head, pk["target"], logp_old, pk["weight"], pk["seq_id"], dw.advantage, N,
                          cfg.eps_low, cfg.eps_high, cfg.loss_scale, err_flag=err)
        torch.cuda.synchronize()
        return int(err.item())

    assert call(pk["hidden"], pk["logp_old"]) == 0
    h = pk["hidden"].clone()
    h[5] = float("nan")
    assert call(h, pk["logp_old"]) & pspo.DEVERR_NONFINITE
    seq = _to_np(pk["seq_id"][:N])
    i = int(np.nonzero(wl.advantage[seq] != 0)[0][0])      # a token whose loss term is computed
    lo = pk["logp_old"].clone()
    lo[i] = float("-inf")
    assert call(pk["hidden"], lo) == pspo.DEVERR_NONFINITE


# ---------------------------------------------------------------- full size, element-wise


def _chunk_rows(d, V):
    """The backward's vocabulary chunk as the header documents it:
    Vc = 384 * 256 / gcd(ceil(d / 256), 256) rows, or the whole padded vocabulary."""
    import math
    return min(384 * 256 // math.gcd(-(-d // 256), 256), -(-V // 384) * 384)


def _dw_rows(V, Vc, target, k_random=24, seed=19):
    """Rows of d_w_head the full-size test checks: the first and last row of every
    backward chunk of Vc rows, the last row, the ids targeted most often, ids no token
    targets, and random ids."""
    rows = set()
    for v0 in range(0, V, Vc):
        rows.update([v0, min(v0 + Vc, V) - 1])
    rows.add(V - 1)
    ids, cnt = np.unique(target, return_counts=True)
    rows.update(ids[np.argsort(-cnt, kind="stable")[:12]].tolist())
    unused = np.setdiff1d(np.arange(V), ids)
    rng = np.random.default_rng(seed)
    rows.update(rng.choice(unused, min(8, len(unused)), replace=False).tolist())
    rows.update(rng.choice(V, k_random, replace=False).tolist())
    return np.array(sorted(rows))


@pytest.mark.parametrize("name", ["qwen7b", "qwen7b_full", "qwen1.5b", "qwen7b_long"])
def test_full_size(name):
    wl, lp = _workload(name)
    cfg = wl.cfg
    print(f"[{name}] workload ready: {wl.total_tokens} tokens", flush=True)
    dw = pipeline.upload(wl, lp)
    step = pipeline.Step(dw)
    lean = step(seed=0, want_logp=False)    # the benchmark's configuration
    lean = {k: lean[k].clone() for k in ("loss", "d_hidden", "d_w_head", "stats")}
    out = step(seed=0)
    torch.cuda.synchronize()
    print(f"[{name}] GPU pass done, N = {out['N']}", flush=True)
    for k in ("loss", "d_hidden", "d_w_head", "stats"):
        assert torch.equal(lean[k], out[k]), k
    del lean
    H, pk = oracle_sample_pack(wl, lp, 0)
    _check_pack(out, H, pk)
    N = pk["n_tokens"]
    src = pk["src_row"]
    el, eh, scale = f32(cfg.eps_low), f32(cfg.eps_high), f32(cfg.loss_scale)

    # every token's log-prob against the oracle's: the stored old log-probs are the
    # float64 oracle's log-probs plus the workload's noise, rounded to float32
    lp_ref = lp.astype(np.float64)[src] - wl.lp_noise[src]
    lp_gpu = _to_np(out["logp_new"]).astype(np.float64)
    err_lp = np.abs(lp_gpu - lp_ref)
    print(f"[{name}] log-probs: max abs err {err_lp.max():.2e} over {N} tokens", flush=True)
    assert err_lp.max() <= LOGP_ATOL

    # the loss from the oracle's per-token terms
    t = ohead.loss_terms(lp_ref, pk["logp_old"], pk["weight"], pk["seq_id"], wl.advantage, el, eh, scale)
    loss = float(out["loss"].item())
    print(f"[{name}] loss {loss:.9e} oracle {t['loss']:.9e} rel {abs(loss - t['loss']) / abs(t['loss']):.2e}",
          flush=True)
    assert abs(loss - t["loss"]) <= LOSS_RTOL * abs(t["loss"])
    st = _to_np(out["stats"])
    assert st[0] == pytest.approx(t["abs_mass"], rel=LOSS_RTOL)

    # the clip decision of a token whose ratio sits within float32 reach of a bound is the
    # kernel's (taken here in float32 from the GPU's own log-prob); every other token's is
    # the oracle's.  Then delta, and the per-token lse from the oracle's target logits.
    amb = (np.abs(t["rho"] - (1 + eh)) < 1e-5) | (np.abs(t["rho"] - (1 - el)) < 1e-5)
    A = wl.advantage[pk["seq_id"]].astype(np.float64)
    rho32 = np.exp(lp_gpu.astype(np.float32) - pk["logp_old"].astype(np.float32)).astype(np.float64)
    mu32 = ((A > 0) & (rho32 <= np.float32(1 + eh))) | ((A < 0) & (rho32 >= np.float32(1 - el)))
    mu = np.where(amb, mu32, t["mu"] > 0)
    delta = -scale * pk["weight"].astype(np.float64) * mu * t["rho"] * A
    assert int(st[4]) == int(np.sum(delta != 0))
    hid = wl.hidden_bits[src]
    lse = ohead.target_logits(hid, wl.w_bits, pk["target"]) - lp_ref
    print(f"[{name}] {int(amb.sum())} tokens near a clip bound; oracle rows next", flush=True)

    # 64-odd rows of d_w_head (dW product over K = every backward token, chunk edges,
    # the partial last tile) against the oracle row by row
    rows = _dw_rows(cfg.V, _chunk_rows(cfg.d, cfg.V), pk["target"])
    ref_rows = ohead.grad_w_rows(hid, wl.w_bits, pk["target"], lse, delta, rows)
    got_rows = _to_np(out["d_w_head"][torch.from_numpy(rows).cuda()]).astype(np.float64)
    errs = [rel_l2(got_rows[k], ref_rows[k]) for k in range(len(rows))]
    print(f"[{name}] {len(rows)} d_w_head rows: max rel L2 {max(errs):.2e}, "
          f"whole {rel_l2(got_rows, ref_rows):.2e}", flush=True)
    assert max(errs) <= GRAD_REL_L2

    # 48 rows of d_hidden, each against the oracle's full-vocabulary computation
    rng = np.random.default_rng(17)
    idx = np.unique(np.concatenate([[0, N - 1, N - 2], rng.choice(N, 45, replace=False)]))
    sub = {k: pk[k][idx] for k in ("src_row", "seq_id", "weight", "target", "logp_old")}
    ref = oracle_loss(wl, sub)
    dh = _to_np(out["d_hidden"][torch.from_numpy(idx).cuda()]).astype(np.float64)
    for k in range(len(idx)):
        if amb[idx[k]]:
            continue
        if delta[idx[k]] == 0:
            assert not dh[k].any()
        else:
            assert rel_l2(dh[k], ref["d_hidden"][k]) <= GRAD_REL_L2, (k, idx[k])
    print(f"[{name}] sampled d_hidden rows match", flush=True)

    # identities of the gradient at any size: softmax rows sum to one, and
    # <dW, W> = <dH, H> = sum_{i,v} G_iv z_iv
    dW = out["d_w_head"].double()
    col = dW.sum(dim=0)
    assert float(col.norm() / dW.norm()) <= GRAD_REL_L2
    Wd = dw.w_head.double()
    Hd = out["pack"]["hidden"][:N].double()
    a = float((dW * Wd).sum())
    b = float((out["d_hidden"].double() * Hd).sum())
    assert abs(a - b) <= GRAD_REL_L2 * max(abs(a), abs(b))
    print(f"[{name}] identities hold", flush=True)
