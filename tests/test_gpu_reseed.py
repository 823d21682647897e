"""GPU: the truncated update averaged over 64 cutoff draws against the full-trajectory update.

PS-PPO's estimate (Sec. 3.2; App. B) is linear in the keep indicators, so the
mean of 64 truncated calls (loss, dW, dH rows at their full positions) must
equal one call over every completion token weighted by n_t c_t / 64 (n_t: how
many draws kept token t, c_t its cutoff weight).  That identity is checked to
the parity tolerances, the weighted call against the float64 oracle, and the
counts n_t against the oracle's sampler.  The distance of the 64-draw mean from
the unweighted full update is the estimator's noise; it is printed next to
App. C's diagonal prediction sqrt(sum_t (1/xi_t - 1) ||g_t||^2 / 64) (a report:
the weights 1/xi_t are heavy-tailed, so a 64-draw sample of it is not a gate).
"""
import numpy as np
import pytest
import torch

from oracle import cutoffs as ocut
from paper_2606_29758_amd import pipeline, pspo, synth

from parity_util import GRAD_REL_L2, LOSS_RTOL, f32, logp_old_for, rel_l2
from oracle import ppo_head as ohead

pytestmark = pytest.mark.gpu

SEEDS = list(range(64))
MINI7B = synth.custom("mini7b", "qwen7b", P=2, K=2, length_law=("uniform", 150, 420), data_seed=31)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    pspo.load()


def _run(cfg):
    wl = synth.make_workload(cfg)
    lp = logp_old_for(wl)
    dw = pipeline.upload(wl, lp, device="cuda")
    res = pipeline.reseed_mean(pipeline.Step(dw), SEEDS, want_logp=True)
    torch.cuda.synchronize()
    return wl, lp, dw, res


def _np(t):
    return t.detach().double().cpu().numpy()


def _rel(a, b):
    return float(torch.linalg.vector_norm((a - b).double()) / torch.linalg.vector_norm(b.double()))


def _check_identity(dw, res, name):
    """The S-draw mean against the weighted full call (rounding only), and the mean's
    distance from the plain full update (the estimator's noise; a report)."""
    loss_rel = abs(res["mean_loss"] - res["weighted_loss"]) / abs(res["weighted_loss"])
    dw_rel = _rel(res["mean_dw"], res["weighted_dw"])
    dh_rel = _rel(res["mean_dh"], res["weighted_dh"])
    dev = _rel(res["mean_dw"], res["full_dw"])
    print(f"[{name}] identity: loss rel {loss_rel:.2e}, dW rel L2 {dw_rel:.2e}, dH rel L2 {dh_rel:.2e}; "
          f"64-draw mean vs full update: dW rel dev {dev:.3e}", flush=True)
    assert loss_rel <= LOSS_RTOL
    assert dw_rel <= GRAD_REL_L2
    assert dh_rel <= GRAD_REL_L2
    assert np.isfinite(dev)


def test_reseed_mean_equals_weighted_full_call_tiny():
    wl, lp, dw, res = _run(synth.CONFIGS["tiny"])
    cfg = wl.cfg
    _check_identity(dw, res, "tiny")
    # the keep counts against the oracle's sampler over the same seeds
    n = np.zeros(wl.total_tokens, dtype=np.int64)
    off = np.concatenate([[0], np.cumsum(wl.lengths)])
    for s in SEEDS:
        H = ocut.sample_cutoffs(wl.xi, wl.xi_off, wl.lengths, cfg.P, cfg.K, s, 0)
        for r in range(cfg.P * cfg.K):
            n[off[r]:off[r] + H[r]] += 1
    assert np.array_equal(res["kept"].cpu().numpy(), n)
    # the weighted full call against the float64 oracle
    H_full = wl.lengths.astype(np.int32)
    pk = ocut.pack_prefixes(H_full, wl.lengths, wl.xi, wl.xi_off, cfg.P, cfg.K, wl.target_full, lp)
    w = (pk["weight"].astype(np.float32) * n.astype(np.float32) / np.float32(len(SEEDS))).astype(np.float32)
    ref = ohead.loss_fwd_bwd(wl.hidden_bits[pk["src_row"]], wl.w_bits, pk["target"], pk["logp_old"], w,
                             pk["seq_id"], wl.advantage, f32(cfg.eps_low), f32(cfg.eps_high), f32(cfg.loss_scale))
    assert abs(res["weighted_loss"] - ref["loss"]) <= LOSS_RTOL * abs(ref["loss"])
    assert rel_l2(_np(res["weighted_dw"]), ref["d_w"]) <= GRAD_REL_L2
    assert rel_l2(_np(res["weighted_dh"]), ref["d_hidden"]) <= GRAD_REL_L2


def test_reseed_mean_equals_weighted_full_call_mini7b():
    wl, lp, dw, res = _run(MINI7B)
    _check_identity(dw, res, "mini7b")
