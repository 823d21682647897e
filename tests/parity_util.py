"""Helpers shared by the GPU parity tests: run the oracle on a workload and compare."""
import os

import numpy as np

from oracle import cutoffs as ocut
from oracle import ppo_head as ohead
from paper_2606_29758_amd import synth

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")

# Tolerances for bf16 inputs with fp32 accumulation (the loss is reduced in fp64).
LOSS_RTOL = 1e-4
GRAD_REL_L2 = 1e-2
LOGP_ATOL = 2e-4


def f32(x):
    """The float32 value the kernels see for a scalar parameter, as a float64."""
    return float(np.float32(x))


def oracle_logp_old(wl):
    """logp_old = logp_new + noise with logp_new from the float64 oracle (small workloads)."""
    return (ohead.target_logprob(wl.hidden_bits, wl.w_bits, wl.target_full) + wl.lp_noise).astype(np.float32)


def logp_old_for(wl):
    try:
        return synth.load_stored_logp_old(wl, GOLDEN)
    except FileNotFoundError:
        if wl.total_tokens * wl.cfg.V * wl.cfg.d > 5e12:
            raise
        return oracle_logp_old(wl)


def oracle_sample_pack(wl, logp_old_full, seed, offset=0):
    cfg = wl.cfg
    H = ocut.sample_cutoffs(wl.xi, wl.xi_off, wl.lengths, cfg.P, cfg.K, seed, offset)
    pk = ocut.pack_prefixes(H, wl.lengths, wl.xi, wl.xi_off, cfg.P, cfg.K, wl.target_full, logp_old_full)
    return H, pk


def oracle_loss(wl, pk, advantage=None, want_grads=True):
    cfg = wl.cfg
    adv = wl.advantage if advantage is None else advantage
    return ohead.loss_fwd_bwd(wl.hidden_bits[pk["src_row"]], wl.w_bits, pk["target"], pk["logp_old"],
                              pk["weight"], pk["seq_id"], adv, f32(cfg.eps_low), f32(cfg.eps_high),
                              f32(cfg.loss_scale), want_grads=want_grads)


def rel_l2(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    nb = np.linalg.norm(b)
    return np.linalg.norm(a - b) / nb if nb > 0 else np.linalg.norm(a)


def ambiguous_clip(ref, eps_low, eps_high, band=1e-5):
    """Tokens whose ratio sits so close to a clip bound that float32 and float64 may disagree."""
    rho = ref["rho"]
    return (np.abs(rho - (1 + f32(eps_high))) < band) | (np.abs(rho - (1 - f32(eps_low))) < band)
