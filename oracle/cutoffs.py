"""Cutoff sampling and prefix packing, written from PS-PPO Sec. 3.2 and Algorithm 1.

Oracle only (test infrastructure).

Model (Sec. 3.2, "Unbiased Stochastic Truncation"): for prompt p the cutoff H
of each completion is a random variable with survival Pr(H >= t | x) = xi_t,
1 >= xi_1 >= ... >= xi_T > 0.  Algorithm 1 draws one independent cutoff per
completion and keeps tokens t <= H, reweighting each kept token by 1/xi_t
(the truncated estimator G-hat of Sec. 3.2, restated in Sec. 3.3).

Readings fixed here (the paper is silent on them):

* quantisation: the survival table is realised exactly on 32-bit uniforms:
  q_{p,0} = 2^32 and q_{p,t} = max(1, floor(xi_{p,t} * 2^32)).  With x uniform
  on [0, 2^32), Pr(x < q_t) = q_t / 2^32, so the effective survival is q/2^32
  and the weight of a kept token is 2^32 / q_t (float64 division, then
  rounded to float32), which is exactly unbiased for the sampler used;
* inverse-survival draw: H'_r = max{t in [0, T_p] : x_r < q_{p,t}}, then
  H_r = min(T_r, H'_r) -- a completion shorter than its prompt's horizon T_p
  is cut at its own end;
* rollout order r = p*K + k; packed row j of rollout r is timestep t = j+1.
"""
from __future__ import annotations

import numpy as np

from .philox import cutoff_word

TWO32 = 4294967296  # 2^32


def validate_xi(xi: np.ndarray, xi_off: np.ndarray) -> None:
    """Raise ValueError unless every table is in (0, 1] and non-increasing (Sec. 3.2)."""
    xi = np.asarray(xi, dtype=np.float64)
    P = len(xi_off) - 1
    for p in range(P):
        seg = xi[xi_off[p]:xi_off[p + 1]]
        if seg.size == 0:
            continue
        if not np.all(np.isfinite(seg)) or np.any(seg <= 0.0) or np.any(seg > 1.0):
            raise ValueError(f"prompt {p}: xi must lie in (0, 1]")
        if np.any(np.diff(seg) > 0.0):
            raise ValueError(f"prompt {p}: xi must be non-increasing")


def quantise(xi_seg: np.ndarray) -> np.ndarray:
    """Thresholds q_0..q_T as Python ints: q_0 = 2^32, q_t = max(1, floor(xi_t * 2^32)).

    xi_t * 2^32 is exact in float64 (a power-of-two scaling) and so is floor.
    """
    q = [TWO32]
    for v in np.asarray(xi_seg, dtype=np.float64):
        q.append(max(1, int(np.floor(float(v) * float(TWO32)))))
    return q


def token_weight(q: int) -> np.float32:
    """1/xi_t realised as float32(float64(2^32) / float64(q))."""
    return np.float32(np.float64(TWO32) / np.float64(q))


def sample_cutoffs(xi, xi_off, lengths, P: int, K: int, seed: int, offset: int) -> np.ndarray:
    """Cutoffs H_r in [0, T_r], one independent draw per completion."""
    validate_xi(xi, xi_off)
    lengths = np.asarray(lengths)
    H = np.zeros(P * K, dtype=np.int32)
    for p in range(P):
        q = quantise(np.asarray(xi)[xi_off[p]:xi_off[p + 1]])
        for k in range(K):
            r = p * K + k
            x = cutoff_word(r, seed, offset)
            kept = [t for t in range(len(q)) if x < q[t]]   # contains t = 0 always
            H[r] = min(int(lengths[r]), max(kept))
    return H


def pack_prefixes(H, lengths, xi, xi_off, P: int, K: int, target_full=None, logp_old_full=None):
    """Varlen packing of the kept prefixes.

    Returns a dict with cu_seqlens [R+1], full_off [R+1] (offsets of each
    completion in the unpacked token arrays), src_row, seq_id, weight [N], and
    the gathered target / logp_old when given.
    """
    lengths = np.asarray(lengths)
    R = P * K
    # a cutoff never exceeds its completion's length nor its prompt's table horizon
    horizon = np.diff(np.asarray(xi_off))
    H = np.array([max(0, min(int(H[r]), int(lengths[r]), int(horizon[r // K]))) for r in range(R)], dtype=np.int64)
    cu = np.zeros(R + 1, dtype=np.int32)
    full_off = np.zeros(R + 1, dtype=np.int32)
    for r in range(R):
        cu[r + 1] = cu[r] + int(H[r])
        full_off[r + 1] = full_off[r] + int(lengths[r])
    N = int(cu[R])
    src_row = np.zeros(N, dtype=np.int32)
    seq_id = np.zeros(N, dtype=np.int32)
    weight = np.zeros(N, dtype=np.float32)
    for p in range(P):
        q = quantise(np.asarray(xi)[xi_off[p]:xi_off[p + 1]])
        for k in range(K):
            r = p * K + k
            for j in range(int(H[r])):
                i = int(cu[r]) + j
                src_row[i] = full_off[r] + j
                seq_id[i] = r
                weight[i] = token_weight(q[j + 1])
    out = dict(cu_seqlens=cu, full_off=full_off, src_row=src_row, seq_id=seq_id,
               weight=weight, n_tokens=N)
    if target_full is not None:
        out["target"] = np.asarray(target_full)[src_row].astype(np.int32)
    if logp_old_full is not None:
        out["logp_old"] = np.asarray(logp_old_full)[src_row].astype(np.float32)
    return out


def cutoff_pmf(xi_seg, T_r: int) -> np.ndarray:
    """Exact law of H_r = min(T_r, H') under the quantised sampler.

    Pr(H' = h) = (q_h - q_{h+1}) / 2^32 with q_{T_p+1} = 0; the mass of h > T_r
    collapses onto T_r.  Returned as float64 [T_r + 1].
    """
    q = quantise(xi_seg) + [0]
    pmf = np.zeros(T_r + 1, dtype=np.float64)
    for h in range(len(q) - 1):
        pmf[min(h, T_r)] += (q[h] - q[h + 1]) / float(TWO32)
    return pmf
