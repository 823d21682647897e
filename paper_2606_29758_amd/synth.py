"""Seeded synthetic workloads for the prefix-truncated PPO LM-head path.

This module only draws random inputs; it holds none of the method's arithmetic
(no sampling of cutoffs, no packing, no softmax, no loss). Both the CPU oracle
and the HIP path consume exactly the arrays produced here.

What is drawn, per workload (stand-ins for the paper's MATH rollouts from a
Qwen2.5-Math-7B-shaped policy, K = 8 completions per prompt, Sec. 4 setup and
the implementation appendix; none of that data is reproduced):

* completion lengths T_r, r = p*K + k (prompt-major);
* a per-prompt survival table xi_{p,t} = Pr(H >= t), t = 1..T_p, with
  T_p = max_k T_{pK+k}.  It is the discrete Beta law of H = ceil(f * T_p),
  f ~ Beta(a, b): xi_{p,t} = Pr(f > (t-1)/T_p) = I_{(T_p-t+1)/T_p}(b, a),
  made non-increasing by a running minimum (the "heuristic cummin" variant of
  Sec. 4's cutoff comparison) and floored at a tiny positive value so that
  every xi_t > 0 as Sec. 3.2 requires.  The full-trajectory control uses
  xi == 1;
* binary rewards R_r and the broadcast critic-free advantage A_r = R_r - mean
  of the group's rewards, optionally divided by the group's std (GRPO-style
  normalisation, one of the paper's baselines) (Sec. 3.1, broadcast advantage with a group-mean
  baseline);
* target token ids o_t, uniform over the vocabulary;
* Gaussian noise eps_t ~ N(0, sigma_lp^2) per token, from which the caller
  forms logp_old = logp_new + eps (logp_new itself is not computed here);
* final hidden states h_t ~ N(0, 1) and an LM head W ~ N(0, 0.02^2), both
  rounded to bf16 (round to nearest even) and returned as raw uint16 bits.

Random streams: numpy PCG64 children of SeedSequence(data_seed), one child per
array, so a consumer may skip the large matrices.
"""
from __future__ import annotations

import dataclasses
import hashlib
import math
from typing import Optional

import numpy as np
from scipy import special

_TINY_XI = 2.0 ** -60  # keeps xi_t > 0; quantises to the smallest threshold


@dataclasses.dataclass(frozen=True)
class SynthConfig:
    name: str
    P: int
    K: int
    d: int
    V: int
    length_law: tuple          # ("uniform", lo, hi) or ("lognormal", median, sigma, lo, hi)
    beta_law: tuple            # ("fixed", a, b) or ("uniform", lo, hi)
    reward_law: tuple          # ("bernoulli", p) or ("bernoulli_prompt_uniform",)
    sigma_lp: float
    data_seed: int
    full_trajectory: bool = False   # xi == 1 (the standard, untruncated update)
    h_std: float = 1.0
    w_std: float = 0.02
    eps_low: float = 0.1
    eps_high: float = 0.1
    # "mean": A = R - group mean (the broadcast critic-free advantage);
    # "std": additionally divided by the group's population std + 1e-6 (GRPO)
    adv_norm: str = "mean"

    @property
    def R(self) -> int:
        return self.P * self.K

    @property
    def loss_scale(self) -> float:
        # (1/K) per prompt as in the full and truncated update directions of
        # Sec. 3.2, averaged over the P prompts of the batch.  It never depends
        # on the sampled cutoffs, which keeps the estimator unbiased.
        return 1.0 / float(self.P * self.K)


# The five workloads the path is measured and tested on.
CONFIGS = {
    "tiny": SynthConfig("tiny", P=2, K=4, d=128, V=2048,
                        length_law=("uniform", 32, 128), beta_law=("fixed", 2.0, 2.0),
                        reward_law=("bernoulli", 0.5), sigma_lp=0.05, data_seed=1),
    "qwen1.5b": SynthConfig("qwen1.5b", P=16, K=8, d=1536, V=151936,
                            length_law=("lognormal", 1024, 0.5, 64, 4096),
                            beta_law=("uniform", 1.0, 4.0),
                            reward_law=("bernoulli_prompt_uniform",), sigma_lp=0.05,
                            data_seed=2),
    "qwen7b": SynthConfig("qwen7b", P=8, K=8, d=3584, V=152064,
                          length_law=("lognormal", 2048, 0.5, 128, 8192),
                          beta_law=("uniform", 1.0, 4.0),
                          reward_law=("bernoulli_prompt_uniform",), sigma_lp=0.1,
                          data_seed=3),
    "qwen7b_long": SynthConfig("qwen7b_long", P=4, K=8, d=3584, V=152064,
                               length_law=("lognormal", 8192, 0.5, 1024, 16384),
                               beta_law=("fixed", 1.5, 4.0),
                               reward_law=("bernoulli_prompt_uniform",), sigma_lp=0.1,
                               data_seed=4),
    # Identical data to "qwen7b" (same data seed), cutoff pinned to the full length.
    "qwen7b_full": SynthConfig("qwen7b_full", P=8, K=8, d=3584, V=152064,
                               length_law=("lognormal", 2048, 0.5, 128, 8192),
                               beta_law=("uniform", 1.0, 4.0),
                               reward_law=("bernoulli_prompt_uniform",), sigma_lp=0.1,
                               data_seed=3, full_trajectory=True),
}


def custom(name: str, base: str, **overrides) -> SynthConfig:
    """A derived workload, e.g. the 7B vocabulary and width with few short rollouts."""
    return dataclasses.replace(CONFIGS[base], name=name, **overrides)


@dataclasses.dataclass
class Workload:
    cfg: SynthConfig
    lengths: np.ndarray        # int32 [R]
    horizon: np.ndarray        # int32 [P]      T_p
    xi: np.ndarray             # float64 [sum T_p]
    xi_off: np.ndarray         # int64 [P+1]
    rewards: np.ndarray        # float64 [R]
    advantage: np.ndarray      # float32 [R]
    target_full: np.ndarray    # int32 [sum T_r]
    lp_noise: np.ndarray       # float64 [sum T_r]
    hidden_bits: Optional[np.ndarray]  # uint16 [sum T_r, d] (bf16 bits)
    w_bits: Optional[np.ndarray]       # uint16 [V, d] (bf16 bits)

    @property
    def total_tokens(self) -> int:
        return int(self.lengths.sum())

    def fingerprint(self) -> str:
        """Digest identifying the token data (not the cutoff tables) a stored file belongs to."""
        h = hashlib.sha256()
        h.update(np.array([self.cfg.d, self.cfg.V, self.cfg.data_seed], dtype=np.int64).tobytes())
        for a in (self.lengths, self.target_full, self.lp_noise):
            h.update(np.ascontiguousarray(a).tobytes())
        return h.hexdigest()[:16]


def load_stored_logp_old(wl: "Workload", directory: str) -> np.ndarray:
    """Old-policy log-probs stored for this workload's token data (float32 [sum T_r]).

    Looks for ``logp_old_*.json`` in `directory` whose fingerprint matches, and raises
    if none does (the stored file was made from different data).
    """
    import glob
    import json
    import os

    fp = wl.fingerprint()
    for meta_path in sorted(glob.glob(os.path.join(directory, "logp_old_*.json"))):
        with open(meta_path) as f:
            meta = json.load(f)
        if meta.get("fingerprint") == fp:
            arr = np.load(meta_path[:-5] + ".npy", allow_pickle=False)
            if arr.shape != (wl.total_tokens,) or arr.dtype != np.float32:
                raise ValueError(f"{meta_path}: stored array does not match the workload's shape")
            return arr
    raise FileNotFoundError(f"no stored old log-probs for workload {wl.cfg.name} (fingerprint {fp}) in {directory}")


def round_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit pattern, round to nearest, ties to even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    return ((u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)


def _normal_bf16(rng: np.random.Generator, shape, std: float, block_rows: int = 8192) -> np.ndarray:
    rows, cols = shape
    out = np.empty(shape, dtype=np.uint16)
    for r0 in range(0, rows, block_rows):
        r1 = min(rows, r0 + block_rows)
        blk = rng.standard_normal((r1 - r0, cols), dtype=np.float32)
        if std != 1.0:
            blk *= np.float32(std)
        out[r0:r1] = round_to_bf16_bits(blk)
    return out


def beta_survival_table(a: float, b: float, T: int) -> np.ndarray:
    """xi_t = Pr(ceil(f*T) >= t) for f ~ Beta(a, b), t = 1..T (float64, non-increasing, > 0).

    Uses the symmetric form I_{(T-t+1)/T}(b, a) of the survival function, which avoids
    the cancellation of 1 - I near t = T.
    """
    t = np.arange(1, T + 1, dtype=np.float64)
    y = (T - t + 1.0) / T
    xi = special.betainc(b, a, y)
    xi = np.minimum.accumulate(np.clip(xi, 0.0, 1.0))
    return np.maximum(xi, _TINY_XI)


def make_workload(cfg, with_matrices: bool = True) -> Workload:
    if isinstance(cfg, str):
        cfg = CONFIGS[cfg]
    P, K, R = cfg.P, cfg.K, cfg.R
    kids = np.random.SeedSequence(cfg.data_seed).spawn(8)
    g_len, g_beta, g_rew, g_tgt, g_noise, g_h, g_w, _ = [np.random.Generator(np.random.PCG64(s)) for s in kids]

    law = cfg.length_law
    if law[0] == "uniform":
        lengths = g_len.integers(law[1], law[2] + 1, size=R)
    elif law[0] == "lognormal":
        _, median, sigma, lo, hi = law
        raw = np.exp(math.log(median) + sigma * g_len.standard_normal(R))
        lengths = np.clip(np.rint(raw), lo, hi)
    else:
        raise ValueError(law)
    lengths = lengths.astype(np.int32)
    horizon = lengths.reshape(P, K).max(axis=1).astype(np.int32)

    bl = cfg.beta_law
    if bl[0] == "fixed":
        ab = np.tile(np.array([bl[1], bl[2]], dtype=np.float64), (P, 1))
    elif bl[0] == "uniform":
        ab = g_beta.uniform(bl[1], bl[2], size=(P, 2))
    else:
        raise ValueError(bl)

    xi_off = np.zeros(P + 1, dtype=np.int64)
    xi_off[1:] = np.cumsum(horizon.astype(np.int64))
    xi = np.empty(int(xi_off[-1]), dtype=np.float64)
    for p in range(P):
        Tp = int(horizon[p])
        if cfg.full_trajectory:
            xi[xi_off[p]:xi_off[p + 1]] = 1.0
        else:
            xi[xi_off[p]:xi_off[p + 1]] = beta_survival_table(ab[p, 0], ab[p, 1], Tp)

    rl = cfg.reward_law
    if rl[0] == "bernoulli":
        rewards = (g_rew.random(R) < rl[1]).astype(np.float64)
    elif rl[0] == "bernoulli_prompt_uniform":
        p_prompt = g_rew.random(P)
        rewards = (g_rew.random((P, K)) < p_prompt[:, None]).astype(np.float64).reshape(R)
    else:
        raise ValueError(rl)
    grp = rewards.reshape(P, K)
    centred = grp - grp.mean(axis=1, keepdims=True)
    if cfg.adv_norm == "std":
        centred = centred / (grp.std(axis=1, keepdims=True) + 1e-6)
    elif cfg.adv_norm != "mean":
        raise ValueError(cfg.adv_norm)
    advantage = centred.reshape(R).astype(np.float32)

    S = int(lengths.sum())
    target_full = g_tgt.integers(0, cfg.V, size=S).astype(np.int32)
    lp_noise = cfg.sigma_lp * g_noise.standard_normal(S)

    hidden_bits = w_bits = None
    if with_matrices:
        hidden_bits = _normal_bf16(g_h, (S, cfg.d), cfg.h_std)
        w_bits = _normal_bf16(g_w, (cfg.V, cfg.d), cfg.w_std)

    return Workload(cfg=cfg, lengths=lengths, horizon=horizon, xi=xi, xi_off=xi_off,
                    rewards=rewards, advantage=advantage, target_full=target_full,
                    lp_noise=lp_noise, hidden_bits=hidden_bits, w_bits=w_bits)


def make_topk(wl: "Workload", k: int = 16, pool: int = 64, seed: int = 0):
    """Synthetic top-k next-token lists of every completion token, in the shape a
    rollout engine reports them: k distinct token ids per row, log-probs sorted in
    decreasing order, with total mass below one.  The ids of one prompt's rows are
    drawn from a pool of `pool` ids so that the lists of different completions
    overlap.  Returns (ids int32 [S, k], logp float32 [S, k])."""
    cfg = wl.cfg
    rng = np.random.default_rng(np.random.SeedSequence([cfg.data_seed, 7919, seed]))
    S = int(wl.total_tokens)
    ids = np.empty((S, k), dtype=np.int32)
    pools = [rng.choice(cfg.V, size=pool, replace=False) for _ in range(cfg.P)]
    off = 0
    for r, T in enumerate(wl.lengths):
        p = r // cfg.K
        for j in range(int(T)):
            ids[off + j] = pools[p][rng.permutation(pool)[:k]]
        off += int(T)
    mass = rng.uniform(0.5, 0.95, S)
    probs = -np.sort(-rng.dirichlet(np.full(k, 0.3), S), axis=1) * mass[:, None]
    probs = np.maximum(probs, 1e-30)
    return ids, np.log(probs).astype(np.float32)
