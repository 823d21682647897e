"""Cutoff design of PS-PPO in float64 (test infrastructure only).

Per prompt x with K completions of lengths T_k (T = max_k T_k), Sec. 3.3 and
Algorithm 1 ("Computing xi") build timestep weights w_t = gbar_t * u_t from

* the output-head score proxy gamma of every completion token (App. D),
  averaged over the completions that reach step t:  gbar_t;
* the reward-uncertainty proxy (App. E)
      u_t = 1/2 - 1/2 || p pibar_G(.|t) - (1 - p) pibar_B(.|t) ||_1,
  estimated from the completions alive at t: with n_t of them, G_t / B_t the
  successful / unsuccessful ones and pi_k(.|t) completion k's next-token
  distribution at t,  p pibar_G - (1-p) pibar_B = (1/n_t)(sum_{G_t} pi_k - sum_{B_t} pi_k).
  Each pi_k is known through its top-k entries (the rollout engine's top-k
  log-probs); the mass outside them is one further coordinate "rest", shared by
  all completions.

and then solve (Eq. design_problem; App. F)

      min_xi  sum_t w_t / xi_t   s.t.  sum_t xi_t = B,  1 >= xi_1 >= ... >= xi_T > 0.

App. F: without monotonicity the optimum is xi_t = B sqrt(w_t) / sum_j sqrt(w_j);
under monotonicity it is blockwise constant, xi_m = B s_m / sum_j L_j s_j with
s_m = sqrt(W_m / L_m) over contiguous blocks (W_m = summed weight, L_m =
length), and Pooling Adjacent Violators merges neighbouring blocks until the
scores are non-increasing.  The cap xi <= 1 saturates a prefix (App. F's
remark); here the capped optimum is min(1, kappa s_m) with kappa fixed by the
budget.  Variants of the paper's ablation: Uniform (H uniform on 1..T), Time
prior (xi_t = exp(-lambda (t - 1))) and Heuristic (the unconstrained closed
form, capped at 1, made non-increasing by a running minimum).

Every xi is floored at 2^-32, the resolution of the sampler's thresholds.
"""
import math

import numpy as np

XI_FLOOR = 2.0 ** -32
OPTIMIZED, HEURISTIC, UNIFORM, TIME_PRIOR = 0, 1, 2, 3


def proxy_weights(gamma, topk_ids, topk_logp, lengths, rewards, P: int, K: int) -> dict:
    """Per prompt p and step t = 1..T_p: gbar_t, u_t and w_t = gbar_t u_t, concatenated over
    prompts (the layout of the xi tables).  gamma [S], topk_ids/topk_logp [S, k] over the
    completion tokens laid out completion after completion; rewards [P K], success = R > 1/2."""
    lengths = np.asarray(lengths, dtype=np.int64)
    off = np.concatenate([[0], np.cumsum(lengths)])
    gamma = np.asarray(gamma, dtype=np.float64)
    probs = np.exp(np.asarray(topk_logp, dtype=np.float64))
    ids = np.asarray(topk_ids)
    gbar, u = [], []
    for p in range(P):
        rows = range(p * K, (p + 1) * K)
        Tp = int(max(lengths[r] for r in rows))
        for t in range(1, Tp + 1):
            alive = [r for r in rows if lengths[r] >= t]
            n = len(alive)
            gbar.append(sum(gamma[off[r] + t - 1] for r in alive) / n)
            diff = {}
            rest = 0.0
            for r in alive:
                sign = 1.0 if rewards[r] > 0.5 else -1.0
                row = off[r] + t - 1
                mass = 0.0
                for v, pr in zip(ids[row], probs[row]):
                    diff[int(v)] = diff.get(int(v), 0.0) + sign * pr
                    mass += pr
                rest += sign * max(0.0, 1.0 - mass)
            l1 = sum(abs(x) for x in diff.values()) + abs(rest)
            n_succ = sum(1 for r in alive if rewards[r] > 0.5)
            if n_succ == 0 or n_succ == n:
                # equal rewards among the alive completions: p is 0 or 1 and the norm is
                # exactly 1, so u = 0 (taken exactly, not through rounding)
                u.append(0.0)
            else:
                # the norm is at most 1 (triangle inequality), so u >= 0: clamp rounding below it
                u.append(max(0.0, 0.5 - 0.5 * l1 / n))
    gbar = np.array(gbar)
    u = np.array(u)
    return dict(gbar=gbar, u=u, w=gbar * u)


def pav_blocks(w):
    """Pooling Adjacent Violators: contiguous blocks (start, length, W) whose scores
    sqrt(W / L) are non-increasing (App. F)."""
    stack = []   # [start, L, W]
    for t, wt in enumerate(np.asarray(w, dtype=np.float64)):
        blk = [t, 1, float(wt)]
        while stack and math.sqrt(stack[-1][2] / stack[-1][1]) < math.sqrt(blk[2] / blk[1]):
            prev = stack.pop()
            blk = [prev[0], prev[1] + blk[1], prev[2] + blk[2]]
        stack.append(blk)
    return stack


def design_xi(w, budget: float, variant: int = OPTIMIZED, lam: float = 0.0) -> np.ndarray:
    """The survival table xi_1..xi_T of one prompt."""
    w = np.asarray(w, dtype=np.float64)
    T = len(w)
    t = np.arange(T, dtype=np.float64)
    if variant == UNIFORM:
        return (T - t) / T
    if variant == TIME_PRIOR:
        return np.maximum(np.exp(-lam * t), XI_FLOOR)
    if budget >= T:
        return np.ones(T)
    root = np.sqrt(w)
    if root.sum() == 0.0:                      # every weight zero: any feasible table is optimal
        return np.full(T, budget / T)
    if variant == HEURISTIC:
        xi = np.minimum(1.0, budget * root / root.sum())
        xi = np.minimum.accumulate(xi)
        return np.maximum(xi, XI_FLOOR)
    blocks = pav_blocks(w)
    score = [math.sqrt(W / L) for _, L, W in blocks]
    # rest[m] = sum_{j >= m} L_j s_j, accumulated from the last block
    rest = [0.0] * len(blocks)
    acc = 0.0
    for m in range(len(blocks) - 1, -1, -1):
        acc += blocks[m][1] * score[m]
        rest[m] = acc
    xi = np.empty(T)
    saturated = 0
    for m in range(len(blocks)):
        if rest[m] == 0.0:                      # only zero-weight blocks left
            kappa = None
            break
        kappa = (budget - saturated) / rest[m]
        if kappa * score[m] <= 1.0:
            break
        saturated += blocks[m][1]
    for (start, L, _), s in zip(blocks, score):
        if kappa is None:
            val = 1.0 if start < saturated else (budget - saturated) / (T - saturated)
        else:
            val = min(1.0, kappa * s)
        xi[start:start + L] = val
    return np.maximum(xi, XI_FLOOR)


def design_tables(w, xi_off, budget: float, variant: int = OPTIMIZED, lam: float = 0.0) -> np.ndarray:
    """design_xi for every prompt; w and the result use the xi_off layout."""
    xi_off = np.asarray(xi_off, dtype=np.int64)
    out = np.empty(xi_off[-1])
    for p in range(len(xi_off) - 1):
        a, b = xi_off[p], xi_off[p + 1]
        out[a:b] = design_xi(w[a:b], budget, variant, lam)
    return out
