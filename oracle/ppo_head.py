"""LM-head + clipped-ratio PPO loss with cutoff weights, and its gradient (float64).

Oracle only (test infrastructure).

Per packed token i (a kept timestep of completion r = seq_id[i]):

* logits z_i = W h_i, no bias (App. D: z_t = W h_t + b, p_t = softmax(z_t));
* log-probability of the sampled token l_i = z_{i,o_i} - logsumexp(z_i)
  (App. D, the first log-sum-exp reduction);
* ratio rho_i = exp(l_i - l_old_i) (Sec. 3.1, the per-timestep importance
  weight pi_theta / pi_old);
* surrogate s_i = min(rho_i A, clip(rho_i, 1 - eps_low, 1 + eps_high) A) with
  the broadcast advantage A of the completion (Sec. 3.1, PPO objective);
* truncated, reweighted objective (Sec. 3.2 / 3.3, G-hat; Algorithm 1 asks to
  reweight token losses by 1/xi_t): J = loss_scale * sum_i c_i s_i with
  c_i = the token weight; the loss is L = -J (gradient descent on -J).

Gradient: dL/dl_i = delta_i = -loss_scale * c_i * mu_i * rho_i * A, where
mu_i = 1 when the unclipped branch is the active one (A > 0 and rho <= 1+eps_high,
or A < 0 and rho >= 1-eps_low; ties pass the gradient), else 0.  Since
d l_i / d z_i = e_{o_i} - p_i (App. D), G_i = delta_i (e_{o_i} - p_i),
dH_i = G_i W (rows of the packed hidden states) and dW = sum_i G_i^T h_i.

The work is done in token chunks; a chunk's logits are held in memory, each
chunk costs three dense products (logits, dH, dW) in float64.
"""
from __future__ import annotations

import numpy as np


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns (uint16) to float64."""
    u = np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def as_f64(x: np.ndarray) -> np.ndarray:
    x = np.asarray(x)
    if x.dtype == np.uint16:
        return bf16_bits_to_f64(x)
    return x.astype(np.float64, copy=False)


def advantages(rewards: np.ndarray, K: int, std_normalise: bool = False, eps: float = 1e-6) -> np.ndarray:
    """Broadcast critic-free advantage A = R - b(x), b = mean reward of the K completions
    of the same prompt (Sec. 3.1).  Optional division by the group's population std."""
    g = np.asarray(rewards, dtype=np.float64).reshape(-1, K)
    a = g - g.mean(axis=1, keepdims=True)
    if std_normalise:
        a = a / (g.std(axis=1, keepdims=True) + eps)
    return a.reshape(-1)


def log_softmax_rows(z: np.ndarray) -> np.ndarray:
    m = z.max(axis=1, keepdims=True)
    return z - (m + np.log(np.exp(z - m).sum(axis=1, keepdims=True)))


def target_logprob(hidden, w, target, chunk: int = 256) -> np.ndarray:
    """log pi(o_t | s_t) for every row of `hidden` under head `w` (float64)."""
    h = as_f64(hidden)
    W = as_f64(w)
    target = np.asarray(target)
    out = np.empty(h.shape[0], dtype=np.float64)
    for s in range(0, h.shape[0], chunk):
        z = h[s:s + chunk] @ W.T
        lp = log_softmax_rows(z)
        out[s:s + chunk] = lp[np.arange(lp.shape[0]), target[s:s + chunk]]
    return out


def loss_fwd_bwd(hidden, w, target, logp_old, weight, seq_id, advantage,
                 eps_low: float, eps_high: float, loss_scale: float,
                 chunk: int = 256, want_grads: bool = True):
    """Returns a dict: loss, d_hidden [N,d], d_w [V,d], logp_new, lse, rho, mu, delta, surrogate."""
    h = as_f64(hidden)
    W = as_f64(w)
    target = np.asarray(target, dtype=np.int64)
    lp_old = np.asarray(logp_old, dtype=np.float64)
    c = np.asarray(weight, dtype=np.float64)
    A = np.asarray(advantage, dtype=np.float64)[np.asarray(seq_id, dtype=np.int64)]
    N = h.shape[0]
    V, d = W.shape

    logp = np.zeros(N)
    lse = np.zeros(N)
    dH = np.zeros((N, d)) if want_grads else None
    dW = np.zeros((V, d)) if want_grads else None
    rho = np.zeros(N)
    mu = np.zeros(N)
    delta = np.zeros(N)
    surr = np.zeros(N)

    for s in range(0, N, chunk):
        e = min(N, s + chunk)
        rows = np.arange(e - s)
        z = h[s:e] @ W.T
        m = z.max(axis=1)
        lse_c = m + np.log(np.exp(z - m[:, None]).sum(axis=1))
        l_c = z[rows, target[s:e]] - lse_c
        r_c = np.exp(l_c - lp_old[s:e])
        a_c = A[s:e]
        clipped = np.clip(r_c, 1.0 - eps_low, 1.0 + eps_high)
        s_c = np.minimum(r_c * a_c, clipped * a_c)
        mu_c = (((a_c > 0) & (r_c <= 1.0 + eps_high)) | ((a_c < 0) & (r_c >= 1.0 - eps_low))).astype(np.float64)
        d_c = -loss_scale * c[s:e] * mu_c * r_c * a_c

        logp[s:e], lse[s:e], rho[s:e], mu[s:e], delta[s:e], surr[s:e] = l_c, lse_c, r_c, mu_c, d_c, s_c
        if want_grads:
            p = np.exp(z - lse_c[:, None])
            G = -p * d_c[:, None]
            G[rows, target[s:e]] += d_c
            dH[s:e] = G @ W
            dW += G.T @ h[s:e]

    loss = -loss_scale * float(np.sum(c * surr))
    return dict(loss=loss, d_hidden=dH, d_w=dW, logp_new=logp, lse=lse, rho=rho, mu=mu,
                delta=delta, surrogate=surr, abs_mass=loss_scale * float(np.sum(np.abs(c * surr))))


def loss_terms(logp, logp_old, weight, seq_id, advantage, eps_low: float, eps_high: float, loss_scale: float):
    """The per-token PPO terms and the loss from given log-probs (the part of
    loss_fwd_bwd after the log-softmax): rho = exp(l - l_old) (Sec. 3.1 ratio),
    s = min(rho A, clip(rho) A) (Sec. 3.1 objective), loss = -loss_scale sum c s
    (Sec. 3.2 / 3.3 reweighted estimator), mu and delta = -loss_scale c mu rho A.
    Lets a caller form the exact loss of a large batch from stored log-probs."""
    l = np.asarray(logp, dtype=np.float64)
    lo = np.asarray(logp_old, dtype=np.float64)
    c = np.asarray(weight, dtype=np.float64)
    A = np.asarray(advantage, dtype=np.float64)[np.asarray(seq_id, dtype=np.int64)]
    rho = np.exp(l - lo)
    s = np.minimum(rho * A, np.clip(rho, 1.0 - eps_low, 1.0 + eps_high) * A)
    mu = (((A > 0) & (rho <= 1.0 + eps_high)) | ((A < 0) & (rho >= 1.0 - eps_low))).astype(np.float64)
    delta = -loss_scale * c * mu * rho * A
    return dict(rho=rho, mu=mu, delta=delta, surrogate=s, loss=-loss_scale * float(np.sum(c * s)),
                abs_mass=loss_scale * float(np.sum(np.abs(c * s))))


def target_logits(hidden, w, target, chunk: int = 4096) -> np.ndarray:
    """z_{i, o_i} = W[o_i] . h_i in float64 (App. D logits at the sampled token)."""
    target = np.asarray(target, dtype=np.int64)
    out = np.empty(len(target))
    for s in range(0, len(target), chunk):
        e = min(len(target), s + chunk)
        out[s:e] = np.einsum("ij,ij->i", as_f64(hidden[s:e]), as_f64(w[target[s:e]]))
    return out


def grad_w_rows(hidden, w, target, lse, delta, rows, chunk: int = 4096) -> np.ndarray:
    """Selected rows of dW = sum_i G_i^T h_i with G_{i,v} = delta_i (1[v = o_i] - exp(z_{i,v} - lse_i))
    (App. D head score times dL/dl_i), given every token's lse and delta: O(N d) per row, so
    rows of a large batch can be checked without its [N, V] logits."""
    rows = np.asarray(rows, dtype=np.int64)
    target = np.asarray(target, dtype=np.int64)
    lse = np.asarray(lse, dtype=np.float64)
    delta = np.asarray(delta, dtype=np.float64)
    Wr = as_f64(np.asarray(w)[rows])                      # [R, d]
    out = np.zeros((len(rows), Wr.shape[1]))
    for s in range(0, len(target), chunk):
        e = min(len(target), s + chunk)
        h = as_f64(hidden[s:e])
        z = h @ Wr.T                                        # [c, R]
        G = -delta[s:e, None] * np.exp(z - lse[s:e, None])
        G += delta[s:e, None] * (target[s:e, None] == rows[None, :])
        out += G.T @ h
    return out
