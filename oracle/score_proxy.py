"""Output-head score proxy of the cutoff design, in float64 (test infrastructure only).

For a completion token with last-layer hidden state h, logits z = W h (no bias,
as for the Qwen head), p = softmax(z) and the token actually generated o, the
squared Frobenius norm of the output-head score is (App. D, output-head score
proxy)

    gamma = || grad_W log p(o) ||_F^2 = ||h||^2 * ||e_o - p||^2,

which the paper uses as a forward-only stand-in for the full score norm in the
cutoff weights (Sec. 3.3, Eq. gamma_proxy).  This module computes it from that
definition: the squared distance between the one-hot target and the softmax,
summed over the vocabulary.  The paper's cheaper route through two log-sum-exp
reductions (1 - 2 p(o) + exp(l2 - 2 l1)) is what the GPU path does; here it is
only a test of the definition, not the computation.

Only tests/, the package's smoke check and the benchmark's CPU baseline use this.
"""
import numpy as np

from .ppo_head import as_f64, log_softmax_rows


def score_proxy(hidden, w, target, chunk: int = 256) -> dict:
    """gamma, log p(o) and ||p||^2 for every row of `hidden` (bf16 bits or floats) under
    head `w`; `target` holds the generated token of each row."""
    h = as_f64(hidden)
    W = as_f64(w)
    target = np.asarray(target, dtype=np.int64)
    n = h.shape[0]
    gamma = np.empty(n)
    logp = np.empty(n)
    psq = np.empty(n)
    for s in range(0, n, chunk):
        hs = h[s:s + chunk]
        lp = log_softmax_rows(hs @ W.T)
        p = np.exp(lp)
        rows = np.arange(hs.shape[0])
        o = target[s:s + chunk]
        diff = -p
        diff[rows, o] += 1.0                       # e_o - p
        gamma[s:s + chunk] = (hs * hs).sum(axis=1) * (diff * diff).sum(axis=1)
        logp[s:s + chunk] = lp[rows, o]
        psq[s:s + chunk] = (p * p).sum(axis=1)
    return dict(gamma=gamma, logp=logp, p_sq=psq)
