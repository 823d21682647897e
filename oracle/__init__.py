"""CPU oracle for the prefix-truncated PPO LM-head path (PS-PPO).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this package: only the tests, the smoke check of the package entry
file and the CPU-baseline leg of the benchmark do.  It shares no code with the
HIP path and imports nothing from it.

It is a plain, slow, float64 implementation written from the paper:

* ``philox``  -- Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11), the
  counter-based generator that draws one cutoff per completion.
* ``cutoffs`` -- quantised survival thresholds, inverse-survival cutoff
  sampling H ~ xi (Sec. 3.2: Pr(H >= t | x) = xi_t; Algorithm 1, sampling of
  one independent cutoff per completion) and prefix packing with the 1/xi_t
  token weights of the truncated estimator (Sec. 3.2 / Sec. 3.3, G-hat).
* ``ppo_head`` -- the LM-head logits z = W h (App. D), the log-softmax, the
  clipped ratio surrogate (Sec. 3.1, PPO objective) weighted by the cutoff
  correction, and its exact gradients with respect to the hidden rows and the
  head (App. D: grad_W log p(o) = (e_o - p) h^T).
* ``cutoff_design`` -- the cutoff design: per-step weights w_t = gbar_t u_t
  from the score proxy and the reward-uncertainty proxy (App. E), the
  budgeted monotone optimum by pooling adjacent violators with the xi <= 1 cap
  (App. F) and the Uniform / Time-prior / Heuristic variants.
* ``score_proxy`` -- the output-head score proxy of the cutoff design,
  gamma = ||h||^2 ||e_o - p||^2 (Sec. 3.3, Eq. gamma_proxy; App. D), from its
  definition.

Parity pins (what fixes each function other than itself) live in the
``-m "not gpu"`` tests: Philox known-answer vectors, the exact counting law of
the sampler, closed forms of the discrete Beta survival, brute-force
enumeration of every cutoff (App. B unbiasedness), float64 autograd of the
plain formula, finite differences, softmax invariants and special cases.
"""
from . import philox, cutoffs, ppo_head  # noqa: F401
