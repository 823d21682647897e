"""Write the stored old-policy log-probabilities of the large synthetic workloads.

logp_old = logp_new + eps, where logp_new = log softmax(W h_t)[o_t] is computed
by the float64 oracle (and nothing else) over every token of every completion,
and eps is the workload's seeded Gaussian noise.  The result is rounded to
float32, the dtype the loss consumes, and saved as
``logp_old_<workload>.npy`` next to a JSON file holding the workload's
fingerprint, so a consumer can refuse a file that does not match its data.

Usage:  python tests/golden/make_logp_old.py [workload ...]
(minutes of CPU per workload: about 2 V d flops per token in float64)
"""
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle import ppo_head  # noqa: E402
from paper_2606_29758_amd import synth  # noqa: E402

DEFAULT = ["qwen1.5b", "qwen7b", "qwen7b_long"]


def main(names):
    for name in names:
        t0 = time.time()
        wl = synth.make_workload(name)
        lp = ppo_head.target_logprob(wl.hidden_bits, wl.w_bits, wl.target_full, chunk=512)
        logp_old = (lp + wl.lp_noise).astype(np.float32)
        np.save(os.path.join(HERE, f"logp_old_{name}.npy"), logp_old)
        meta = dict(workload=name, fingerprint=wl.fingerprint(), tokens=int(wl.total_tokens),
                    generator="oracle.ppo_head.target_logprob (float64) + synth noise")
        with open(os.path.join(HERE, f"logp_old_{name}.json"), "w") as f:
            json.dump(meta, f, indent=1)
        print(f"{name}: {wl.total_tokens} tokens in {time.time() - t0:.0f}s", flush=True)


if __name__ == "__main__":
    main(sys.argv[1:] or DEFAULT)
