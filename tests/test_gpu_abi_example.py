"""GPU: one update pass driven from C++ through the C ABI alone (tests/abi_example.cpp:
hipMalloc'd buffers, a stream of its own, no Python or torch in the process),
checked against the float64 oracle: cutoffs bit-exact, loss, log-probs and
gradients within the parity tolerances, the statistics' counts exact.

The program is built by __graft_entry__.build() (tests/abi_example_build.py)
and runs as a child process of the test.
"""
import os
import subprocess

import numpy as np
import pytest

from oracle import cutoffs as ocut
from oracle import ppo_head as ohead

from parity_util import GRAD_REL_L2, LOGP_ATOL, LOSS_RTOL

pytestmark = pytest.mark.gpu

EXE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "abi_example")


def _rel_l2(a, b):
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


def test_update_pass_from_cpp(tmp_path):
    assert os.path.exists(EXE), "tests/abi_example is not built (run __graft_entry__.build())"
    print(f"[abi_example] running {EXE}", flush=True)
    run = subprocess.run([EXE, str(tmp_path)], capture_output=True, text=True, timeout=120)
    assert run.returncode == 0, (run.stdout + run.stderr)[-2000:]
    print(run.stdout.strip(), flush=True)

    def arr(name, dtype):
        return np.fromfile(os.path.join(tmp_path, name), dtype=dtype)

    P, K, d, V, seed, offset, el, eh, scale, N, flag = open(os.path.join(tmp_path, "meta.txt")).read().split()
    P, K, d, V, N, flag = int(P), int(K), int(d), int(V), int(N), int(flag)
    seed, offset = int(seed), int(offset)
    el, eh, scale = (float(np.float32(float(x))) for x in (el, eh, scale))
    assert flag == 0
    lengths, xi, xi_off = arr("lengths.i32", np.int32), arr("xi.f64", np.float64), arr("xi_off.i64", np.int64)
    adv = arr("adv.f32", np.float32)
    hidden = arr("hidden.bf16", np.uint16).reshape(-1, d)
    w = arr("w.bf16", np.uint16).reshape(V, d)
    target, logp_old = arr("target.i32", np.int32), arr("logp_old.f32", np.float32)

    H = ocut.sample_cutoffs(xi, xi_off, lengths, P, K, seed, offset)
    assert np.array_equal(arr("cutoffs.i32", np.int32), H)
    pk = ocut.pack_prefixes(H, lengths, xi, xi_off, P, K, target, logp_old)
    assert pk["n_tokens"] == N and N > 0
    ref = ohead.loss_fwd_bwd(hidden[pk["src_row"]], w, pk["target"], pk["logp_old"], pk["weight"], pk["seq_id"],
                             adv, el, eh, scale)
    loss = float(arr("loss.f64", np.float64)[0])
    assert abs(loss - ref["loss"]) <= LOSS_RTOL * max(abs(ref["loss"]), ref["abs_mass"] * 1e-3)
    np.testing.assert_allclose(arr("logp.f32", np.float32), ref["logp_new"], rtol=0, atol=LOGP_ATOL)
    assert _rel_l2(arr("dh.f32", np.float32).reshape(N, d), ref["d_hidden"]) <= GRAD_REL_L2
    assert _rel_l2(arr("dw.f32", np.float32).reshape(V, d), ref["d_w"]) <= GRAD_REL_L2
    stats = arr("stats.f64", np.float64)
    A = adv.astype(np.float64)[pk["seq_id"]]
    assert stats[2] == np.count_nonzero(A == 0)                       # zero-advantage tokens
    assert stats[4] == np.count_nonzero(ref["delta"])                  # tokens in the backward
    assert stats[1] == np.count_nonzero((A != 0) & (ref["mu"] == 0))   # clipped tokens
