"""bench.py's host-side contract without a GPU: more than one GPU is refused with a
message that says why, and the source digest that gates the committed counters
ignores comments and whitespace but not code."""
import importlib.util
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_more_than_one_gpu_is_refused():
    run = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                         text=True, timeout=120, cwd=ROOT)
    assert run.returncode == 2
    line = json.loads(run.stdout.strip().splitlines()[-1])
    assert "one GPU" in line["error"] and line["n_gpus_requested"] == 2


def test_committed_counters_match_the_sources():
    """The committed counter files name the sources they were taken on; while they match, the
    bench lines carry their memory-side bytes (a mismatch would silently drop them)."""
    b = _bench()
    digest = b.source_hash()
    for name in ("loss_fwd_bwd_qwen7b_traffic.json", "computing_xi_qwen7b_traffic.json"):
        with open(os.path.join(ROOT, "profiles", name)) as f:
            assert json.load(f)["source_hash"] == digest, name
