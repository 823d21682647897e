"""The host code of libpspo under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

tests/abi_sanitize.cpp drives every argument check of the C ABI, the host
validation of survival tables and the workspace queries at extreme sizes; it is
linked with the library's sources, the sanitizers applied to the host code only
(the device code is built as usual).  No call reaches a kernel launch.
"""
import os
import shutil
import subprocess

import pytest

from paper_2606_29758_amd import build as pbuild

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="hipcc not available")
def test_host_code_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "abi_sanitize")
    flags = [f for f in pbuild.HIPCC_FLAGS if f not in ("-shared", "-fPIC", "-O3")]
    san = ["-O1", "-g", "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
    srcs = [os.path.join(pbuild.CSRC, s) for s in pbuild.SOURCES] + [os.path.join(HERE, "abi_sanitize.cpp")]
    cmd = [pbuild.hipcc(), *flags, *san, "-I", pbuild.INCLUDE, "-I", pbuild.CSRC, *srcs, "-o", exe, *pbuild.LINK_FLAGS]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-3000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1", HIP_VISIBLE_DEVICES="")
    run = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    assert run.returncode == 0, (run.stdout + run.stderr)[-3000:]
    assert "abi_sanitize: ok" in run.stdout
    assert "runtime error" not in run.stderr and "AddressSanitizer" not in run.stderr
