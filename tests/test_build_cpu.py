"""Compile-time guard for the matrix-core kernels (CPU only: hipcc cross-compiles for gfx950).

Every product's accumulators are updated by inline-asm MFMAs with the accumulator
tied in place, and the compiler does not know their latency.  Spill code or a
private-memory copy of an accumulator placed right after its last MFMA would read
the value before the MFMA has written it (such copies, produced by an epilogue
that indexed the accumulators in a loop the compiler did not unroll, lost the
last K step of the first block after a barrier in a harness).  So every
instantiation of the product kernel must use no scratch memory and spill no
VGPRs.
"""
import os
import re
import shutil
import subprocess

import pytest

from paper_2606_29758_amd import build as pbuild

SOURCES = ["loss.hip", "proxy.hip"]


def _remarks(src):
    cmd = [pbuild.hipcc(), *[f for f in pbuild.HIPCC_FLAGS if f != "-shared"], "-c",
           "-I", pbuild.INCLUDE, "-I", pbuild.CSRC, os.path.join(pbuild.CSRC, src),
           "-o", os.devnull, "-Rpass-analysis=kernel-resource-usage"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-2000:]
    kernels, cur = {}, None
    for line in res.stderr.splitlines():
        m = re.search(r"remark: Function Name: (\S+)", line)
        if m:
            cur = kernels.setdefault(m.group(1), {})
            continue
        m = re.search(r"remark:\s+([A-Za-z ]+?)(?: \[bytes/lane\])?: (\d+)", line)
        if m and cur is not None:
            cur[m.group(1).strip()] = int(m.group(2))
    return kernels


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="hipcc not available")
@pytest.mark.parametrize("src", SOURCES)
def test_products_use_no_scratch(src):
    kernels = _remarks(src)
    gemm = {k: v for k, v in kernels.items() if "gemm_nt_kernel" in k}
    assert gemm, f"no product kernel found in {src}"
    for name, r in gemm.items():
        assert r.get("ScratchSize") == 0, (name, r)
        assert r.get("VGPRs Spill") == 0, (name, r)
        assert r.get("AGPRs") == 256, (name, r)   # the accumulators fill the AGPR file
