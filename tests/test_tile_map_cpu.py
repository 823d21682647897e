"""Host build of the product kernel's tile placement (CPU only).

The functions that place tiles on work-groups (the spread row order, whole and
whole-rounds launches, the K-split tail) are host-and-device code in gemm.h;
tile_map_check.cpp compiles them for the host and checks that every tile is
covered exactly once, that each tail tile's K parts partition its K steps, and
that the spread order is a bijection keeping its first tiles in order, and
that the groups dealt to the XCDs keep all eight on the same column tiles.
"""
import os
import shutil
import subprocess

import pytest

from paper_2606_29758_amd import build as pbuild

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="hipcc not available")
def test_tile_placement_host_build(tmp_path):
    exe = str(tmp_path / "tile_map_check")
    cmd = [pbuild.hipcc(), "--offload-arch=gfx950", "-O1", "-std=c++17", "-x", "hip", "-I", pbuild.INCLUDE,
           "-I", pbuild.CSRC, os.path.join(HERE, "tile_map_check.cpp"), "-o", exe]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-2000:]
    run = subprocess.run([exe], capture_output=True, text=True, timeout=300)
    assert run.returncode == 0 and run.stdout.strip() == "ok", run.stdout + run.stderr
