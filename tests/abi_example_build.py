"""Builds tests/abi_example (a C++ program that runs one update pass through
libpspo's C ABI alone) next to this file, linked against the in-tree library.

    python tests/abi_example_build.py        (also run by __graft_entry__.build())
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
sys.path.insert(0, ROOT)

from paper_2606_29758_amd import build as pbuild  # noqa: E402

EXE = os.path.join(HERE, "abi_example")


def build(verbose: bool = False) -> str:
    lib_dir = os.path.dirname(pbuild.LIB_PATH)
    cmd = [pbuild.hipcc(), "--offload-arch=gfx950", "-O2", "-std=c++17", "-Wall", "-I", pbuild.INCLUDE,
           os.path.join(HERE, "abi_example.cpp"), "-o", EXE + ".tmp", "-L", lib_dir, "-lpspo",
           "-Wl,-rpath,$ORIGIN/" + os.path.relpath(lib_dir, HERE)]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"hipcc failed with exit code {res.returncode}")
    os.replace(EXE + ".tmp", EXE)
    return EXE


if __name__ == "__main__":
    print(build(verbose=True))
