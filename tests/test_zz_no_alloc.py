"""GPU: the no-allocation design entry point against the one that takes a workspace.

pspo_design_cutoffs_noalloc runs the same solve with its block stack in the
library's static device scratch.  Two calls in a row, the second on a smaller
input (fewer prompts and steps, so stale entries of the first call sit in the
scratch), each bitwise equal to pspo_design_cutoffs on the same weights, and
within 1e-12 of the float64 oracle.
"""
import numpy as np
import pytest
import torch

from oracle import cutoff_design as ocd
from paper_2606_29758_amd import pspo

pytestmark = pytest.mark.gpu


def _case(seed, P, T_max):
    rng = np.random.default_rng(seed)
    T = rng.integers(T_max // 2, T_max + 1, P)
    off = np.concatenate([[0], np.cumsum(T)]).astype(np.int64)
    w = rng.gamma(0.6, 1.0, off[-1]) * rng.choice([0.02, 1.0, 30.0], off[-1])
    w[rng.random(off[-1]) < 0.05] = 0.0
    return w, off


@pytest.mark.parametrize("variant", [pspo.PSPO_DESIGN_OPTIMIZED, pspo.PSPO_DESIGN_HEURISTIC])
def test_noalloc_matches_workspace_entry(variant):
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    pspo.load()
    dev = "cuda"
    for seed, P, T_max, budget in ((1, 12, 3000, 96.0), (2, 3, 700, 40.0)):   # the second call is smaller
        w, off = _case(seed, P, T_max)
        total = int(off[-1])
        tw = torch.from_numpy(w).to(dev)
        toff = torch.from_numpy(off).to(dev)
        err = torch.zeros(1, dtype=torch.int32, device=dev)
        ref = pspo.design_cutoffs(tw, toff, P, total, budget, variant=variant, err_flag=err).clone()
        out = torch.full((total,), float("nan"), dtype=torch.float64, device=dev)
        got = pspo.design_cutoffs_noalloc(tw, toff, P, total, budget, out, variant=variant, err_flag=err)
        torch.cuda.synchronize()
        print(f"[noalloc seed {seed}] P={P} total_T={total} variant={variant}", flush=True)
        assert int(err.item()) == 0
        assert torch.equal(got, ref)
        want = ocd.design_tables(w, off, budget, variant)
        np.testing.assert_allclose(got.cpu().numpy(), want, rtol=1e-12, atol=0)
