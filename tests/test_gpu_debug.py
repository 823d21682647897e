"""GPU: the PSPO_DEBUG mode (a synchronisation and error check after every
kernel launch) changes no result.

Every call of the library runs once normally and once with PSPO_DEBUG=1 on the
same inputs: the sampled cutoffs, the packing, the loss, log-probs, gradients
and statistics, the score proxy and the designed tables must agree bit for
bit, and no call may report an error.
"""
import os

import numpy as np
import pytest
import torch

from paper_2606_29758_amd import pipeline, pspo, synth

from parity_util import logp_old_for

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    pspo.load()


def _pass(dw, wl, debug):
    if debug:
        os.environ["PSPO_DEBUG"] = "1"
    try:
        out = pipeline.Step(dw)(seed=5)
        N = out["N"]
        res = {"cutoffs": out["cutoffs"].clone(), "loss": out["loss"].clone(), "stats": out["stats"].clone(),
               "logp": out["logp_new"].clone(), "d_hidden": out["d_hidden"].clone(),
               "d_w": out["d_w_head"].clone()}
        res["pack_cu_seqlens"] = out["pack"]["cu_seqlens"].clone()
        for k in ("src_row", "seq_id", "weight", "target", "logp_old", "hidden"):   # rows past N are not written
            res["pack_" + k] = out["pack"][k][:N].clone()
        total = int(wl.total_tokens)
        prox = pspo.score_proxy(dw.hidden_full, dw.w_head, dw.target_full, total, want_p_sq=True)
        res.update(gamma=prox["gamma"].clone(), proxy_logp=prox["logp"].clone(), p_sq=prox["p_sq"].clone())
        ids, logp = synth.make_topk(wl)
        dev = "cuda"
        full_off = torch.from_numpy(np.concatenate([[0], np.cumsum(wl.lengths)]).astype(np.int32)).to(dev)
        T = int(wl.xi_off[-1])
        wts = pspo.design_weights(prox["gamma"], torch.from_numpy(ids).to(dev), torch.from_numpy(logp).to(dev),
                                  dw.lengths, full_off, torch.from_numpy(wl.rewards.astype(np.float32)).to(dev),
                                  dw.xi_off, dw.P, dw.K, T)
        res["xi"] = pspo.design_cutoffs(wts["w"], dw.xi_off, dw.P, T, 16.0).clone()
        torch.cuda.synchronize()
        return N, res
    finally:
        os.environ.pop("PSPO_DEBUG", None)


@pytest.mark.parametrize("name", ["tiny", "mini7b"])
def test_debug_mode_same_bits(name):
    cfg = "tiny" if name == "tiny" else synth.custom("mini7b_dbg", "qwen7b", P=2, K=2,
                                                      length_law=("uniform", 150, 420), data_seed=7)
    wl = synth.make_workload(cfg)
    dw = pipeline.upload(wl, logp_old_for(wl), device="cuda")
    n0, a = _pass(dw, wl, debug=False)
    n1, b = _pass(dw, wl, debug=True)
    assert n0 == n1 and n0 > 0
    for k in a:
        assert torch.equal(a[k], b[k]), k
