"""GPU: the library's calls can be captured in a HIP graph and replayed.

No call allocates, synchronises, or records a memset: their buffers are the
caller's, and the few device words that must start at zero are cleared by
kernels.  The update pass (cutoff sampling, packing, and the loss call at the
packed token count of the draw) and the xi pass (score proxy, design weights,
designed tables) are each captured once and replayed three times, with eager
work of the program and a synchronisation between replays; every replay must
reproduce the eager results bit for bit (all kernels are deterministic).
"""
import numpy as np
import pytest
import torch

from paper_2606_29758_amd import pipeline, pspo, synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    pspo.load()


@pytest.fixture(scope="module")
def batch():
    cfg = synth.custom("graphs", "qwen7b", P=2, K=2, length_law=("uniform", 150, 420), data_seed=21)
    wl = synth.make_workload(cfg)
    # old log-probs near log(1/V) plus the generator's noise (graph against eager, no oracle here)
    logp_old = (wl.lp_noise - np.log(cfg.V)).astype(np.float32)
    return wl, pipeline.upload(wl, logp_old)


def _capture(fn):
    """fn() once eagerly on a side stream (warm-up), then captured; returns (graph, captured outputs)."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        out = fn()
    torch.cuda.synchronize()
    return g, out


def test_update_pass_graph_replays(batch):
    wl, dw = batch
    seed = 7
    ref_out = pipeline.Step(dw)(seed=seed)
    N = ref_out["N"]
    ref = {k: ref_out[k].clone() for k in ("loss", "stats", "cutoffs")}
    ref.update(logp=ref_out["logp_new"].clone(), d_hidden=ref_out["d_hidden"].clone(),
               d_w=ref_out["d_w_head"].clone())
    print(f"[graphs] update pass: N = {N} of {int(wl.total_tokens)} tokens", flush=True)

    step = pipeline.Step(dw)
    step.reserve(N)   # every buffer exists before the capture

    def one_pass():
        pk = step.sample_and_pack(seed)
        out = step.loss(pk, N)
        return pk, out

    g, (pk, out) = _capture(one_pass)
    other = pipeline.Step(dw)
    for rep in range(3):
        # eager work between replays: the captured outputs overwritten, another pass run
        out["d_w_head"].fill_(float("nan"))
        out["d_hidden"].fill_(float("nan"))
        out["loss"].fill_(float("nan"))
        other(seed=100 + rep)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert int(pk["n_tokens"].item()) == N
        got = {"loss": out["loss"], "stats": out["stats"], "cutoffs": step.cutoffs, "logp": out["logp_new"],
               "d_hidden": out["d_hidden"], "d_w": out["d_w_head"]}
        for k in ref:
            assert torch.equal(got[k], ref[k]), (rep, k)
        assert int(step.err.item()) == 0


def test_xi_pass_graph_replays(batch):
    wl, dw = batch
    dev = "cuda"
    total = int(wl.total_tokens)
    T = int(wl.xi_off[-1])
    ids, logp = synth.make_topk(wl)
    ids_t, logp_t = torch.from_numpy(ids).to(dev), torch.from_numpy(logp).to(dev)
    full_off = torch.from_numpy(np.concatenate([[0], np.cumsum(wl.lengths)]).astype(np.int32)).to(dev)
    rewards = torch.from_numpy(wl.rewards.astype(np.float32)).to(dev)
    ws = torch.empty(pspo.score_proxy_workspace_bytes(total, dw.d, dw.V), dtype=torch.uint8, device=dev)

    def xi_pass():
        prox = pspo.score_proxy(dw.hidden_full, dw.w_head, dw.target_full, total, workspace=ws)
        wts = pspo.design_weights(prox["gamma"], ids_t, logp_t, dw.lengths, full_off, rewards, dw.xi_off,
                                  dw.P, dw.K, T)
        xi = pspo.design_cutoffs(wts["w"], dw.xi_off, dw.P, T, 16.0)
        return prox["gamma"], wts["w"], xi

    ref = [t.clone() for t in xi_pass()]
    torch.cuda.synchronize()
    g, outs = _capture(xi_pass)
    for rep in range(3):
        for t in outs:
            t.fill_(float("nan"))
        pipeline.Step(dw)(seed=200 + rep)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k, (got, want) in enumerate(zip(outs, ref)):
            assert torch.equal(got, want), (rep, k)
