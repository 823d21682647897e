"""GPU: the per-product timing of the measurement mode (pspo_timing_start /
pspo_timing_stop).

With timing on, every loss call records one forward-product interval and one
logit-gradient, dW and dH interval per vocabulary chunk, and every score-proxy
call one proxy-product interval, all on the call's own stream; the intervals
lie inside the calls (their sum is below the calls' own duration), and the
results are the bits of the same calls without timing.
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


def test_product_timing():
    cfg = synth.custom("timing", "qwen7b", P=2, K=2, length_law=("uniform", 150, 420), data_seed=31)
    wl = synth.make_workload(cfg)
    dw = pipeline.upload(wl, (wl.lp_noise - np.log(cfg.V)).astype(np.float32))
    total = int(wl.total_tokens)
    step = pipeline.Step(dw)
    ref = step(seed=2)
    N = ref["N"]
    ref = {k: ref[k].clone() for k in ("loss", "d_hidden", "d_w_head", "logp_new", "stats")}
    ref_gamma = pspo.score_proxy(dw.hidden_full, dw.w_head, dw.target_full, total)["gamma"].clone()
    pk = step.sample_and_pack(2)
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream()
    calls = 3
    pspo.timing_start(256)
    with pytest.raises(pspo.PspoError, match="already started"):
        pspo.timing_start(8)
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record(stream)
    for _ in range(calls):
        out = step.loss(pk, N)
    gamma = pspo.score_proxy(dw.hidden_full, dw.w_head, dw.target_full, total)["gamma"]
    e.record(stream)
    torch.cuda.synchronize()
    t = pspo.timing_stop()
    wall = s.elapsed_time(e)
    print(f"[timing] N = {N}: {t}, calls {wall:.3f} ms", flush=True)

    assert t["forward"]["count"] == calls and t["proxy"]["count"] == 1
    chunks = t["logit_grad"]["count"] // calls
    assert chunks >= 1 and t["logit_grad"]["count"] == calls * chunks
    assert t["dw"]["count"] == calls * chunks and t["dh"]["count"] == calls * chunks
    assert all(v["ms"] > 0 for v in t.values())
    assert sum(v["ms"] for v in t.values()) < wall
    for k in ref:
        assert torch.equal(out[k], ref[k]), k
    assert torch.equal(gamma, ref_gamma)
    # stopped: a second stop is an error, and calls record nothing
    with pytest.raises(pspo.PspoError, match="not started"):
        pspo.timing_stop()
    pspo.timing_start(4)
    t0 = pspo.timing_stop()
    assert all(v["count"] == 0 and v["ms"] == 0.0 for v in t0.values())
    # a record budget smaller than the products: the first ones are timed, the rest not
    pspo.timing_start(2)
    step.loss(pk, N)
    torch.cuda.synchronize()
    t2 = pspo.timing_stop()
    assert sum(v["count"] for v in t2.values()) == 2
    assert t2["forward"]["count"] == 1 and t2["logit_grad"]["count"] == 1
