"""Benchmark of the PS-PPO hot path on one MI355X: prefix tokens/s of one update pass.

A step is one pass of the whole hot path over one batch of synthetic rollouts
already resident in HBM: Philox cutoff sampling, prefix packing (with the
hidden-row gather), the 4-byte read of the packed token count, and the fused
LM-head + prefix-weighted PPO loss forward and backward (loss, dHidden, dW;
per-token log-probs are not requested, so the forward skips the tokens of
zero-advantage completions, whose loss terms and gradients are exactly zero).

Workload: the 7B-shaped batch (Qwen2.5-Math-7B head dims d = 3584,
V = 152064; 8 prompts x 8 rollouts; lengths lognormal around 2048, clipped
to [128, 8192]; per-prompt discrete Beta(a, b) cutoff laws, a, b ~ U[1, 4];
old log-probs = new + N(0, 0.1^2)).

Prints one JSON line.  `roofline` is that of the dominant kernel, the forward
logit product (one launch per call, about a quarter of a step): achieved = its
algorithmic flops per launch, 2 n_fwd V d, / its mean duration, timed live
over the timed steps with HIP events that the library records on the call's
own stream around each of its matrix-core products (pspo_timing_start; the
rocprofv3 kernel trace of the same command gives the same average).  n_fwd
counts the tokens of completions with a nonzero advantage (the only ones whose
loss term can be nonzero).  `products` gives the same for each product of the
call (the logit-gradient recompute, dW and dH per vocabulary chunk, with their
K-split tails), and `loss_call` the whole call: (2 n_fwd + 4 n_bwd) V d needed
flops / mean call duration, n_bwd counting the tokens whose logit gradient is
not identically zero (the others add nothing to dH or dW; the kernels skip
them); `pct_bf16_peak` is that whole-call figure.
`dense_equivalent_tflops` is 6 N V d / duration, the rate a path that ran the
gradient products over every token would need for the same throughput.
`full_trajectory_control` times the untruncated update on the same batch, and
`reseed_check` (after the timed steps) averages the truncated update over 64
cutoff draws: that mean must equal one weighted full-trajectory call (the
estimator is linear in the keep indicators), and its distance from the plain
full update is reported next to the paper's diagonal variance prediction.
The headline path stores no logit at all (the backward recomputes every logit
tile).  `keep_logits_control` times the same loss calls with the opt-in
PSPO_KEEP_LOGITS (the forward keeps the first vocabulary chunk's logits as
fp16 offsets and the backward converts them instead of recomputing that
chunk: less matrix-core work for Vc x N x 2 bytes of workspace), and `mfma_loop_peak` is the
matrix cores' sustained bf16 rate on the products' MFMA form with no memory
traffic (the ceiling at the clock the chip holds, next to the published peak).
`cpu_baseline` times the float64 CPU oracle on a bounded sample of the same step
(all cutoffs and packing, then the loss of the first --cpu-tokens packed
tokens), with the BLAS library it ran on and a single-thread rate on a
sixteenth of that sample.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6     # MI355X dense bf16 MFMA (256 CUs x 2.4 GHz x 4096 flop/clk)
GOLDEN = os.path.join(ROOT, "tests", "golden")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "loss_fwd_bwd_qwen7b_traffic.json")
XI_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "computing_xi_qwen7b_traffic.json")


def source_hash():
    """Digest of the HIP/C++ sources of libpspo with comments and whitespace removed
    (identifies the kernels counters were taken on; a comment edit changes no kernel)."""
    import hashlib
    import re
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2606_29758_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, name), encoding="utf-8") as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(name.encode() + " ".join(text.split()).encode())
    return h.hexdigest()[:16]


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="qwen7b")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cpu-tokens", type=int, default=4096)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-full-control", action="store_true",
                    help="skip the full-trajectory control on the same batch: its timing (every xi = 1) "
                         "and the reseed check")
    ap.add_argument("--no-keep-control", action="store_true",
                    help="skip the timing of the same calls with PSPO_KEEP_LOGITS (profiling runs)")
    ap.add_argument("--no-mfma-peak", action="store_true",
                    help="skip the matrix-core rate probe (profiling runs)")
    ap.add_argument("--reseeds", type=int, default=64,
                    help="cutoff draws averaged by the reseed check (after the timed steps; 0 skips it): "
                         "their mean update against the full-trajectory one")
    ap.add_argument("--pass", dest="which", choices=["update", "xi"], default="update",
                    help="update: the policy-update hot path (default); xi: computing the cutoff "
                         "tables (score proxy over every completion token + cutoff design)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a device copy of known size (HBM counter calibration) and exit")
    return ap.parse_args()


def copy_calibration():
    import torch
    n = 1 << 30   # 1 GiB read + 1 GiB written per copy
    a = torch.ones(n, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": n, "launches": 3}), flush=True)


def cpu_baseline(wl, logp_old, ntok, seed):
    """The oracle as it stands: sampling + packing of the whole batch, then the loss and
    gradients of the first `ntok` packed tokens.  Returns the object for the JSON line."""
    from threadpoolctl import threadpool_info
    from oracle import cutoffs as ocut
    from oracle import ppo_head as ohead

    cfg = wl.cfg
    t0 = time.perf_counter()
    H = ocut.sample_cutoffs(wl.xi, wl.xi_off, wl.lengths, cfg.P, cfg.K, seed, 0)
    pk = ocut.pack_prefixes(H, wl.lengths, wl.xi, wl.xi_off, cfg.P, cfg.K, wl.target_full, logp_old)
    sel = slice(0, min(ntok, pk["n_tokens"]))
    src = pk["src_row"][sel]
    ohead.loss_fwd_bwd(wl.hidden_bits[src], wl.w_bits, pk["target"][sel], pk["logp_old"][sel],
                       pk["weight"][sel], pk["seq_id"][sel], wl.advantage, float(np.float32(cfg.eps_low)),
                       float(np.float32(cfg.eps_high)), float(np.float32(cfg.loss_scale)))
    dt = time.perf_counter() - t0
    n = sel.stop
    blas = [p for p in threadpool_info() if p.get("user_api") == "blas"]
    threads = max([p.get("num_threads", 1) for p in blas] or [1])
    # the same loss on one BLAS thread, on a smaller sample of the same tokens
    from threadpoolctl import threadpool_limits
    n1 = min(ntok // 16, n)
    with threadpool_limits(limits=1, user_api="blas"):
        t1 = time.perf_counter()
        s1 = slice(0, n1)
        ohead.loss_fwd_bwd(wl.hidden_bits[src[s1]], wl.w_bits, pk["target"][s1], pk["logp_old"][s1],
                           pk["weight"][s1], pk["seq_id"][s1], wl.advantage, float(np.float32(cfg.eps_low)),
                           float(np.float32(cfg.eps_high)), float(np.float32(cfg.loss_scale)))
        dt1 = time.perf_counter() - t1
    return {"value": n / dt, "unit": "prefix tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"cutoffs and packing of all {cfg.R} rollouts, then loss + gradients of the first "
                      f"{n} packed tokens (float64 numpy, {dt:.1f} s)",
            "blas": ", ".join(f"{p.get('internal_api')} {p.get('version')}" for p in blas) or "unknown",
            "single_core": {"value": n1 / dt1, "unit": "prefix tokens/s",
                            "sample": f"loss + gradients of the first {n1} packed tokens on one BLAS thread "
                                      f"({dt1:.1f} s)"}}


def reseed_summary(dw, res):
    """Scalars of a pipeline.reseed_mean result (a report of the benchmark, not a step of the path).

    identity: how far the S-draw mean is from the weighted full call (rounding only):
    loss relative error, dW and dH relative L2 errors.  mean_vs_full: the relative
    distance of the mean dW from the full update G, and App. C's diagonal prediction of
    it, sqrt(sum_t (1/xi_t - 1) ||g_t||^2 / S) / ||G||, with ||g_t||^2 = delta_t^2 ||h_t||^2
    ||e_o - p_t||^2 = delta_t^2 gamma_t (gamma from the score proxy, delta_t the token's
    logit-gradient scale at weight 1, from the full call's log-probs).  Needs
    res['logp_full'] (reseed_mean(..., want_logp=True)).
    """
    import torch
    from paper_2606_29758_amd import pspo
    f32 = lambda x: float(np.float32(x))
    rel = lambda a, b: float(torch.linalg.vector_norm((a - b).double()) / torch.linalg.vector_norm(b.double()))
    S = res["seeds"]
    total = res["tokens"]
    G = res["full_dw"]
    gamma = pspo.score_proxy(dw.hidden_full, dw.w_head, dw.target_full, total, want_logp=False)["gamma"].double()
    rho = torch.exp(res["logp_full"].double() - dw.logp_old_full[:total].double())
    seq = torch.repeat_interleave(torch.arange(dw.P * dw.K, device=G.device), dw.lengths.long())
    A = dw.advantage.double()[seq]
    mu = ((A > 0) & (rho <= 1 + f32(dw.eps_high))) | ((A < 0) & (rho >= 1 - f32(dw.eps_low)))
    delta = -f32(dw.loss_scale) * mu.double() * rho * A
    var = torch.sum((res["weight_full"].double() - 1.0) * delta ** 2 * gamma) / S
    return {
        "seeds": S,
        "tokens": total,
        "identity": {"loss_rel": abs(res["mean_loss"] - res["weighted_loss"]) / abs(res["weighted_loss"]),
                     "dw_rel_l2": rel(res["mean_dw"], res["weighted_dw"]),
                     "dh_rel_l2": rel(res["mean_dh"], res["weighted_dh"])},
        "mean_vs_full": {"dw_rel_dev": rel(res["mean_dw"], G),
                         "app_c_diagonal_prediction": float(torch.sqrt(var) / torch.linalg.vector_norm(G.double())),
                         "loss_mean": res["mean_loss"], "loss_full": res["full_loss"]},
    }


def mfma_loop_peak(iters=32768, blocks=1024):
    """The matrix cores' sustained bf16 rate on the products' MFMA form with no memory
    traffic (pspo_mfma_loop), timed with events on the current stream."""
    import torch
    from paper_2606_29758_amd import pspo
    out = pspo.mfma_loop(iters, blocks)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    reps = 3
    s.record(stream)
    for _ in range(reps):
        pspo.mfma_loop(iters, blocks, out)
    e.record(stream)
    torch.cuda.synchronize()
    ms = s.elapsed_time(e) / reps
    flops = blocks * 4.0 * iters * 16 * 16384
    tf = flops / (ms * 1e-3) / 1e12
    return {"achieved": tf, "unit": "TFLOP/s", "frac_of_peak": tf / PEAK_BF16_TFLOPS,
            "what": f"{blocks} work-groups x 4 waves x {iters} rounds of 16 independent "
                    f"v_mfma_f32_16x16x32_bf16 on random bf16 operands, no memory traffic ({ms:.1f} ms)"}


def bench_proxy(args):
    """The "Computing xi" stage before an update: the output-head score proxy of every
    completion token on the matrix cores, the per-step weights and the designed survival
    tables (budget 128, the paper's default)."""
    import torch
    from paper_2606_29758_amd import pipeline, pspo, synth

    wl = synth.make_workload(args.workload)
    cfg = wl.cfg
    dw = pipeline.upload(wl, np.zeros(wl.total_tokens, dtype=np.float32))
    N = int(wl.total_tokens)
    ids, logp = synth.make_topk(wl)
    dev = "cuda"
    t_ids = torch.from_numpy(ids).to(dev)
    t_logp = torch.from_numpy(logp).to(dev)
    full_off = torch.from_numpy(np.concatenate([[0], np.cumsum(wl.lengths)]).astype(np.int32)).to(dev)
    rewards = torch.from_numpy(wl.rewards.astype(np.float32)).to(dev)
    total_T = int(wl.xi_off[-1])
    ws = torch.empty(pspo.score_proxy_workspace_bytes(N, cfg.d, cfg.V), dtype=torch.uint8, device=dev)
    xi = torch.empty(total_T, dtype=torch.float64, device=dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    budget = 128.0
    stream = torch.cuda.current_stream()
    ev = lambda: torch.cuda.Event(enable_timing=True)

    def run(marks=None):
        if marks:
            marks[0].record(stream)
        prox = pspo.score_proxy(dw.hidden_full, dw.w_head, dw.target_full, N, want_logp=False,
                                workspace=ws, err_flag=err)
        if marks:
            marks[1].record(stream)
        wts = pspo.design_weights(prox["gamma"], t_ids, t_logp, dw.lengths, full_off, rewards, dw.xi_off,
                                  cfg.P, cfg.K, total_T, err_flag=err)
        pspo.design_cutoffs(wts["w"], dw.xi_off, cfg.P, total_T, budget, out=xi, err_flag=err)

    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    s, e = ev(), ev()
    proxy_ms = []
    pspo.timing_start(4 * args.steps)   # events on the call's stream around its matrix-core product
    s.record(stream)
    for _ in range(args.steps):
        m = (ev(), ev())
        run(m)
        proxy_ms.append(m)
    e.record(stream)
    torch.cuda.synchronize()
    timing = pspo.timing_stop()
    assert timing["proxy"]["count"] == args.steps, timing["proxy"]
    prod_ms = timing["proxy"]["ms"] / timing["proxy"]["count"]
    ms = s.elapsed_time(e) / args.steps
    pms = float(np.mean([a.elapsed_time(b) for a, b in proxy_ms]))
    assert int(err.item()) == 0, "device error flag raised"
    flops = 2.0 * N * cfg.V * cfg.d
    achieved = flops / (pms * 1e-3) / 1e12
    prod_achieved = flops / (prod_ms * 1e-3) / 1e12
    # memory-side bytes per launch of the score-proxy product from the committed counter
    # runs, only while the kernels are the ones they were taken on
    traffic, counters = None, None
    if os.path.exists(XI_TRAFFIC_FILE):
        with open(XI_TRAFFIC_FILE) as f:
            t = json.load(f)
        if t.get("N") == N and t.get("workload") == args.workload and t.get("source_hash") == source_hash():
            traffic = t["bytes_per_launch"]
            counters = {"source": os.path.relpath(XI_TRAFFIC_FILE, ROOT) + " (rocprofv3 --pmc runs of the same "
                                                                           "kernel on this batch, not re-measured here)",
                        "mfma_busy_pct": t.get("mfma_busy_pct"), "clock_ghz": t.get("clock_ghz"),
                        "memory_read_GBps": t["fetch_bytes_per_launch"] / (prod_ms * 1e-3) / 1e9,
                        "memory_write_GBps": t["write_bytes_per_launch"] / (prod_ms * 1e-3) / 1e9}
    result = {
        "metric": "completion tokens/sec for computing xi (score proxy on the matrix cores + cutoff design); "
                  "% of bf16 MFMA peak",
        "value": N / (ms * 1e-3), "unit": "completion tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"{args.workload}: every completion token, d={cfg.d}, V={cfg.V}, top-16 lists, "
                               f"budget {budget:g}", "tokens": N, "steps_designed": total_T},
        "score_proxy_ms": pms, "design_ms": ms - pms,
        "roofline": {"bound": "mfma",
                     "kernel": "gemm_nt_kernel<EpiProxy> (the score-proxy logit product: bf16 MFMA, two-sum "
                               "epilogue), timed live with HIP events the library records around it",
                     "flops": "2 N V d per launch", "launch_ms": prod_ms, "achieved": prod_achieved,
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": prod_achieved / PEAK_BF16_TFLOPS,
                     "traffic": traffic},
        "score_proxy_call": {"what": "the whole pspo_score_proxy call (operand copies, the product, row norms, "
                                     "finalize): 2 N V d flops / its mean duration",
                             "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                             "frac": achieved / PEAK_BF16_TFLOPS},
    }
    if counters is not None:
        result["counters"] = counters
    if not args.no_cpu_baseline:
        from threadpoolctl import threadpool_info
        from oracle import cutoff_design as ocd
        from oracle import score_proxy as osp
        n = min(args.cpu_tokens, N)
        t0 = time.perf_counter()
        g = osp.score_proxy(wl.hidden_bits[:n], wl.w_bits, wl.target_full[:n])["gamma"]
        # the design of the first completion's prompt, on its first n tokens
        L = np.minimum(wl.lengths[:cfg.K], max(n // cfg.K, 1))
        off = np.concatenate([[0], np.cumsum(wl.lengths[:cfg.K])])
        rows = np.concatenate([np.arange(off[k], off[k] + L[k]) for k in range(cfg.K)])
        gs = np.concatenate([g, np.zeros(max(0, rows.max() + 1 - n))])[rows]
        w = ocd.proxy_weights(gs, ids[rows], logp[rows], L, wl.rewards[:cfg.K], 1, cfg.K)["w"]
        ocd.design_xi(w, budget)
        dt = time.perf_counter() - t0
        threads = max([p.get("num_threads", 1) for p in threadpool_info() if p.get("user_api") == "blas"] or [1])
        result["cpu_baseline"] = {"value": n / dt, "unit": "completion tokens/s", "cores": int(threads),
                                  "kind": "oracle",
                                  "sample": f"score proxy of the first {n} completion tokens and the design of one "
                                            f"prompt over them (float64 numpy, {dt:.1f} s)"}
    print(json.dumps(result), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this implementation runs on one GPU only (no multi-GPU path); --gpus must be 1",
                          "n_gpus_requested": args.gpus}), flush=True)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration()
        return
    if args.which == "xi":
        bench_proxy(args)
        return

    import torch
    from paper_2606_29758_amd import pipeline, pspo, synth

    wl = synth.make_workload(args.workload)
    cfg = wl.cfg
    logp_old = synth.load_stored_logp_old(wl, GOLDEN)
    dw = pipeline.upload(wl, logp_old)
    step = pipeline.Step(dw)
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream()
    ev = lambda: torch.cuda.Event(enable_timing=True)
    for _ in range(args.warmup):
        step(args.seed, want_logp=False)
    torch.cuda.synchronize()
    torch.cuda.reset_peak_memory_stats()

    loss_ms = []
    starts, ends, pack_marks = [], [], []
    t_start, t_end = ev(), ev()
    pspo.timing_start(64 * args.steps)   # events on the call's stream around each product
    torch.cuda.synchronize()
    t_start.record(stream)
    N = 0
    for _ in range(args.steps):
        p0 = ev()
        p0.record(stream)
        pk = step.sample_and_pack(args.seed)
        p1 = ev()
        p1.record(stream)
        pack_marks.append((p0, p1))
        N = int(pk["n_tokens"].item())
        s, e = ev(), ev()
        s.record(stream)
        out = step.loss(pk, N, want_logp=False)
        e.record(stream)
        starts.append(s)
        ends.append(e)
    t_end.record(stream)
    torch.cuda.synchronize()
    timing = pspo.timing_stop()
    ms_step = t_start.elapsed_time(t_end) / args.steps
    loss_ms = [s.elapsed_time(e) for s, e in zip(starts, ends)]
    loss_avg = float(np.mean(loss_ms))
    pack_avg = float(np.mean([a.elapsed_time(b) for a, b in pack_marks]))
    assert int(step.err.item()) == 0, "device error flag raised"
    peak_bytes = torch.cuda.max_memory_allocated()
    ws_bytes = int(step.workspace.numel())

    # the same loss calls with the opt-in PSPO_KEEP_LOGITS (the first vocabulary
    # chunk's logits kept by the forward as fp16 offsets, converted by the backward)
    keep = None
    if not args.no_keep_control:
        step.loss(pk, N, flags=pspo.PSPO_KEEP_LOGITS, want_logp=False)
        torch.cuda.synchronize()
        rs, re_ = ev(), ev()
        nrep = max(3, args.steps // 2)
        rs.record(stream)
        for _ in range(nrep):
            step.loss(pk, N, flags=pspo.PSPO_KEEP_LOGITS, want_logp=False)
        re_.record(stream)
        torch.cuda.synchronize()
        keep = {"loss_call_ms": rs.elapsed_time(re_) / nrep,
                "workspace_bytes": int(pspo.loss_workspace_bytes(N, cfg.d, cfg.V, pspo.PSPO_KEEP_LOGITS))}
    mfma_peak = None if args.no_mfma_peak else mfma_loop_peak()

    # the full-trajectory control on the same batch (every xi = 1: the standard, untruncated
    # update): its loss-call time against the truncated one
    full = None
    if not args.no_full_control:
        import dataclasses
        dw_full = dataclasses.replace(dw, xi=torch.ones_like(dw.xi))
        step_full = pipeline.Step(dw_full)
        for _ in range(2):
            step_full(args.seed, want_logp=False)
        torch.cuda.synchronize()
        pkf = step_full.sample_and_pack(args.seed)
        Nf = int(pkf["n_tokens"].item())
        fs, fe = ev(), ev()
        fs.record(stream)
        nrep = max(3, args.steps // 2)
        for _ in range(nrep):
            step_full.loss(pkf, Nf, want_logp=False)
        fe.record(stream)
        torch.cuda.synchronize()
        full = {"tokens": Nf, "loss_call_ms": fs.elapsed_time(fe) / nrep}
        del step_full, dw_full
    # the reseed check (after the timed region): the mean of the truncated update over
    # --reseeds cutoff draws against the weighted and the plain full-trajectory calls
    reseed = None
    if not args.no_full_control and args.reseeds > 0:
        t0 = time.perf_counter()
        res = pipeline.reseed_mean(step, range(args.reseeds), want_logp=True)
        reseed = reseed_summary(dw, res)
        del res
        torch.cuda.synchronize()
        reseed["seconds"] = time.perf_counter() - t0
    st = out["stats"].cpu().numpy()
    n_fwd = N - int(st[2])   # tokens of completions with A != 0: the forward's columns
    n_bwd = int(st[4])       # tokens with a nonzero logit-gradient row

    # matrix-core work the step needs: the forward over the n_fwd tokens whose loss
    # term can be nonzero (2 n_fwd V d), dH and dW over the n_bwd tokens whose logit
    # gradient is not zero (4 n_bwd V d); every other token contributes exactly zero
    flops = (2.0 * n_fwd + 4.0 * n_bwd) * cfg.V * cfg.d
    achieved = flops / (loss_avg * 1e-3) / 1e12
    dense_equiv = 6.0 * N * cfg.V * cfg.d / (loss_avg * 1e-3) / 1e12
    # each matrix-core product of the call, timed live (events on the call's stream)
    prod_flops = {"forward": 2.0 * n_fwd * cfg.V * cfg.d, "logit_grad": 2.0 * n_bwd * cfg.V * cfg.d,
                  "dw": 2.0 * n_bwd * cfg.V * cfg.d, "dh": 2.0 * n_bwd * cfg.V * cfg.d}
    products = {}
    for k, f in prod_flops.items():
        t = timing[k]
        assert t["count"] > 0 and t["count"] % args.steps == 0, (k, t)
        per_call = t["ms"] / args.steps
        tf = f / (per_call * 1e-3) / 1e12
        products[k] = {"ms_per_call": per_call, "records_per_call": t["count"] // args.steps,
                       "flops_per_call": f, "achieved": tf, "frac": tf / PEAK_BF16_TFLOPS}
    products["what"] = ("ms per call from HIP events around each product (all its launches; the logit-"
                        "gradient, dW and dH products once per vocabulary chunk, dW and dH with their K-split "
                        "tails); flops: the forward over n_fwd tokens, the other three over n_bwd tokens "
                        "(the logit-gradient product recomputes the logits the forward did not keep)")
    fwd_launch_ms = timing["forward"]["ms"] / timing["forward"]["count"]
    # HBM bytes per call from the committed counter runs, only while the kernels
    # are still the ones those counters were taken on
    traffic, fwd_traffic, counters = None, None, None
    if os.path.exists(TRAFFIC_FILE):
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
        if t.get("N") == N and t.get("workload") == args.workload and t.get("source_hash") == source_hash():
            traffic = t.get("bytes_per_call")
            fwd_traffic = t["per_kernel_fetch_bytes"]["EpiForward"] + t["per_kernel_write_bytes"]["EpiForward"]
            # rocprofv3 counters of the same kernels and batch (committed under profiles/):
            # matrix-core busy fraction and clock of the products, and the memory-side
            # (beyond L2) read and write volume per call as rates at this run's call time
            counters = {"source": os.path.relpath(TRAFFIC_FILE, ROOT) + " (rocprofv3 --pmc runs of the same "
                                                                        "kernels on this batch, not re-measured here)",
                        "mfma_busy_pct": t.get("mfma_busy_pct"),
                        "clock_ghz": t.get("clock_ghz"),
                        "memory_read_GBps": t["fetch_bytes_per_call"] / (loss_avg * 1e-3) / 1e9,
                        "memory_write_GBps": t["write_bytes_per_call"] / (loss_avg * 1e-3) / 1e9}

    result = {
        "metric": "prefix tokens/sec for fused LM-head PPO loss fwd+bwd; % of bf16 MFMA peak",
        "value": N / (ms_step * 1e-3),
        "unit": "prefix tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": f"{args.workload}: {cfg.P} prompts x {cfg.K} rollouts, d={cfg.d}, V={cfg.V}, "
                        f"lengths {cfg.length_law}, cutoff Beta law {cfg.beta_law}"
                        f"{' (pinned to full length)' if cfg.full_trajectory else ''}, "
                        f"logp_old noise sigma {cfg.sigma_lp}",
            "prefix_tokens": N,
            "forward_tokens": n_fwd,
            "backward_tokens": n_bwd,
            "total_tokens": int(wl.total_tokens),
            "kept_fraction": N / wl.total_tokens,
            "global_batch": cfg.R,
            "parallelism": "single GPU",
        },
        "loss_call_ms": loss_avg,
        "loss_call_ms_spread": {"median": float(np.median(loss_ms)), "min": float(np.min(loss_ms)),
                                "max": float(np.max(loss_ms))},
        # the last timed step's own numbers (the loss call's stats output)
        "step_stats": {
            "loss": float(out["loss"].item()),
            "clipped_fraction": float(st[1]) / max(n_fwd, 1),   # of the tokens with A != 0
            "zero_advantage_tokens": int(st[2]),
            "max_weight": float(st[3]),
            "prefix_tokens_per_prompt": N / cfg.P,
            "mean_prefix_length": N / cfg.R,
            "mean_completion_length": int(wl.total_tokens) / cfg.R,
        },
        "sample_pack_ms": pack_avg,
        "memory": {"peak_device_bytes": int(peak_bytes),
                   "loss_workspace_bytes": ws_bytes,
                   "logits_fp32_bytes_avoided": int(N) * int(cfg.V) * 4},
        "pct_bf16_peak": 100.0 * achieved / PEAK_BF16_TFLOPS,
        "dense_equivalent_tflops": dense_equiv,
        "roofline": {
            "bound": "mfma",
            "kernel": "gemm_nt_kernel<EpiForward> (the forward logit product of pspo_loss_fwd_bwd: bf16 MFMA, "
                      "per-token softmax partials in the epilogue, no logit stored)",
            "flops": "2 n_fwd V d per launch (the tokens of completions with A != 0)",
            "launch_ms": fwd_launch_ms,
            "achieved": prod_flops["forward"] / (fwd_launch_ms * 1e-3) / 1e12,
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": prod_flops["forward"] / (fwd_launch_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
            "traffic": fwd_traffic,
        },
        "products": products,
        "loss_call": {
            "what": "the whole pspo_loss_fwd_bwd call: (2 n_fwd + 4 n_bwd) V d needed flops per call (forward "
                    "over the tokens of completions with A != 0, dH and dW over the tokens with a nonzero "
                    "logit gradient) / mean call duration; traffic: memory-side bytes of all its kernels",
            "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
            "frac": achieved / PEAK_BF16_TFLOPS, "traffic": traffic,
        },
    }
    if counters is not None:
        result["counters"] = counters
    if keep is not None:
        result["keep_logits_control"] = dict(
            keep, pct_bf16_peak=100.0 * flops / (keep["loss_call_ms"] * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
            what="the same calls with PSPO_KEEP_LOGITS: the first vocabulary chunk's logits kept by the "
                 "forward (fp16 offsets, Vc x N x 2 bytes) and converted instead of recomputed")
    if mfma_peak is not None:
        result["mfma_loop_peak"] = mfma_peak
    if full is not None:
        result["full_trajectory_control"] = dict(full, prefix_vs_full_ratio=loss_avg / full["loss_call_ms"])
    if reseed is not None:
        result["reseed_check"] = reseed
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(wl, logp_old, args.cpu_tokens, args.seed)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
