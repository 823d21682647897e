"""The C ABI without a GPU: the library loads, exports every symbol the header
declares, and rejects bad arguments with the documented status before any
device work (these paths never reach the HIP runtime)."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2606_29758_amd import pspo

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
OK, INVALID, BAD_XI, WORKSPACE, UNSUPPORTED = 0, 1, 2, 3, 4


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(pspo.LIB_PATH):
        pytest.fail("libpspo.so is not built (run __graft_entry__.build())")
    return pspo.load()


def _declared():
    with open(os.path.join(ROOT, "include", "pspo.h")) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(pspo_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    names = _declared()
    assert len(names) == 17
    for name in names:
        assert hasattr(lib, name), name
    assert sorted(pspo.exported_symbols()) == names


def test_version_and_status_strings(lib):
    assert lib.pspo_abi_version() == 6
    assert lib.pspo_status_string(0) == b"PSPO_OK"
    assert lib.pspo_status_string(3) == b"PSPO_ERR_WORKSPACE"
    assert lib.pspo_status_string(99) == b"PSPO_ERR_UNKNOWN"


def test_timing_argument_errors(lib):
    """The measurement mode's host paths: nothing to stop before a start, a start needs
    1 <= max_records <= 2^20 (the event creation itself needs a device)."""
    ms = (ctypes.c_double * 5)()
    cnt = (ctypes.c_int32 * 5)()
    assert lib.pspo_timing_stop(ms, cnt) == INVALID
    assert b"not started" in lib.pspo_last_error()
    assert lib.pspo_timing_start(0) == INVALID
    assert lib.pspo_timing_start(-3) == INVALID
    assert lib.pspo_timing_start((1 << 20) + 1) == INVALID
    assert lib.pspo_timing_stop(ms, cnt) == INVALID   # still not started
    with pytest.raises(pspo.PspoError, match="INVALID_ARG"):
        pspo.timing_stop()


def _vx(xi, off):
    xi = np.ascontiguousarray(xi, dtype=np.float64)
    off = np.ascontiguousarray(off, dtype=np.int64)
    return pspo.load().pspo_validate_xi_host(xi.ctypes.data_as(ctypes.c_void_p),
                                             off.ctypes.data_as(ctypes.c_void_p), len(off) - 1)


def test_validate_xi_host(lib):
    assert _vx([1.0, 0.5, 0.5, 0.1, 1.0, 2 ** -40], [0, 4, 6]) == OK
    assert _vx([1.0, 0.5, 0.6], [0, 3]) == BAD_XI
    assert b"increases at t = 3" in lib.pspo_last_error()
    assert _vx([1.0, 0.0], [0, 2]) == BAD_XI
    assert _vx([1.25], [0, 1]) == BAD_XI
    assert _vx([np.nan], [0, 1]) == BAD_XI
    assert _vx([1.0], [1, 1]) == INVALID
    assert _vx([1.0, 1.0], [0, 2, 1]) == INVALID
    assert _vx([], [0]) == OK
    with pytest.raises(pspo.PspoError, match="BAD_XI"):
        pspo.validate_xi_host([0.5, 0.7], [0, 2])


FAKE = ctypes.c_void_p(1 << 20)   # aligned, never dereferenced on these paths


def _sample(lib, **kw):
    a = dict(xi=FAKE, xi_off=FAKE, lengths=FAKE, P=1, K=1, seed=0, offset=0, cutoffs=FAKE, err=None, stream=None)
    a.update(kw)
    return lib.pspo_sample_cutoffs(a["xi"], a["xi_off"], a["lengths"], a["P"], a["K"], a["seed"], a["offset"],
                                   a["cutoffs"], a["err"], a["stream"])


def test_sample_cutoffs_argument_errors(lib):
    assert _sample(lib, P=-1) == INVALID
    assert _sample(lib, P=0) == OK          # nothing to do: no device work at all
    assert _sample(lib, K=0) == OK
    assert _sample(lib, xi=None) == INVALID
    assert _sample(lib, cutoffs=None) == INVALID
    assert _sample(lib, lengths=ctypes.c_void_p((1 << 20) + 2)) == INVALID
    assert _sample(lib, P=1 << 16, K=1 << 16) == INVALID


def _pack(lib, **kw):
    a = dict(cut=FAKE, len=FAKE, xi=FAKE, xio=FAKE, P=2, K=2, cap=16, tf=FAKE, lf=FAKE, hf=FAKE, d=64,
             cu=FAKE, fo=FAKE, src=FAKE, seq=FAKE, w=FAKE, t=FAKE, l=FAKE, h=FAKE, n=FAKE, err=None)
    a.update(kw)
    return lib.pspo_pack_prefixes(a["cut"], a["len"], a["xi"], a["xio"], a["P"], a["K"], a["cap"], a["tf"],
                                  a["lf"], a["hf"], a["d"], a["cu"], a["fo"], a["src"], a["seq"], a["w"], a["t"],
                                  a["l"], a["h"], a["n"], a["err"], None)


def test_pack_prefixes_argument_errors(lib):
    assert _pack(lib, cap=-1) == INVALID
    assert _pack(lib, t=None) == INVALID            # target_full given without target
    assert _pack(lib, lf=None) == INVALID
    assert _pack(lib, hf=None) == INVALID
    assert _pack(lib, d=12) == UNSUPPORTED           # 16-byte row gather needs d % 8 == 0
    assert _pack(lib, d=0) == UNSUPPORTED
    assert _pack(lib, h=ctypes.c_void_p((1 << 20) + 8)) == INVALID
    assert _pack(lib, cu=None) == INVALID
    assert _pack(lib, src=None) == INVALID
    assert _pack(lib, P=300, K=300) == UNSUPPORTED   # more than 65535 completions


def _loss(lib, **kw):
    N, d, V = kw.get("N", 100), kw.get("d", 128), kw.get("V", 1000)
    ws_bytes = lib.pspo_loss_workspace_bytes(max(N, 0), d, max(V, 1), 0)
    a = dict(h=FAKE, w=FAKE, t=FAKE, lo=FAKE, c=FAKE, s=FAKE, adv=FAKE, N=N, d=d, V=V, R=4, el=0.1, eh=0.1,
             scale=0.25, flags=0, loss=FAKE, dh=FAKE, dw=FAKE, lp=None, st=None, err=None, ws=FAKE, wsb=ws_bytes)
    a.update(kw)
    return lib.pspo_loss_fwd_bwd(a["h"], a["w"], a["t"], a["lo"], a["c"], a["s"], a["adv"], a["N"], a["d"], a["V"],
                                 a["R"], a["el"], a["eh"], a["scale"], a["flags"], a["loss"], a["dh"], a["dw"],
                                 a["lp"], a["st"], a["err"], a["ws"], a["wsb"], None)


def test_loss_argument_errors(lib):
    assert _loss(lib, N=-1) == INVALID
    assert _loss(lib, d=0) == INVALID
    assert _loss(lib, V=0) == INVALID
    assert _loss(lib, d=100) == UNSUPPORTED          # d % 8 != 0
    # sizes beyond the copy kernels' grid (65535 blocks of 32 rows on its y axis)
    assert _loss(lib, N=2730 * 768 + 1, wsb=0) == UNSUPPORTED        # pads to 2097408 > 2097120 rows
    assert b"at most 2097120" in lib.pspo_last_error()
    assert _loss(lib, V=5461 * 384 + 1) == UNSUPPORTED                # pads to 2097408 rows
    assert _loss(lib, d=65535 * 32 + 8) == UNSUPPORTED
    assert _loss(lib, N=2730 * 768, wsb=0) == WORKSPACE               # 2096640 tokens: within the limit
    assert _loss(lib, V=5461 * 384, wsb=0) == WORKSPACE               # 2097024 rows: within the limit
    _loss(lib, d=96)                                 # d % 8 == 0 passes the argument checks
    assert b"multiple of" not in lib.pspo_last_error()
    assert _loss(lib, R=0) == INVALID
    assert _loss(lib, flags=2) == INVALID            # the retired bit
    assert _loss(lib, flags=8) == INVALID            # unknown flag bit
    assert _loss(lib, el=1.0) == INVALID
    assert _loss(lib, eh=-0.1) == INVALID
    assert _loss(lib, el=float("nan")) == INVALID
    assert _loss(lib, scale=float("inf")) == INVALID
    assert _loss(lib, loss=None) == INVALID
    assert _loss(lib, dw=None) == INVALID
    assert _loss(lib, h=None) == INVALID
    assert _loss(lib, dh=None) == INVALID
    assert _loss(lib, h=ctypes.c_void_p((1 << 20) + 4)) == INVALID
    assert _loss(lib, ws=ctypes.c_void_p((1 << 20) + 16)) == INVALID
    assert _loss(lib, ws=None) == INVALID
    assert _loss(lib, wsb=1024) == WORKSPACE
    assert b"workspace too small" in lib.pspo_last_error()


def test_workspace_bytes_keep_flag(lib):
    # with PSPO_KEEP_LOGITS the forward keeps the first vocabulary chunk's
    # logits as fp16 offsets: Vc x round_up(N, 768) x 2 bytes more (Vc = 50688 at
    # d = 3584, V = 152064: the padded vocabulary split evenly into three chunks
    # of about the round-filling width 49152; the whole padded vocabulary when
    # that is smaller; d = 4096: width 6144, 25 chunks since the remainder of
    # 4608 rows exceeds a quarter of it)
    for N, d, V, vc in ((1000, 3584, 152064, 50688), (300, 128, 2048, 2304), (5000, 4096, 151936, 6144)):
        keep = lib.pspo_loss_workspace_bytes(N, d, V, 4)
        lean = lib.pspo_loss_workspace_bytes(N, d, V, 0)
        npad = -(-N // 768) * 768
        assert keep - lean == vc * npad * 2, (N, d, V)


def test_workspace_bytes(lib):
    assert lib.pspo_loss_workspace_bytes(-1, 128, 100, 0) == 0
    assert lib.pspo_loss_workspace_bytes(10, 0, 100, 0) == 0
    a = lib.pspo_loss_workspace_bytes(1000, 3584, 152064, 0)
    b = lib.pspo_loss_workspace_bytes(2000, 3584, 152064, 0)
    assert 0 < a < b
    # the dominant terms: bf16 logit-gradient chunks in both layouts (2 x Npad x 16384 x 2 B)
    assert b > 2 * 2048 * 16384 * 2


def _proxy(lib, **kw):
    N, d, V = kw.get("N", 100), kw.get("d", 128), kw.get("V", 1000)
    ws_bytes = lib.pspo_score_proxy_workspace_bytes(max(N, 0), d, max(V, 1))
    a = dict(h=FAKE, w=FAKE, t=FAKE, N=N, d=d, V=V, g=FAKE, lp=None, ps=None, err=None, ws=FAKE, wsb=ws_bytes)
    a.update(kw)
    return lib.pspo_score_proxy(a["h"], a["w"], a["t"], a["N"], a["d"], a["V"], a["g"], a["lp"], a["ps"],
                                a["err"], a["ws"], a["wsb"], None)


def test_score_proxy_argument_errors(lib):
    assert _proxy(lib, N=0, h=None, t=None, g=None, ws=None) == OK   # nothing to do, no device work
    assert _proxy(lib, N=-1) == INVALID
    assert _proxy(lib, d=0) == INVALID
    assert _proxy(lib, V=0) == INVALID
    assert _proxy(lib, d=100) == UNSUPPORTED
    assert _proxy(lib, N=65535 * 32 + 1) == UNSUPPORTED              # pads to 2097152 rows
    assert _proxy(lib, V=5461 * 384 + 1) == UNSUPPORTED
    assert _proxy(lib, N=8191 * 256, wsb=0) == WORKSPACE              # 2096896 rows: within the limit
    _proxy(lib, d=96)
    assert b"multiple of" not in lib.pspo_last_error()
    assert _proxy(lib, g=None) == INVALID
    assert _proxy(lib, h=None) == INVALID
    assert _proxy(lib, t=None) == INVALID
    assert _proxy(lib, h=ctypes.c_void_p((1 << 20) + 4)) == INVALID
    assert _proxy(lib, lp=ctypes.c_void_p((1 << 20) + 2)) == INVALID
    assert _proxy(lib, ws=None) == INVALID
    assert _proxy(lib, wsb=1024) == WORKSPACE
    assert b"workspace too small" in lib.pspo_last_error()


def test_score_proxy_workspace_bytes(lib):
    assert lib.pspo_score_proxy_workspace_bytes(-1, 128, 100) == 0
    assert lib.pspo_score_proxy_workspace_bytes(10, 128, 0) == 0
    # three float32 partials per (256-row vocabulary tile, token) plus two per-token arrays
    b = lib.pspo_score_proxy_workspace_bytes(1000, 3584, 152064)
    assert b >= 3 * 594 * 1024 * 4 + 2 * 1024 * 4


def test_design_argument_errors(lib):
    def weights(**kw):
        a = dict(g=FAKE, ids=FAKE, lp=FAKE, k=16, len=FAKE, off=FAKE, rew=FAKE, xo=FAKE, P=2, K=8, T=100,
                 w=FAKE, gb=None, u=None)
        a.update(kw)
        return lib.pspo_design_weights(a["g"], a["ids"], a["lp"], a["k"], a["len"], a["off"], a["rew"], a["xo"],
                                       a["P"], a["K"], a["T"], a["w"], a["gb"], a["u"], None, None)
    assert weights(T=0, g=None, w=None) == OK          # nothing to do, no device work
    assert weights(P=0) == INVALID
    assert weights(K=0) == INVALID
    assert weights(T=-1) == INVALID
    assert weights(K=65) == UNSUPPORTED
    assert weights(k=0) == UNSUPPORTED
    assert weights(K=16, k=17) == UNSUPPORTED          # K * topk > 256
    assert weights(w=None) == INVALID
    assert weights(gb=ctypes.c_void_p((1 << 20) + 4)) == INVALID

    def cutoffs(**kw):
        T = kw.get("T", 100)
        a = dict(w=FAKE, xo=FAKE, P=2, T=T, B=128.0, v=0, lam=0.0, xi=FAKE, ws=FAKE,
                 wsb=lib.pspo_design_workspace_bytes(max(T, 0)))
        a.update(kw)
        return lib.pspo_design_cutoffs(a["w"], a["xo"], a["P"], a["T"], a["B"], a["v"], a["lam"], a["xi"], a["ws"],
                                       a["wsb"], None, None)
    assert cutoffs(T=0, w=None, xi=None, ws=None) == OK
    assert cutoffs(P=0) == INVALID
    assert cutoffs(v=4) == INVALID
    assert cutoffs(B=0.0) == INVALID
    assert cutoffs(B=float("nan")) == INVALID
    assert cutoffs(lam=-1.0) == INVALID
    assert cutoffs(xi=None) == INVALID
    assert cutoffs(ws=None) == INVALID
    assert cutoffs(wsb=64) == WORKSPACE
    assert lib.pspo_design_workspace_bytes(-1) == 0
    assert lib.pspo_design_workspace_bytes(1000) >= 16 * 1000


def test_binding_refuses_host_tensors():
    import torch
    with pytest.raises(ValueError, match="device tensor"):
        pspo.sample_cutoffs(torch.ones(3, dtype=torch.float64), torch.zeros(2, dtype=torch.int64),
                            torch.ones(1, dtype=torch.int32), 1, 1, 0)


def test_mfma_loop_argument_errors(lib):
    out = ctypes.c_void_p(1 << 20)
    assert lib.pspo_mfma_loop(0, 4, out, None) == INVALID
    assert lib.pspo_mfma_loop(4, 0, out, None) == INVALID
    assert lib.pspo_mfma_loop(4, 4, None, None) == INVALID
    assert lib.pspo_mfma_loop(4, 4, ctypes.c_void_p((1 << 20) + 2), None) == INVALID


def test_binding_checks_gradient_shapes():
    """The kernels write d_hidden rows 0..N-1 and every row of d_w_head: the binding refuses
    buffers of another shape before anything reaches the library (shapes are checked ahead of
    devices, so host tensors exercise it)."""
    import torch
    V, d, N = 40, 16, 5
    w = torch.zeros(V, d, dtype=torch.bfloat16)
    h = torch.zeros(N, d, dtype=torch.bfloat16)
    i32 = torch.zeros(N, dtype=torch.int32)
    f = torch.zeros(N, dtype=torch.float32)
    adv = torch.zeros(2, dtype=torch.float32)

    def call(**kw):
        return pspo.loss_fwd_bwd(h, w, i32, f, f, i32, adv, N, 0.1, 0.1, 1.0, **kw)

    with pytest.raises(ValueError, match="d_hidden"):
        call(d_hidden=torch.zeros(N - 1, d))
    with pytest.raises(ValueError, match="d_hidden"):
        call(d_hidden=torch.zeros(N, d + 8))
    with pytest.raises(ValueError, match="d_w_head"):
        call(d_w_head=torch.zeros(V, d + 8))
    with pytest.raises(ValueError, match="d_w_head"):
        call(d_w_head=torch.zeros(V - 1, d))
    with pytest.raises(ValueError, match="fewer than N rows"):
        pspo.loss_fwd_bwd(h[:3], w, i32, f, f, i32, adv, N, 0.1, 0.1, 1.0)
    with pytest.raises(ValueError, match="device tensor"):   # right shapes: the device check follows
        call(d_hidden=torch.zeros(N, d), d_w_head=torch.zeros(V, d))


def test_design_noalloc_argument_errors(lib):
    def call(**kw):
        a = dict(w=FAKE, xo=FAKE, P=2, T=100, B=8.0, v=0, lam=0.0, xi=FAKE)
        a.update(kw)
        return lib.pspo_design_cutoffs_noalloc(a["w"], a["xo"], a["P"], a["T"], a["B"], a["v"], a["lam"], a["xi"],
                                               None, None)
    assert call(T=0, w=None, xi=None) == OK
    assert call(P=0) == INVALID
    assert call(v=4) == INVALID
    assert call(B=-1.0) == INVALID
    assert call(xi=None) == INVALID
    assert call(T=2 ** 19 + 1) == UNSUPPORTED          # beyond the static scratch (8 MiB)
    assert b"2^19" in lib.pspo_last_error()
    assert lib.pspo_design_workspace_bytes(2 ** 19) <= 8 << 20 < lib.pspo_design_workspace_bytes(2 ** 19 + 1)


def test_validate_xi_host_agrees_with_the_oracle(lib):
    """The library's host check of survival tables accepts exactly the tables the
    oracle's check accepts (Sec. 3.2: 1 >= xi_1 >= ... >= xi_T > 0), on random tables
    built to sit on and around every boundary: exact 0 and 1, values just above 1 or
    just below the previous one, NaN, +-inf, denormals, empty prompts."""
    from hypothesis import given, settings, strategies as st
    from oracle import cutoffs as ocut

    edge = st.sampled_from([0.0, 1.0, np.nextafter(1.0, 2.0), 0.5, np.nextafter(0.5, 0.0),
                            np.nextafter(0.5, 1.0), 5e-324, 2.0 ** -40, -0.0, float("nan"), float("inf"),
                            -float("inf"), -1e-300])
    val = st.one_of(edge, st.floats(min_value=0.0, max_value=1.0), st.floats(allow_nan=True))
    prompt = st.lists(val, min_size=0, max_size=6)

    @settings(max_examples=400, deadline=None, derandomize=True)
    @given(st.lists(prompt, min_size=1, max_size=4), st.booleans())
    def check(prompts, sort_desc):
        if sort_desc:   # mostly-valid tables too: each prompt's values sorted non-increasing
            prompts = [sorted(p, reverse=True) if not any(np.isnan(p)) else p for p in prompts]
        xi = np.array([v for p in prompts for v in p], dtype=np.float64)
        off = np.concatenate([[0], np.cumsum([len(p) for p in prompts])]).astype(np.int64)
        try:
            ocut.validate_xi(xi, off)
            want = OK
        except ValueError:
            want = BAD_XI
        assert _vx(xi, off) == want, (prompts, lib.pspo_last_error())

    check()
