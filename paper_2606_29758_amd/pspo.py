"""Python binding of libpspo (ctypes): argument marshalling only.

Every step runs in the HIP kernels of libpspo.so; PyTorch only supplies device
memory (tensors) and the current HIP stream.  If the library is missing the
calls raise: there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libpspo.so")

PSPO_ACCUMULATE_DW = 1
PSPO_KEEP_LOGITS = 4
DEVERR_TARGET, DEVERR_BAD_XI, DEVERR_CAPACITY, DEVERR_SEQ_ID, DEVERR_NONFINITE = 1, 2, 4, 8, 16

_P = ctypes.c_void_p
_I32, _I64, _U32, _U64, _F32, _SZ = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_float, ctypes.c_size_t

_SIGNATURES = {
    "pspo_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "pspo_last_error": (ctypes.c_char_p, []),
    "pspo_abi_version": (ctypes.c_int, []),
    "pspo_validate_xi_host": (ctypes.c_int, [_P, _P, _I32]),
    "pspo_sample_cutoffs": (ctypes.c_int, [_P, _P, _P, _I32, _I32, _U64, _U64, _P, _P, _P]),
    "pspo_pack_prefixes": (ctypes.c_int, [_P, _P, _P, _P, _I32, _I32, _I32, _P, _P, _P, _I32,
                                          _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P]),
    "pspo_loss_workspace_bytes": (_SZ, [_I32, _I32, _I32, _U32]),
    "pspo_loss_fwd_bwd": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P, _I32, _I32, _I32, _I32,
                                         _F32, _F32, _F32, _U32, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "pspo_score_proxy_workspace_bytes": (_SZ, [_I32, _I32, _I32]),
    "pspo_design_weights": (ctypes.c_int, [_P, _P, _P, _I32, _P, _P, _P, _P, _I32, _I32, _I64,
                                           _P, _P, _P, _P, _P]),
    "pspo_design_workspace_bytes": (_SZ, [_I64]),
    "pspo_design_cutoffs": (ctypes.c_int, [_P, _P, _I32, _I64, ctypes.c_double, _I32, ctypes.c_double,
                                           _P, _P, _SZ, _P, _P]),
    "pspo_score_proxy": (ctypes.c_int, [_P, _P, _P, _I32, _I32, _I32, _P, _P, _P, _P, _P, _SZ, _P]),
    "pspo_design_cutoffs_noalloc": (ctypes.c_int, [_P, _P, _I32, _I64, ctypes.c_double, _I32, ctypes.c_double,
                                                   _P, _P, _P]),
    "pspo_mfma_loop": (ctypes.c_int, [_I32, _I32, _P, _P]),
    "pspo_timing_start": (ctypes.c_int, [_I32]),
    "pspo_timing_stop": (ctypes.c_int, [_P, _P]),
}

_lib = None


class PspoError(RuntimeError):
    pass


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Loads libpspo.so (built by paper_2606_29758_amd.build); raises if it is missing."""
    global _lib
    if _lib is None:
        if not os.path.exists(path):
            raise PspoError(f"{path} not found: build it with `python -m paper_2606_29758_amd.build`")
        lib = ctypes.CDLL(path)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def exported_symbols():
    return list(_SIGNATURES)


def _check(rc: int) -> None:
    if rc != 0:
        lib = load()
        raise PspoError(f"{lib.pspo_status_string(rc).decode()}: {lib.pspo_last_error().decode()}")


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _dev(t: torch.Tensor, dtype, name: str) -> torch.Tensor:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.device.index != torch.cuda.current_device():
        raise ValueError(f"{name} is on {t.device}, but the calls run on the current device "
                         f"cuda:{torch.cuda.current_device()}")
    if t.dtype != dtype:
        raise TypeError(f"{name} must have dtype {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def validate_xi_host(xi, xi_off) -> None:
    """Host check of survival tables (numpy float64 / int64 arrays)."""
    import numpy as np
    xi = np.ascontiguousarray(xi, dtype=np.float64)
    xi_off = np.ascontiguousarray(xi_off, dtype=np.int64)
    _check(load().pspo_validate_xi_host(xi.ctypes.data_as(_P), xi_off.ctypes.data_as(_P), len(xi_off) - 1))


def sample_cutoffs(xi, xi_off, lengths, P: int, K: int, seed: int, offset: int = 0,
                   out: Optional[torch.Tensor] = None, err_flag: Optional[torch.Tensor] = None) -> torch.Tensor:
    _dev(xi, torch.float64, "xi")
    _dev(xi_off, torch.int64, "xi_off")
    _dev(lengths, torch.int32, "lengths")
    if out is None:
        out = torch.empty(P * K, dtype=torch.int32, device=lengths.device)
    _dev(out, torch.int32, "cutoffs")
    if err_flag is not None:
        _dev(err_flag, torch.int32, "err_flag")
    _check(load().pspo_sample_cutoffs(_ptr(xi), _ptr(xi_off), _ptr(lengths), P, K,
                                      seed & (2 ** 64 - 1), offset & (2 ** 64 - 1),
                                      _ptr(out), _ptr(err_flag), _stream()))
    return out


def pack_prefixes(cutoffs, lengths, xi, xi_off, P: int, K: int, capacity: int,
                  target_full=None, logp_old_full=None, hidden_full=None,
                  err_flag: Optional[torch.Tensor] = None) -> dict:
    """Returns device tensors: cu_seqlens, full_off, src_row, seq_id, weight, [target, logp_old,
    hidden] (all sized by `capacity`) and n_tokens (int32 [1])."""
    dev = lengths.device
    _dev(cutoffs, torch.int32, "cutoffs")
    _dev(lengths, torch.int32, "lengths")
    _dev(xi, torch.float64, "xi")
    _dev(xi_off, torch.int64, "xi_off")
    R = P * K
    out = dict(
        cu_seqlens=torch.empty(R + 1, dtype=torch.int32, device=dev),
        full_off=torch.empty(R + 1, dtype=torch.int32, device=dev),
        src_row=torch.empty(capacity, dtype=torch.int32, device=dev),
        seq_id=torch.empty(capacity, dtype=torch.int32, device=dev),
        weight=torch.empty(capacity, dtype=torch.float32, device=dev),
        n_tokens=torch.empty(1, dtype=torch.int32, device=dev),
    )
    d = 0
    if target_full is not None:
        _dev(target_full, torch.int32, "target_full")
        out["target"] = torch.empty(capacity, dtype=torch.int32, device=dev)
    if logp_old_full is not None:
        _dev(logp_old_full, torch.float32, "logp_old_full")
        out["logp_old"] = torch.empty(capacity, dtype=torch.float32, device=dev)
    if hidden_full is not None:
        _dev(hidden_full, torch.bfloat16, "hidden_full")
        d = hidden_full.shape[1]
        out["hidden"] = torch.empty((capacity, d), dtype=torch.bfloat16, device=dev)
    if err_flag is not None:
        _dev(err_flag, torch.int32, "err_flag")
    _check(load().pspo_pack_prefixes(
        _ptr(cutoffs), _ptr(lengths), _ptr(xi), _ptr(xi_off), P, K, capacity,
        _ptr(target_full), _ptr(logp_old_full), _ptr(hidden_full), d,
        _ptr(out["cu_seqlens"]), _ptr(out["full_off"]), _ptr(out["src_row"]), _ptr(out["seq_id"]),
        _ptr(out["weight"]), _ptr(out.get("target")), _ptr(out.get("logp_old")), _ptr(out.get("hidden")),
        _ptr(out["n_tokens"]), _ptr(err_flag), _stream()))
    return out


def loss_workspace_bytes(N: int, d: int, V: int, flags: int = 0) -> int:
    return int(load().pspo_loss_workspace_bytes(N, d, V, flags))


def loss_fwd_bwd(hidden, w_head, target, logp_old, weight, seq_id, advantage, N: int,
                 eps_low: float, eps_high: float, loss_scale: float, flags: int = 0,
                 d_w_head: Optional[torch.Tensor] = None, d_hidden: Optional[torch.Tensor] = None,
                 workspace: Optional[torch.Tensor] = None, want_logp: bool = True, want_stats: bool = True,
                 err_flag: Optional[torch.Tensor] = None) -> dict:
    """Loss and gradients for the first N rows of the packed per-token tensors.

    hidden: bf16 [>=N, d]; w_head: bf16 [V, d]; target int32, logp_old/weight float32,
    seq_id int32 (all [>=N]); advantage float32 [R].  d_hidden (float32 [>=N, d]) and
    d_w_head (float32 [V, d]) may be given.  Returns loss (float64 [1]),
    d_hidden (float32 [N, d] view), d_w_head (float32 [V, d]), logp_new, stats.
    Shapes are checked first (the kernels write d_hidden rows 0..N-1 and every row of
    d_w_head, and read the first N rows of the per-token inputs), then devices and dtypes.
    """
    if w_head.dim() != 2:
        raise ValueError("w_head must be [V, d]")
    V, d = w_head.shape
    if N < 0:
        raise ValueError("N must be >= 0")
    if N > 0:
        if hidden.dim() != 2 or hidden.shape[1] != d:
            raise ValueError("hidden and w_head disagree on d")
        for name, t in (("hidden", hidden), ("target", target), ("logp_old", logp_old),
                        ("weight", weight), ("seq_id", seq_id)):
            if t.shape[0] < N:
                raise ValueError(f"{name} has fewer than N rows")
    if d_w_head is not None and tuple(d_w_head.shape) != (V, d):
        raise ValueError(f"d_w_head must be [V, d] = [{V}, {d}], got {list(d_w_head.shape)}")
    if d_hidden is not None and (d_hidden.dim() != 2 or d_hidden.shape[1] != d or d_hidden.shape[0] < N):
        raise ValueError(f"d_hidden must be [>= N, d] = [>= {N}, {d}], got {list(d_hidden.shape)}")
    _dev(w_head, torch.bfloat16, "w_head")
    dev = w_head.device
    _dev(advantage, torch.float32, "advantage")
    if N > 0:
        _dev(hidden, torch.bfloat16, "hidden")
        _dev(target, torch.int32, "target")
        _dev(logp_old, torch.float32, "logp_old")
        _dev(weight, torch.float32, "weight")
        _dev(seq_id, torch.int32, "seq_id")
    if d_w_head is None:
        d_w_head = torch.empty((V, d), dtype=torch.float32, device=dev)
    _dev(d_w_head, torch.float32, "d_w_head")
    if d_hidden is None:
        d_hidden = torch.empty((max(N, 1), d), dtype=torch.float32, device=dev)
    _dev(d_hidden, torch.float32, "d_hidden")
    loss = torch.empty(1, dtype=torch.float64, device=dev)
    logp = torch.empty(max(N, 1), dtype=torch.float32, device=dev) if want_logp else None
    stats = torch.empty(5, dtype=torch.float64, device=dev) if want_stats else None
    need = loss_workspace_bytes(N, d, V, flags)
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=dev)
    _dev(workspace, torch.uint8, "workspace")
    if err_flag is not None:
        _dev(err_flag, torch.int32, "err_flag")
    _check(load().pspo_loss_fwd_bwd(
        _ptr(hidden) if N > 0 else None, _ptr(w_head), _ptr(target) if N > 0 else None,
        _ptr(logp_old) if N > 0 else None, _ptr(weight) if N > 0 else None,
        _ptr(seq_id) if N > 0 else None, _ptr(advantage), N, d, V, advantage.shape[0],
        float(eps_low), float(eps_high), float(loss_scale), flags,
        _ptr(loss), _ptr(d_hidden), _ptr(d_w_head), _ptr(logp), _ptr(stats), _ptr(err_flag),
        _ptr(workspace), workspace.numel(), _stream()))
    return dict(loss=loss, d_hidden=d_hidden[:N], d_w_head=d_w_head,
                logp_new=None if logp is None else logp[:N], stats=stats, workspace=workspace)


def score_proxy_workspace_bytes(N: int, d: int, V: int) -> int:
    return int(load().pspo_score_proxy_workspace_bytes(N, d, V))


def score_proxy(hidden, w_head, target, N: int, want_logp: bool = True, want_p_sq: bool = False,
                workspace: Optional[torch.Tensor] = None, err_flag: Optional[torch.Tensor] = None) -> dict:
    """Output-head score proxy gamma (and optionally log p(o), ||p||^2) of the first N rows."""
    _dev(w_head, torch.bfloat16, "w_head")
    V, d = w_head.shape
    dev = w_head.device
    if N > 0:
        _dev(hidden, torch.bfloat16, "hidden")
        _dev(target, torch.int32, "target")
        if hidden.shape[1] != d:
            raise ValueError("hidden and w_head disagree on d")
        if hidden.shape[0] < N or target.shape[0] < N:
            raise ValueError("hidden or target has fewer than N rows")
    gamma = torch.empty(max(N, 1), dtype=torch.float32, device=dev)
    logp = torch.empty(max(N, 1), dtype=torch.float32, device=dev) if want_logp else None
    p_sq = torch.empty(max(N, 1), dtype=torch.float32, device=dev) if want_p_sq else None
    need = score_proxy_workspace_bytes(N, d, V)
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=dev)
    _dev(workspace, torch.uint8, "workspace")
    if err_flag is not None:
        _dev(err_flag, torch.int32, "err_flag")
    _check(load().pspo_score_proxy(
        _ptr(hidden) if N > 0 else None, _ptr(w_head), _ptr(target) if N > 0 else None, N, d, V,
        _ptr(gamma), _ptr(logp), _ptr(p_sq), _ptr(err_flag), _ptr(workspace), workspace.numel(), _stream()))
    return dict(gamma=gamma[:N], logp=None if logp is None else logp[:N],
                p_sq=None if p_sq is None else p_sq[:N], workspace=workspace)


PSPO_DESIGN_OPTIMIZED, PSPO_DESIGN_HEURISTIC, PSPO_DESIGN_UNIFORM, PSPO_DESIGN_TIME_PRIOR = 0, 1, 2, 3


def design_weights(gamma, topk_ids, topk_logp, lengths, full_off, rewards, xi_off, P: int, K: int,
                   total_T: int, want_parts: bool = False, err_flag: Optional[torch.Tensor] = None) -> dict:
    """Per-step weights w_t = gbar_t u_t of the cutoff design (float64, xi_off layout)."""
    _dev(gamma, torch.float32, "gamma")
    _dev(topk_ids, torch.int32, "topk_ids")
    _dev(topk_logp, torch.float32, "topk_logp")
    _dev(lengths, torch.int32, "lengths")
    _dev(full_off, torch.int32, "full_off")
    _dev(rewards, torch.float32, "rewards")
    _dev(xi_off, torch.int64, "xi_off")
    if topk_ids.dim() != 2 or topk_ids.shape != topk_logp.shape:
        raise ValueError("topk_ids and topk_logp must be [S, k] of the same shape")
    dev = gamma.device
    w = torch.empty(max(total_T, 1), dtype=torch.float64, device=dev)
    gb = torch.empty_like(w) if want_parts else None
    u = torch.empty_like(w) if want_parts else None
    if err_flag is not None:
        _dev(err_flag, torch.int32, "err_flag")
    _check(load().pspo_design_weights(_ptr(gamma), _ptr(topk_ids), _ptr(topk_logp), topk_ids.shape[1],
                                      _ptr(lengths), _ptr(full_off), _ptr(rewards), _ptr(xi_off), P, K,
                                      total_T, _ptr(w), _ptr(gb), _ptr(u), _ptr(err_flag), _stream()))
    return dict(w=w[:total_T], gamma_bar=None if gb is None else gb[:total_T], u=None if u is None else u[:total_T])


def design_cutoffs(w, xi_off, P: int, total_T: int, budget: float, variant: int = PSPO_DESIGN_OPTIMIZED,
                   lam: float = 0.0, out: Optional[torch.Tensor] = None,
                   err_flag: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Survival tables xi (float64, xi_off layout) minimising sum w/xi under the budget."""
    _dev(w, torch.float64, "w")
    _dev(xi_off, torch.int64, "xi_off")
    dev = w.device
    xi = out if out is not None else torch.empty(max(total_T, 1), dtype=torch.float64, device=dev)
    _dev(xi, torch.float64, "xi")
    ws = torch.empty(max(int(load().pspo_design_workspace_bytes(total_T)), 256), dtype=torch.uint8, device=dev)
    if err_flag is not None:
        _dev(err_flag, torch.int32, "err_flag")
    _check(load().pspo_design_cutoffs(_ptr(w), _ptr(xi_off), P, total_T, float(budget), int(variant), float(lam),
                                      _ptr(xi), _ptr(ws), ws.numel(), _ptr(err_flag), _stream()))
    return xi[:total_T]


def design_cutoffs_noalloc(w, xi_off, P: int, total_T: int, budget: float, out: torch.Tensor,
                           variant: int = PSPO_DESIGN_OPTIMIZED, lam: float = 0.0,
                           err_flag: Optional[torch.Tensor] = None) -> torch.Tensor:
    """design_cutoffs without a workspace (the library's static scratch; total_T <= 2^19):
    writes `out` (float64 [>= total_T], caller-allocated) and allocates nothing."""
    _dev(w, torch.float64, "w")
    _dev(xi_off, torch.int64, "xi_off")
    _dev(out, torch.float64, "out")
    if out.numel() < total_T:
        raise ValueError("out needs total_T entries")
    if err_flag is not None:
        _dev(err_flag, torch.int32, "err_flag")
    _check(load().pspo_design_cutoffs_noalloc(_ptr(w), _ptr(xi_off), P, total_T, float(budget), int(variant),
                                              float(lam), _ptr(out), _ptr(err_flag), _stream()))
    return out[:total_T]


def mfma_loop(iters: int, blocks: int, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Enqueues the matrix-core rate probe (blocks * 4 * iters * 16 * 16384 bf16 flops) on the
    current stream; the caller times it."""
    if out is None:
        out = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")
    _dev(out, torch.float32, "out")
    if out.numel() < blocks * 256:
        raise ValueError("out needs blocks * 256 floats")
    _check(load().pspo_mfma_loop(int(iters), int(blocks), _ptr(out), _stream()))
    return out


TIMED_KINDS = ("forward", "logit_grad", "dw", "dh", "proxy")   # PSPO_TIME_* order


def timing_start(max_records: int) -> None:
    """Per-product timing of the loss and score-proxy calls made on this thread (HIP events
    on each call's stream around each matrix-core product), until timing_stop()."""
    _check(load().pspo_timing_start(int(max_records)))


def timing_stop() -> dict:
    """Waits for the recorded events; per product kind (TIMED_KINDS): summed ms and record count."""
    ms = (ctypes.c_double * len(TIMED_KINDS))()
    cnt = (ctypes.c_int32 * len(TIMED_KINDS))()
    _check(load().pspo_timing_stop(ctypes.cast(ms, _P), ctypes.cast(cnt, _P)))
    return {k: {"ms": float(ms[i]), "count": int(cnt[i])} for i, k in enumerate(TIMED_KINDS)}
