"""One pass of the hot path on the GPU: sample cutoffs -> pack prefixes -> loss fwd+bwd.

Orchestration of the three libpspo calls on device-resident inputs (the
workload tensors are uploaded once).  The only host synchronisation inside a
step is the 4-byte read of the packed token count, which sizes the loss call.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np
import torch

from . import pspo


@dataclasses.dataclass
class DeviceWorkload:
    P: int
    K: int
    d: int
    V: int
    capacity: int
    xi: torch.Tensor
    xi_off: torch.Tensor
    lengths: torch.Tensor
    advantage: torch.Tensor
    target_full: torch.Tensor
    logp_old_full: torch.Tensor
    hidden_full: torch.Tensor
    w_head: torch.Tensor
    eps_low: float
    eps_high: float
    loss_scale: float


def upload(wl, logp_old_full: np.ndarray, device="cuda") -> DeviceWorkload:
    """Copies a synth.Workload (with its matrices) and its old log-probs to the device."""
    cfg = wl.cfg
    t = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a)).to(device=device, dtype=dt)
    hidden = torch.from_numpy(wl.hidden_bits.view(np.int16)).to(device).view(torch.bfloat16)
    w = torch.from_numpy(wl.w_bits.view(np.int16)).to(device).view(torch.bfloat16)
    return DeviceWorkload(
        P=cfg.P, K=cfg.K, d=cfg.d, V=cfg.V, capacity=int(wl.total_tokens),
        xi=t(wl.xi, torch.float64), xi_off=t(wl.xi_off, torch.int64), lengths=t(wl.lengths, torch.int32),
        advantage=t(wl.advantage, torch.float32), target_full=t(wl.target_full, torch.int32),
        logp_old_full=t(np.asarray(logp_old_full, dtype=np.float32), torch.float32),
        hidden_full=hidden, w_head=w, eps_low=cfg.eps_low, eps_high=cfg.eps_high, loss_scale=cfg.loss_scale)


class Step:
    """Reusable buffers for repeated passes over one DeviceWorkload.

    The loss workspace and the d_hidden buffer are sized by the packed token
    count N of the calls made so far (grown when a call needs more), not by the
    batch's total token count: a truncated step needs only its prefixes' share.
    """

    def __init__(self, dw: DeviceWorkload, flags: int = 0):
        self.dw = dw
        self.flags = flags
        dev = dw.lengths.device
        self.cutoffs = torch.empty(dw.P * dw.K, dtype=torch.int32, device=dev)
        self.err = torch.zeros(1, dtype=torch.int32, device=dev)
        self.d_w = torch.empty((dw.V, dw.d), dtype=torch.float32, device=dev)
        self.d_h = torch.empty((0, dw.d), dtype=torch.float32, device=dev)
        self.workspace = torch.empty(0, dtype=torch.uint8, device=dev)

    def reserve(self, N: int, flags: int = 0) -> None:
        """Grows the d_hidden buffer and the workspace to what a call over N tokens needs."""
        dw = self.dw
        dev = dw.lengths.device
        if self.d_h.shape[0] < max(N, 1):
            self.d_h = None
            self.d_h = torch.empty((max(N, 1), dw.d), dtype=torch.float32, device=dev)
        need = max(pspo.loss_workspace_bytes(N, dw.d, dw.V, flags), 256)
        if self.workspace.numel() < need:
            self.workspace = None
            self.workspace = torch.empty(need, dtype=torch.uint8, device=dev)

    def sample_and_pack(self, seed: int, offset: int = 0) -> dict:
        dw = self.dw
        pspo.sample_cutoffs(dw.xi, dw.xi_off, dw.lengths, dw.P, dw.K, seed, offset,
                            out=self.cutoffs, err_flag=self.err)
        return pspo.pack_prefixes(self.cutoffs, dw.lengths, dw.xi, dw.xi_off, dw.P, dw.K, dw.capacity,
                                  target_full=dw.target_full, logp_old_full=dw.logp_old_full,
                                  hidden_full=dw.hidden_full, err_flag=self.err)

    def loss(self, pk: dict, N: int, flags: Optional[int] = None, want_logp: bool = True) -> dict:
        """want_logp=False: no per-token log-probs, and the forward skips the tokens of
        zero-advantage completions (their loss terms and gradients are exactly zero).
        flags: the library's loss flags (default: the Step's)."""
        dw = self.dw
        flags = self.flags if flags is None else flags
        self.reserve(N, flags)
        return pspo.loss_fwd_bwd(pk["hidden"], dw.w_head, pk["target"], pk["logp_old"], pk["weight"],
                                 pk["seq_id"], dw.advantage, N, dw.eps_low, dw.eps_high, dw.loss_scale,
                                 flags=flags, d_w_head=self.d_w, d_hidden=self.d_h,
                                 workspace=self.workspace, err_flag=self.err, want_logp=want_logp)

    def __call__(self, seed: int, offset: int = 0, flags: Optional[int] = None, want_logp: bool = True) -> dict:
        pk = self.sample_and_pack(seed, offset)
        N = int(pk["n_tokens"].item())   # the one host sync of a step
        out = self.loss(pk, N, flags, want_logp)
        out["pack"] = pk
        out["N"] = N
        out["cutoffs"] = self.cutoffs
        return out


def reseed_mean(step: "Step", seeds, want_logp: bool = False) -> dict:
    """Mean of the truncated update over cutoff draws, and the full-trajectory calls it is checked against.

    PS-PPO's truncated estimate (Sec. 3.2; App. B) is linear in the keep
    indicators: the clip mask depends on the ratio only, never on the cutoff.
    So the mean over S seeds of the loss, dW and dH (dH rows accumulated at
    their full-trajectory positions) equals one call over every completion
    token with weight n_t c_t / S, where c_t is the token's cutoff weight and
    n_t the number of seeds that kept it.  That identity holds up to rounding.
    A call with every weight 1 gives the full update G that the estimator is
    unbiased for; the distance of the S-draw mean from it is a sample of the
    estimator's noise (App. C).

    Returns float64 host scalars and device tensors: mean_loss, weighted_loss, full_loss,
    mean_dw, weighted_dw, full_dw, mean_dh, weighted_dh, full_dh (dH rows in full order),
    kept (n_t, int32), weight_full (c_t), logp_full (log-probs of the full call, if asked),
    tokens.
    """
    dw = step.dw
    seeds = list(seeds)
    S = len(seeds)
    if S == 0:
        raise ValueError("need at least one seed")
    dev = dw.lengths.device
    total = dw.capacity
    acc_dw = torch.zeros((dw.V, dw.d), dtype=torch.float32, device=dev)
    acc_dh = torch.zeros((max(total, 1), dw.d), dtype=torch.float32, device=dev)
    kept = torch.zeros(max(total, 1), dtype=torch.int32, device=dev)
    loss_sum = 0.0
    for i, s in enumerate(seeds):
        pk = step.sample_and_pack(s)
        N = int(pk["n_tokens"].item())
        out = step.loss(pk, N, flags=step.flags | (pspo.PSPO_ACCUMULATE_DW if i > 0 else 0), want_logp=False)
        loss_sum += float(out["loss"].item())
        if N > 0:
            src = pk["src_row"][:N].long()
            acc_dh.index_add_(0, src, out["d_hidden"])
            kept.index_add_(0, src, torch.ones(N, dtype=torch.int32, device=dev))
    acc_dw.copy_(step.d_w)   # the accumulated sum over the S draws
    # every token of every completion: cutoffs at the lengths; c_t is the weight the packer gives it
    full_cut = dw.lengths.clone()
    pk = pspo.pack_prefixes(full_cut, dw.lengths, dw.xi, dw.xi_off, dw.P, dw.K, total,
                            target_full=dw.target_full, logp_old_full=dw.logp_old_full,
                            hidden_full=dw.hidden_full, err_flag=step.err)
    c_full = pk["weight"][:total].clone()

    def call(weight):
        pk["weight"][:total] = weight
        out = step.loss(pk, total, want_logp=want_logp)
        return (float(out["loss"].item()), step.d_w.clone(), out["d_hidden"][:total].clone(),
                None if out["logp_new"] is None else out["logp_new"][:total].clone())

    wl, wdw, wdh, _ = call(c_full * kept[:total].to(torch.float32) / S)
    fl, fdw, fdh, flp = call(torch.ones_like(c_full))
    return dict(mean_loss=loss_sum / S, weighted_loss=wl, full_loss=fl,
                mean_dw=acc_dw / S, weighted_dw=wdw, full_dw=fdw,
                mean_dh=acc_dh[:total] / S, weighted_dh=wdh, full_dh=fdh,
                kept=kept[:total], weight_full=c_full, logp_full=flp, tokens=total, seeds=S)
