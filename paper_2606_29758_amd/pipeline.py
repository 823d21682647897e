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
    """Reusable buffers for repeated passes over one DeviceWorkload."""

    def __init__(self, dw: DeviceWorkload):
        self.dw = dw
        dev = dw.lengths.device
        self.cutoffs = torch.empty(dw.P * dw.K, dtype=torch.int32, device=dev)
        self.err = torch.zeros(1, dtype=torch.int32, device=dev)
        self.d_w = torch.empty((dw.V, dw.d), dtype=torch.float32, device=dev)
        self.d_h = torch.empty((max(dw.capacity, 1), dw.d), dtype=torch.float32, device=dev)
        self.workspace = torch.empty(max(pspo.loss_workspace_bytes(dw.capacity, dw.d, dw.V), 256),
                                     dtype=torch.uint8, device=dev)

    def sample_and_pack(self, seed: int, offset: int = 0) -> dict:
        dw = self.dw
        pspo.sample_cutoffs(dw.xi, dw.xi_off, dw.lengths, dw.P, dw.K, seed, offset,
                            out=self.cutoffs, err_flag=self.err)
        return pspo.pack_prefixes(self.cutoffs, dw.lengths, dw.xi, dw.xi_off, dw.P, dw.K, dw.capacity,
                                  target_full=dw.target_full, logp_old_full=dw.logp_old_full,
                                  hidden_full=dw.hidden_full, err_flag=self.err)

    def loss(self, pk: dict, N: int, flags: int = 0, want_logp: bool = True) -> dict:
        """want_logp=False: no per-token log-probs, and the forward skips the tokens of
        zero-advantage completions (their loss terms and gradients are exactly zero)."""
        dw = self.dw
        return pspo.loss_fwd_bwd(pk["hidden"], dw.w_head, pk["target"], pk["logp_old"], pk["weight"],
                                 pk["seq_id"], dw.advantage, N, dw.eps_low, dw.eps_high, dw.loss_scale,
                                 flags=flags, d_w_head=self.d_w, d_hidden=self.d_h,
                                 workspace=self.workspace, err_flag=self.err, want_logp=want_logp)

    def __call__(self, seed: int, offset: int = 0, flags: int = 0, want_logp: bool = True) -> dict:
        pk = self.sample_and_pack(seed, offset)
        N = int(pk["n_tokens"].item())   # the one host sync of a step
        out = self.loss(pk, N, flags, want_logp)
        out["pack"] = pk
        out["N"] = N
        out["cutoffs"] = self.cutoffs
        return out
