"""Device buffers for one workload and the fwd + bwd call sequence.

Allocation and marshalling only: inputs drawn by ``workloads.generate`` are
copied to the GPU (bfloat16 workloads as torch.bfloat16, which is exact for
their bfloat16-representable values), outputs are allocated, and the two
C-ABI entry points are called on the current torch stream.
"""
from __future__ import annotations

from typing import Optional

import numpy as np
import torch

from .lstmloop import LL_CELL_GRU, LL_CELL_LSTM, LL_CELL_LSTM_ACT, LL_CELL_LSTM_SKIP, LL_CELL_RNN, Plan


class DeviceCase:
    def __init__(self, inputs: dict, H: int, I: int, layers: int, dtype: str,
                 device: str = "cuda:0", cell: str = "lstm", ponder_max: int = 0):
        dev = torch.device(device)
        self.dev = dev
        self.dtype = dtype
        self.cell = cell
        self.ponder_max = ponder_max
        op = torch.bfloat16 if dtype == "bf16" else torch.float32
        f32 = torch.float32
        T, B, _ = inputs["x"].shape
        self.T, self.B, self.I, self.H, self.L = T, B, I, H, layers

        def t(a, dt=f32):
            return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(dev, dt)

        self.x = t(inputs["x"], op)
        self.seq_len = t(inputs["seq_len"], torch.int32)
        self.W = [t(w, op) for w in inputs["W"]]
        self.bias = [t(b) for b in inputs["bias"]]
        self.h0 = t(inputs.get("h0"))
        self.c0 = t(inputs.get("c0"))
        self.dy = t(inputs.get("dy"))
        self.dhT = t(inputs.get("dhT"))
        self.dcT = t(inputs.get("dcT"))
        L = layers
        z = lambda *shape: torch.empty(*shape, device=dev, dtype=f32)
        self.y = z(T, B, H)
        self.hT = z(L, B, H)
        self.cT = z(L, B, H)
        self.trip = torch.empty(1, device=dev, dtype=torch.int32)
        self.dx = z(T, B, I)
        self.dW = [z(w.shape[0], w.shape[1]) for w in self.W]
        self.dbias = [z(b.shape[0]) for b in self.bias]
        self.dh0 = z(L, B, H)
        self.dc0 = z(L, B, H)

    def plan(self, **kw) -> Plan:
        cell = {"lstm": LL_CELL_LSTM, "rnn": LL_CELL_RNN, "gru": LL_CELL_GRU,
                "skip": LL_CELL_LSTM_SKIP, "act": LL_CELL_LSTM_ACT}[self.cell]
        return Plan(self.T, self.B, self.I, self.H, layers=self.L, dtype=self.dtype, cell=cell,
                    ponder_max=self.ponder_max if self.cell == "act" else 0, **kw)

    def fwd(self, plan: Plan, save: bool = True, use_h0: bool = True) -> None:
        plan.fwd(self.x, self.seq_len, self.W, self.bias,
                 self.h0 if use_h0 else None, self.c0 if use_h0 else None,
                 self.y, self.hT, self.cT, self.trip, save_for_backward=save)

    def bwd(self, plan: Plan, with_dy: bool = True) -> None:
        plan.bwd(self.x, self.seq_len, self.W, self.dy if with_dy else None, self.dhT,
                 self.dcT, self.dx, self.dW, self.dbias, self.dh0, self.dc0)

    def results(self) -> dict:
        torch.cuda.synchronize(self.dev)
        c = lambda a: a.detach().cpu().numpy().astype(np.float64)
        return dict(y=c(self.y), hT=c(self.hT), cT=c(self.cT), dx=c(self.dx),
                    dW=[c(w) for w in self.dW], dbias=[c(b) for b in self.dbias],
                    dh0=c(self.dh0), dc0=c(self.dc0), T_eff=int(self.trip.item()))
