"""Seeded synthetic inputs for the device-side LSTM while-loop.

This module only draws random numbers and lays them out; it contains none of
the loop's arithmetic, so both the CPU oracle and the HIP path can be fed from
it without sharing code.  Every array is produced host-side in float32 with
``numpy.random.default_rng(seed)`` in a fixed draw order:
``seq_len, x, W, bias, dy, h0, c0``.

The five named workloads follow the shapes the paper evaluates (Section 6.2:
one-layer LSTM with 512 units; Section 6.3: sequence length 200, and 2048
units at batch 256), all with synthetic data.  bfloat16 workloads store x and
W rounded to bfloat16 (round to nearest even), so the same float32 values can
be passed to the oracle and, bit-exactly, as bfloat16 tensors to the GPU.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Optional

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    I: int
    H: int
    T_max: int
    dtype: str                 # "f32" or "bf16": storage type of x and W
    len_lo: int                # seq_len ~ U{len_lo .. len_hi}
    len_hi: int
    layers: int = 1
    w_scale: Optional[float] = None   # U(-s, s) for W and bias; None = 1/sqrt(H)
    force_zero_len: bool = False      # make sure one sequence has length 0
    with_dy: bool = True              # dy ~ N(0,1); False -> no per-step gradient
    random_state: bool = False        # h0, c0 ~ N(0, 0.5^2) instead of zeros
    spill: bool = False
    seed: int = 0
    cell: str = "lstm"                # "lstm" (4 gate blocks), "gru" (3), "rnn" (Elman, 1),
                                      # "skip" (the LSTM body with a cond), "act" (the
                                      # LSTM body with a nested loop)
    ponder_max: int = 4               # "act": at most this many ponder steps per step
    extra: dict = field(default_factory=dict)

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)

    @property
    def gates(self) -> int:
        return {"lstm": 4, "gru": 3, "rnn": 1, "skip": 4, "act": 4}[self.cell]

    def bias_len(self, layer: int = 0) -> int:
        """Bias entries of a layer: G*H, the GRU's extra b_hn block, the cond
        body's predicate weights over [x_t, h_{t-1}] and its offset."""
        if self.cell == "gru":
            return 4 * self.H
        if self.cell == "skip":
            return 4 * self.H + (self.I if layer == 0 else self.H) + self.H + 1
        if self.cell == "act":
            return 5 * self.H + 1
        return self.gates * self.H


# The five workloads.  Seeds are 1000 + index.
TINY = Workload("lstm_tiny_b4_h32_t16_f32", B=4, I=32, H=32, T_max=16, dtype="f32",
                len_lo=0, len_hi=16, w_scale=0.1, force_zero_len=True,
                with_dy=False, seed=1001)
FIXED_H512 = Workload("lstm_b64_h512_t100_f32", B=64, I=512, H=512, T_max=100,
                      dtype="f32", len_lo=100, len_hi=100, seed=1002)
VAR_H1024 = Workload("lstm_b128_h1024_tmax200_varlen_bf16", B=128, I=1024, H=1024,
                     T_max=200, dtype="bf16", len_lo=20, len_hi=200, seed=1003)
LONG_SPILL = Workload("lstm_b64_h512_t2000_f32_spill", B=64, I=512, H=512, T_max=2000,
                      dtype="f32", len_lo=2000, len_hi=2000, spill=True, seed=1004)
TWO_LAYER = Workload("lstm2_b256_h2048_tmax128_varlen_bf16", B=256, I=2048, H=2048,
                     T_max=128, dtype="bf16", len_lo=64, len_hi=128, layers=2,
                     seed=1005)

# The same loop with the Elman RNN body (the loop engine is not tied to one
# cell), at the H = 1024 variable-length shape.
RNN_VAR_H1024 = Workload("rnn_b128_h1024_tmax200_varlen_bf16", B=128, I=1024, H=1024,
                         T_max=200, dtype="bf16", len_lo=20, len_hi=200, cell="rnn",
                         seed=1006)

# ... and with the GRU body.
GRU_VAR_H1024 = Workload("gru_b128_h1024_tmax200_varlen_bf16", B=128, I=1024, H=1024,
                         T_max=200, dtype="bf16", len_lo=20, len_hi=200, cell="gru",
                         seed=1007)

# ... and with the LSTM body holding a data-dependent cond (a row runs the
# step or keeps its state; the predicate weights are drawn with the bias).
SKIP_VAR_H1024 = Workload("skip_b128_h1024_tmax200_varlen_bf16", B=128, I=1024, H=1024,
                          T_max=200, dtype="bf16", len_lo=20, len_hi=200, cell="skip",
                          seed=1008)

# ... and with the LSTM body holding a nested loop (ACT's halting rule: each
# input pondered 1 to 4 times; the halting weights are drawn with the bias).
ACT_VAR_H1024 = Workload("act_b128_h1024_tmax200_varlen_bf16", B=128, I=1024, H=1024,
                         T_max=200, dtype="bf16", len_lo=20, len_hi=200, cell="act",
                         ponder_max=4, seed=1009)

ALL = (TINY, FIXED_H512, VAR_H1024, LONG_SPILL, TWO_LAYER, RNN_VAR_H1024, GRU_VAR_H1024,
       SKIP_VAR_H1024, ACT_VAR_H1024)
BY_NAME = {w.name: w for w in ALL}


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even), returned as
    float32.  Used only to prepare bfloat16-representable inputs."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) & 0xFFFF0000).astype(np.uint32)
    out = r.view(np.float32).copy()
    nan = np.isnan(a)
    out[nan] = np.nan
    return out


def generate(w: Workload, seed: Optional[int] = None, nan_padding: bool = False):
    """Draw the inputs of workload ``w``.

    Returns a dict of float32 / int32 numpy arrays:
      seq_len [B] int32, x [T_max,B,I], W [layers][I_l+H,G*H], bias [layers][bias_len(l)],
      dy [T_max,B,H] or None, h0/c0 [layers,B,H], dhT [layers,B,H] (ones on
      the top layer), dcT [layers,B,H] (zeros).
    With ``nan_padding`` the x entries at t >= seq_len[b] are NaN.
    """
    rng = np.random.default_rng(w.seed if seed is None else seed)
    B, I, H, T = w.B, w.I, w.H, w.T_max
    seq_len = rng.integers(w.len_lo, w.len_hi + 1, size=B).astype(np.int32)
    if w.force_zero_len and not (seq_len == 0).any():
        seq_len[int(rng.integers(0, B))] = 0
    x = rng.standard_normal((T, B, I), dtype=np.float32)
    s = w.w_scale if w.w_scale is not None else 1.0 / np.sqrt(H)
    Ws, biases = [], []
    G = w.gates
    for l in range(w.layers):
        in_w = I if l == 0 else H
        Ws.append(rng.uniform(-s, s, size=(in_w + H, G * H)).astype(np.float32))
        biases.append(rng.uniform(-s, s, size=(w.bias_len(l),)).astype(np.float32))
    dy = rng.standard_normal((T, B, H), dtype=np.float32) if w.with_dy else None
    if w.random_state:
        h0 = (0.5 * rng.standard_normal((w.layers, B, H))).astype(np.float32)
        c0 = (0.5 * rng.standard_normal((w.layers, B, H))).astype(np.float32)
    else:
        h0 = np.zeros((w.layers, B, H), np.float32)
        c0 = np.zeros((w.layers, B, H), np.float32)
    if w.dtype == "bf16":
        x = round_to_bf16(x)
        Ws = [round_to_bf16(Wl) for Wl in Ws]
    if nan_padding:
        t_idx = np.arange(T)[:, None]
        x[t_idx >= seq_len[None, :]] = np.nan
    dhT = np.zeros((w.layers, B, H), np.float32)
    dhT[-1] = 1.0
    dcT = np.zeros((w.layers, B, H), np.float32)
    return dict(seq_len=seq_len, x=x, W=Ws, bias=biases, dy=dy, h0=h0, c0=c0,
                dhT=dhT, dcT=dcT)


def algorithmic_flops(w: Workload, seq_len: np.ndarray) -> float:
    """Forward + backward flops the method needs: 6*G*H*(I_l+H) per valid
    (timestep, sequence) per layer (G = 4 gate blocks for the LSTM, 3 for
    the GRU, 1 for the RNN: one product forward, three backward); masked
    steps and padding excluded."""
    n = float(np.asarray(seq_len, dtype=np.int64).sum())
    tot = 0.0
    for l in range(w.layers):
        in_w = w.I if l == 0 else w.H
        tot += 6.0 * w.gates * w.H * (in_w + w.H) * n
    return tot
