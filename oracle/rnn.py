"""CPU oracle for the while-loop with an Elman RNN body, and its gradient loop.

TEST INFRASTRUCTURE ONLY, like the LSTM oracle beside it: only the
test-suite, the smoke check and the benchmark's CPU-baseline leg may import
it, and it shares no code with the HIP library.

The loop construct is the one of the LSTM oracle (Sections 4.2, 5.1, 5.2 of
Dynamic Control Flow in Large-Scale Machine Learning): predicate
``t < max_b seq_len[b]``, a stack pushed by the forward loop and popped in
reverse by the gradient loop, gradients of loop constants summed over
iterations, the gradient of reading x_t a write of dx_t.  Only the body
differs: the Elman recurrence

    h_t = tanh([x_t, h_{t-1}] W + b),   W [I+H, H], b [H]

(rows 0..I-1 of W multiply x_t, rows I.. multiply h_{t-1}).  Rows whose
sequence has ended keep h and output 0.  The gradient of one step:
dz = (dh + dy_t) * (1 - h_t^2); dh_{t-1} = dz W_h^T; dx_t = dz W_x^T;
dW += [x_t, h_{t-1}]^T dz; db += sum over rows of dz.

Precision modes as in the LSTM oracle: "fp64"; "bf16" (float64 arithmetic,
bfloat16 rounding of h_{t-1} before the recurrent product and of dz before
the products that give dx, dh_{t-1} and dW; db sums unrounded dz); "fp32"
(CPU timing only).
"""
from __future__ import annotations

import numpy as np

from .lstm import bf16_round

__all__ = ["rnn_forward_literal", "rnn_forward", "rnn_backward",
           "stacked_rnn_forward", "stacked_rnn_backward"]


def _dtype(precision):
    if precision not in ("fp64", "fp32", "bf16"):
        raise ValueError(f"unknown precision {precision!r}")
    return np.float32 if precision == "fp32" else np.float64


def _operand(v, precision):
    return bf16_round(v) if precision == "bf16" else v


def rnn_forward_literal(x, seq_len, W, bias, h0=None):
    """float64, one sequence at a time: the plain definition of the result.
    Returns y [T_max,B,H] (0 at t >= seq_len[b]) and hT [B,H]."""
    x = np.asarray(x, np.float64)
    W = np.asarray(W, np.float64)
    bias = np.asarray(bias, np.float64)
    T_max, B, I = x.shape
    H = W.shape[1]
    y = np.zeros((T_max, B, H))
    hT = np.zeros((B, H))
    for b in range(B):
        h = np.zeros(H) if h0 is None else np.array(h0[b], np.float64)
        for t in range(int(seq_len[b])):
            h = np.tanh(np.concatenate([x[t, b], h]) @ W + bias)
            y[t, b] = h
        hT[b] = h
    return y, hT


def rnn_forward(x, seq_len, W, bias, h0=None, precision="fp64"):
    """Forward while-loop over the batch with a validity mask.
    Returns (y, hT, tape); the tape is the stack of pushed values."""
    dt = _dtype(precision)
    seq_len = np.asarray(seq_len, np.int64)
    x = np.asarray(x, dt)
    W = np.asarray(W, dt)
    bias = np.asarray(bias, dt)
    T_max, B, I = x.shape
    H = W.shape[1]
    if W.shape[0] != I + H:
        raise ValueError("W must have I+H rows")
    if (seq_len < 0).any() or (seq_len > T_max).any():
        raise ValueError("seq_len outside [0, T_max]")
    Wx, Wh = W[:I], W[I:]
    h = np.zeros((B, H), dt) if h0 is None else np.array(h0, dt)
    y = np.zeros((T_max, B, H), dt)
    T_eff = int(seq_len.max()) if B else 0
    stack = []
    t = 0
    while t < T_eff:
        valid = (t < seq_len)[:, None]
        h_op = _operand(h, precision)
        h_new = np.tanh(x[t] @ Wx + h_op @ Wh + bias)
        stack.append(dict(h=h_new, h_op=h_op, valid=valid))
        h = np.where(valid, h_new, h)
        y[t] = np.where(valid, h_new, 0.0)
        t += 1
    tape = dict(stack=stack, T_eff=T_eff, x=x, W=W, precision=precision, I=I, H=H)
    return y, h, tape


def rnn_backward(tape, dy=None, dhT=None):
    """Gradient while-loop: the forward's trip count, in reverse.
    Returns dict(dx, dW [I+H,H], dbias [H], dh0 [B,H])."""
    precision = tape["precision"]
    dt = _dtype(precision)
    x, W = tape["x"], tape["W"]
    I, H = tape["I"], tape["H"]
    T_max, B, _ = x.shape
    Wx, Wh = W[:I], W[I:]
    dh = np.zeros((B, H), dt) if dhT is None else np.array(dhT, dt)
    dx = np.zeros((T_max, B, I), dt)
    dWx = np.zeros_like(Wx)
    dWh = np.zeros_like(Wh)
    db = np.zeros(H, dt)
    stack = list(tape["stack"])
    t = tape["T_eff"]
    while t > 0:
        t -= 1
        s = stack.pop()
        valid = s["valid"]
        dh_tot = dh + (np.where(valid, np.asarray(dy[t], dt), 0.0) if dy is not None else 0.0)
        dz = np.where(valid, dh_tot * (1.0 - s["h"] * s["h"]), 0.0)
        dz_op = _operand(dz, precision)
        x_t = np.where(valid, x[t], 0.0)
        dx[t] = dz_op @ Wx.T
        dWx += x_t.T @ dz_op
        dWh += s["h_op"].T @ dz_op
        db += dz.sum(axis=0)
        dh = np.where(valid, dz_op @ Wh.T, dh)
    assert not stack
    return dict(dx=dx, dW=np.concatenate([dWx, dWh], axis=0), dbias=db, dh0=dh)


def stacked_rnn_forward(x, seq_len, Ws, biases, h0=None, precision="fp64"):
    """L layers; layer l+1 reads layer l's y (bfloat16-rounded in "bf16")."""
    tapes, hTs = [], []
    inp = x
    y = None
    for l, (Wl, bl) in enumerate(zip(Ws, biases)):
        y, hT, tape = rnn_forward(inp, seq_len, Wl, bl, None if h0 is None else h0[l], precision)
        tapes.append(tape)
        hTs.append(hT)
        inp = _operand(y, precision)
    return y, np.stack(hTs), tapes


def stacked_rnn_backward(tapes, dy=None, dhT=None):
    L = len(tapes)
    g_out = dy
    dWs, dbs, dh0s = [None] * L, [None] * L, [None] * L
    for l in reversed(range(L)):
        r = rnn_backward(tapes[l], g_out, None if dhT is None else dhT[l])
        dWs[l], dbs[l], dh0s[l] = r["dW"], r["dbias"], r["dh0"]
        g_out = r["dx"]
    return dict(dx=g_out, dW=dWs, dbias=dbs, dh0=np.stack(dh0s))
