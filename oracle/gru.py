"""CPU oracle for the while-loop with a GRU body, and its gradient loop.

TEST INFRASTRUCTURE ONLY, like the LSTM and RNN oracles beside it; it
shares no code with the HIP library.

The loop construct is the one of the LSTM oracle (Sections 4.2, 5.1, 5.2 of
Dynamic Control Flow in Large-Scale Machine Learning); only the body
differs.  The GRU with the reset gate applied after the recurrent product
(the form whose recurrent product can be computed at once for all gates):

    zx = x_t W_x + b_x           (gate blocks r, u, n; W [I+H, 3H], b_x [3H])
    zh = h_{t-1} W_h             (the same blocks)
    r = sigmoid(zx_r + zh_r),  u = sigmoid(zx_u + zh_u)
    n = tanh(zx_n + r * (zh_n + b_hn))                       (b_hn [H])
    h_t = (1 - u) * n + u * h_{t-1}

The bias argument is [4H] = [b_x (3H), b_hn (H)].  Rows whose sequence has
ended keep h and output 0.

Gradient of one step (dh_tot = dh + dy_t; a = pre-activations):
    da_u = dh_tot * (h_{t-1} - n) * u (1 - u)
    da_n = dh_tot * (1 - u) * (1 - n^2)
    da_r = da_n * (zh_n + b_hn) * r (1 - r)
    dzx = [da_r, da_u, da_n]           (input side: dx, dW_x, db_x)
    dzh = [da_r, da_u, da_n * r]       (recurrent side: dh, dW_h, db_hn)
    dh_{t-1} = dh_tot * u + dzh W_h^T
    dx_t = dzx W_x^T, dW_x += x_t^T dzx, dW_h += h_{t-1}^T dzh,
    db_x += sum dzx, db_hn += sum (da_n * r)

Precision modes as in the other oracles; in "bf16" the operands of the
products are rounded: h_{t-1} (forward and dW_h), dzx (dx, dW_x), dzh
(dh_{t-1}, dW_h); the bias sums use unrounded values.
"""
from __future__ import annotations

import numpy as np

from .lstm import bf16_round, sigmoid

__all__ = ["gru_forward_literal", "gru_forward", "gru_backward",
           "stacked_gru_forward", "stacked_gru_backward"]


def _dtype(precision):
    if precision not in ("fp64", "fp32", "bf16"):
        raise ValueError(f"unknown precision {precision!r}")
    return np.float32 if precision == "fp32" else np.float64


def _operand(v, precision):
    return bf16_round(v) if precision == "bf16" else v


def gru_forward_literal(x, seq_len, W, bias, h0=None):
    """float64, one sequence at a time.  Returns y [T_max,B,H], hT [B,H]."""
    x = np.asarray(x, np.float64)
    W = np.asarray(W, np.float64)
    bias = np.asarray(bias, np.float64)
    T_max, B, I = x.shape
    H = W.shape[1] // 3
    Wx, Wh = W[:I], W[I:]
    y = np.zeros((T_max, B, H))
    hT = np.zeros((B, H))
    for b in range(B):
        h = np.zeros(H) if h0 is None else np.array(h0[b], np.float64)
        for t in range(int(seq_len[b])):
            zx = x[t, b] @ Wx + bias[:3 * H]
            zh = h @ Wh
            r = sigmoid(zx[:H] + zh[:H])
            u = sigmoid(zx[H:2 * H] + zh[H:2 * H])
            n = np.tanh(zx[2 * H:] + r * (zh[2 * H:] + bias[3 * H:]))
            h = (1.0 - u) * n + u * h
            y[t, b] = h
        hT[b] = h
    return y, hT


def gru_forward(x, seq_len, W, bias, h0=None, precision="fp64"):
    """Forward while-loop over the batch.  Returns (y, hT, tape)."""
    dt = _dtype(precision)
    seq_len = np.asarray(seq_len, np.int64)
    x = np.asarray(x, dt)
    W = np.asarray(W, dt)
    bias = np.asarray(bias, dt)
    T_max, B, I = x.shape
    H = W.shape[1] // 3
    if W.shape[0] != I + H or bias.shape[0] != 4 * H:
        raise ValueError("W must be [I+H, 3H] and bias [4H]")
    if (seq_len < 0).any() or (seq_len > T_max).any():
        raise ValueError("seq_len outside [0, T_max]")
    Wx, Wh = W[:I], W[I:]
    bx, bhn = bias[:3 * H], bias[3 * H:]
    h = np.zeros((B, H), dt) if h0 is None else np.array(h0, dt)
    y = np.zeros((T_max, B, H), dt)
    T_eff = int(seq_len.max()) if B else 0
    stack = []
    t = 0
    while t < T_eff:
        valid = (t < seq_len)[:, None]
        h_op = _operand(h, precision)
        zx = x[t] @ Wx + bx
        zh = h_op @ Wh
        r = sigmoid(zx[:, :H] + zh[:, :H])
        u = sigmoid(zx[:, H:2 * H] + zh[:, H:2 * H])
        hn = zh[:, 2 * H:] + bhn
        n = np.tanh(zx[:, 2 * H:] + r * hn)
        h_new = (1.0 - u) * n + u * h
        stack.append(dict(r=r, u=u, n=n, hn=hn, h_prev=h, h_op=h_op, valid=valid))
        h = np.where(valid, h_new, h)
        y[t] = np.where(valid, h_new, 0.0)
        t += 1
    tape = dict(stack=stack, T_eff=T_eff, x=x, W=W, precision=precision, I=I, H=H)
    return y, h, tape


def gru_backward(tape, dy=None, dhT=None):
    """Gradient while-loop.  Returns dict(dx, dW [I+H,3H], dbias [4H], dh0)."""
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
    dbx = np.zeros(3 * H, dt)
    dbhn = np.zeros(H, dt)
    stack = list(tape["stack"])
    t = tape["T_eff"]
    while t > 0:
        t -= 1
        s = stack.pop()
        valid = s["valid"]
        r, u, n, hn = s["r"], s["u"], s["n"], s["hn"]
        dh_tot = dh + (np.where(valid, np.asarray(dy[t], dt), 0.0) if dy is not None else 0.0)
        da_u = dh_tot * (s["h_prev"] - n) * u * (1.0 - u)
        da_n = dh_tot * (1.0 - u) * (1.0 - n * n)
        da_r = da_n * hn * r * (1.0 - r)
        dzx = np.where(valid, np.concatenate([da_r, da_u, da_n], axis=1), 0.0)
        dzh = np.where(valid, np.concatenate([da_r, da_u, da_n * r], axis=1), 0.0)
        dzx_op = _operand(dzx, precision)
        dzh_op = _operand(dzh, precision)
        x_t = np.where(valid, x[t], 0.0)
        dx[t] = dzx_op @ Wx.T
        dWx += x_t.T @ dzx_op
        dWh += s["h_op"].T @ dzh_op
        dbx += dzx.sum(axis=0)
        dbhn += dzh[:, 2 * H:].sum(axis=0)
        dh_prev = dh_tot * u + dzh_op @ Wh.T
        dh = np.where(valid, dh_prev, dh)
    assert not stack
    return dict(dx=dx, dW=np.concatenate([dWx, dWh], axis=0),
                dbias=np.concatenate([dbx, dbhn]), dh0=dh)


def stacked_gru_forward(x, seq_len, Ws, biases, h0=None, precision="fp64"):
    tapes, hTs = [], []
    inp = x
    y = None
    for l, (Wl, bl) in enumerate(zip(Ws, biases)):
        y, hT, tape = gru_forward(inp, seq_len, Wl, bl, None if h0 is None else h0[l], precision)
        tapes.append(tape)
        hTs.append(hT)
        inp = _operand(y, precision)
    return y, np.stack(hTs), tapes


def stacked_gru_backward(tapes, dy=None, dhT=None):
    L = len(tapes)
    g_out = dy
    dWs, dbs, dh0s = [None] * L, [None] * L, [None] * L
    for l in reversed(range(L)):
        r = gru_backward(tapes[l], g_out, None if dhT is None else dhT[l])
        dWs[l], dbs[l], dh0s[l] = r["dW"], r["dbias"], r["dh0"]
        g_out = r["dx"]
    return dict(dx=g_out, dW=dWs, dbias=dbs, dh0=np.stack(dh0s))
