"""CPU oracle for the while-loop whose LSTM body holds a data-dependent cond.

TEST INFRASTRUCTURE ONLY, like the other oracles beside it; it shares no
code with the HIP library.

The loop construct is that of the LSTM oracle (Sections 4.2, 5.1, 5.2 of
Dynamic Control Flow in Large-Scale Machine Learning).  The body is a
conditional (Section 2.1, cond(pred, true_fn, false_fn)) whose predicate is
computed from the step's input and the loop state at every iteration:

    s = [x_t, h_{t-1}] . w_p + b_p     (one value per row; w_p [I+H], b_p scalar)
    (h_t, c_t) = cond(s > 0, lstm_step(x_t, h_{t-1}, c_{t-1}), (h_{t-1}, c_{t-1}))

so a row either runs the LSTM cell or keeps its state (it "skips" the step);
y_t is the resulting h_t at every valid step (with the input in the
predicate, a row that skipped can run again later).  Rows whose sequence has
ended keep their state and output 0, as in the plain loop.

Because the predicate depends on the state, it cannot be recomputed in the
gradient loop: the forward pushes the guard value of every iteration onto
the stack and the gradient loop pops it to control the conditional's
gradient (Section 5.1, the paragraph on control flow nested in a loop).  The
gradient of cond(p, f, g) is cond(p, grad f, grad g) (Section 5.1): the
LSTM-step gradient for rows that ran the cell, the identity for rows that
skipped (dh_{t-1} = dh_t + dy_t, dc_{t-1} = dc_t, dz = 0 so no contribution
to dW, db or dx_t).  The predicate is a step function, so w_p and b_p get no
gradient.

The bias argument is [4H + I + H + 1] = [b (4H), w_p (I + H: x part, then h
part, like a column of W), b_p]; dbias has the same length with zeros in the
predicate part.

Decision precision: the predicate is an integer decided by floating point,
so the oracle decides it in float32, the precision of the kernel's sums:
s = (s_x + s_h) + b_p in float32, s_x and s_h the float32 sums of the
products of x_t and op(h_{t-1}) with op(w_p), op the matrix-core operand
form (bfloat16 rounding in "bf16" mode, the identity otherwise).  The tape
keeps |s| of every valid decision so that a test can check that no decision
sits closer to the threshold than the two sides' differing summation orders
and trajectories could move it.
"""
from __future__ import annotations

import numpy as np

from .lstm import bf16_round, sigmoid

__all__ = ["skip_forward_literal", "skip_forward", "skip_backward",
           "stacked_skip_forward", "stacked_skip_backward"]


def _dtype(precision):
    if precision not in ("fp64", "fp32", "bf16"):
        raise ValueError(f"unknown precision {precision!r}")
    return np.float32 if precision == "fp32" else np.float64


def _operand(v, precision):
    return bf16_round(v) if precision == "bf16" else v


def _score(xt, h_op, wp_op, bp):
    """float32 predicate value of each row."""
    I = np.shape(xt)[-1]
    sx = np.asarray(xt, np.float32) @ np.asarray(wp_op[:I], np.float32)
    sh = np.asarray(h_op, np.float32) @ np.asarray(wp_op[I:], np.float32)
    return ((sx + sh) + np.float32(bp)).astype(np.float32)


def _split_bias(bias, I, H):
    bias = np.asarray(bias)
    if bias.shape[0] != 4 * H + I + H + 1:
        raise ValueError("bias must be [4H + I + H + 1] = [b (4H), w_p (I + H), b_p]")
    return bias[:4 * H], bias[4 * H:4 * H + I + H], float(bias[-1])


def _lstm_step(xt, h_op, c, Wx, Wh, b, H):
    z = xt @ Wx + h_op @ Wh + b
    i = sigmoid(z[..., 0:H])
    f = sigmoid(z[..., H:2 * H])
    g = np.tanh(z[..., 2 * H:3 * H])
    o = sigmoid(z[..., 3 * H:4 * H])
    c_new = f * c + i * g
    return i, f, g, o, c_new, o * np.tanh(c_new)


def skip_forward_literal(x, seq_len, W, bias, h0=None, c0=None, precision="fp64"):
    """One sequence at a time, the conditional as a Python branch.
    Returns y [T_max,B,H], hT, cT [B,H]."""
    x = np.asarray(x, np.float64)
    W = np.asarray(W, np.float64)
    T_max, B, I = x.shape
    H = W.shape[1] // 4
    b, wp, bp = _split_bias(np.asarray(bias, np.float64), I, H)
    wp_op = _operand(wp, precision)
    y = np.zeros((T_max, B, H))
    hT = np.zeros((B, H))
    cT = np.zeros((B, H))
    for r in range(B):
        h = np.zeros(H) if h0 is None else np.array(h0[r], np.float64)
        c = np.zeros(H) if c0 is None else np.array(c0[r], np.float64)
        for t in range(int(seq_len[r])):
            h_op = _operand(h, precision)
            if _score(x[t, r], h_op, wp_op, bp) > 0:   # cond(pred, true_fn, false_fn)
                _, _, _, _, c, h = _lstm_step(x[t, r], h_op, c, W[:I], W[I:], b, H)
            y[t, r] = h
        hT[r] = h
        cT[r] = c
    return y, hT, cT


def skip_forward(x, seq_len, W, bias, h0=None, c0=None, precision="fp64"):
    """Forward while-loop over the batch.  Returns (y, hT, cT, tape)."""
    dt = _dtype(precision)
    seq_len = np.asarray(seq_len, np.int64)
    x = np.asarray(x, dt)
    W = np.asarray(W, dt)
    T_max, B, I = x.shape
    H = W.shape[1] // 4
    if W.shape[0] != I + H:
        raise ValueError("W must have I+H rows")
    if (seq_len < 0).any() or (seq_len > T_max).any():
        raise ValueError("seq_len outside [0, T_max]")
    b, wp, bp = _split_bias(np.asarray(bias, dt), I, H)
    wp_op = _operand(wp, precision)
    Wx, Wh = W[:I], W[I:]
    h = np.zeros((B, H), dt) if h0 is None else np.array(h0, dt)
    c = np.zeros((B, H), dt) if c0 is None else np.array(c0, dt)
    y = np.zeros((T_max, B, H), dt)
    guards = np.zeros((T_max, B), np.int8)
    margin = np.full((T_max, B), np.inf)       # |s| of every valid decision
    T_eff = int(seq_len.max()) if B else 0
    stack = []
    t = 0
    while t < T_eff:
        valid = (t < seq_len)
        h_op = _operand(h, precision)
        s = _score(x[t], h_op, wp_op, bp)
        guard = valid & (s > 0)                      # pushed: it depends on the state
        i, f, g, o, c_new, h_new = _lstm_step(x[t], h_op, c, Wx, Wh, b, H)
        stack.append(dict(i=i, f=f, g=g, o=o, c_prev=c, c=c_new, h_op=h_op,
                          valid=valid[:, None], guard=guard[:, None]))
        c = np.where(guard[:, None], c_new, c)
        h = np.where(guard[:, None], h_new, h)
        y[t] = np.where(valid[:, None], h, 0.0)
        guards[t] = guard
        margin[t] = np.where(valid, np.abs(s), np.inf)
        t += 1
    tape = dict(stack=stack, T_eff=T_eff, x=x, W=W, precision=precision, I=I, H=H,
                guards=guards, margin=margin, min_margin=float(margin.min()) if margin.size else np.inf)
    return y, h, c, tape


def skip_backward(tape, dy=None, dhT=None, dcT=None):
    """Gradient while-loop; pops the guards to pick each row's branch gradient.
    Returns dict(dx, dW [I+H,4H], dbias [4H+I+H+1], dh0, dc0)."""
    precision = tape["precision"]
    dt = _dtype(precision)
    x, W = tape["x"], tape["W"]
    I, H = tape["I"], tape["H"]
    T_max, B, _ = x.shape
    Wx, Wh = W[:I], W[I:]
    dh = np.zeros((B, H), dt) if dhT is None else np.array(dhT, dt)
    dc = np.zeros((B, H), dt) if dcT is None else np.array(dcT, dt)
    dx = np.zeros((T_max, B, I), dt)
    dWx = np.zeros_like(Wx)
    dWh = np.zeros_like(Wh)
    db = np.zeros(4 * H, dt)
    stack = list(tape["stack"])
    t = tape["T_eff"]
    while t > 0:
        t -= 1
        s = stack.pop()
        valid, guard = s["valid"], s["guard"]
        i, f, g, o = s["i"], s["f"], s["g"], s["o"]
        dh_tot = dh + (np.where(valid, np.asarray(dy[t], dt), 0.0) if dy is not None else 0.0)
        # true branch: the LSTM step's gradient
        tc = np.tanh(s["c"])
        dc_tot = dc + dh_tot * o * (1.0 - tc * tc)
        dz = np.concatenate([dc_tot * g * i * (1.0 - i), dc_tot * s["c_prev"] * f * (1.0 - f),
                             dc_tot * i * (1.0 - g * g), dh_tot * tc * o * (1.0 - o)], axis=1)
        dz = np.where(guard, dz, 0.0)
        dz_op = _operand(dz, precision)
        x_t = np.where(guard, x[t], 0.0)
        dx[t] = dz_op @ Wx.T
        dWx += x_t.T @ dz_op
        dWh += s["h_op"].T @ dz_op
        db += dz.sum(axis=0)
        # cond gradient: the branch each row took; finished rows pass through
        dh = np.where(guard, dz_op @ Wh.T, np.where(valid, dh_tot, dh))
        dc = np.where(guard, dc_tot * f, dc)
    assert not stack
    dbias = np.concatenate([db, np.zeros(I + H + 1, dt)])
    return dict(dx=dx, dW=np.concatenate([dWx, dWh], axis=0), dbias=dbias, dh0=dh, dc0=dc)


def stacked_skip_forward(x, seq_len, Ws, biases, h0=None, c0=None, precision="fp64"):
    tapes, hTs, cTs = [], [], []
    inp = x
    y = None
    for l, (Wl, bl) in enumerate(zip(Ws, biases)):
        y, hT, cT, tape = skip_forward(inp, seq_len, Wl, bl, None if h0 is None else h0[l],
                                       None if c0 is None else c0[l], precision)
        tapes.append(tape)
        hTs.append(hT)
        cTs.append(cT)
        inp = _operand(y, precision)
    return y, np.stack(hTs), np.stack(cTs), tapes


def stacked_skip_backward(tapes, dy=None, dhT=None, dcT=None):
    L = len(tapes)
    g_out = dy
    dWs, dbs, dh0s, dc0s = [None] * L, [None] * L, [None] * L, [None] * L
    for l in reversed(range(L)):
        r = skip_backward(tapes[l], g_out, None if dhT is None else dhT[l],
                          None if dcT is None else dcT[l])
        dWs[l], dbs[l], dh0s[l], dc0s[l] = r["dW"], r["dbias"], r["dh0"], r["dc0"]
        g_out = r["dx"]
    return dict(dx=g_out, dW=dWs, dbias=dbs, dh0=np.stack(dh0s), dc0=np.stack(dc0s))
