"""CPU oracle for the while-loop whose LSTM body holds a nested while-loop
with a data-dependent trip count (Adaptive Computation Time's halting rule).

TEST INFRASTRUCTURE ONLY, like the other oracles beside it; it shares no
code with the HIP library.

The outer loop is the LSTM loop of the other oracles (Sections 4.2, 5.1 and
5.2 of Dynamic Control Flow in Large-Scale Machine Learning).  Its body is a
second while-loop (Section 2.2 motivates such bodies with Adaptive
Computation Time, where an RNN "ponders" each input a data-dependent number
of times): for every row still running at step t,

    (h, c) = (h_{t-1}, c_{t-1});  P = 0;  n = 0
    while True:                               # the inner ("ponder") loop
        (h, c) = lstm_step(x_t, h, c);  n += 1
        if n == M: break                      # at most M ponder steps
        P += sigmoid(h . w_p + b_p)           # halting unit on the new state
        if P >= 1 - eps: break                # cumulative halting probability
    (h_t, c_t) = (h, c);  y_t = h_t;  N(t, row) = n

with the same x_t at every ponder step.  ACT's halting rule (halt once the
summed halting probabilities reach 1 - eps, eps = 0.01) decides the inner
trip count from the state; ACT's mean-field output (a probability-weighted
average of the ponder states) and its ponder cost are not part of this
body: the loop keeps the last ponder state, so the halting unit only
decides how often the body runs.  The decision is a step function of the
state, so w_p and b_p get no gradient.

Gradient (Section 5.1, nested loops): the inner loop's trip count depends
on the state and cannot be recomputed backwards, so the forward pushes every
inner trip count N(t, row) and the values of every ponder step onto the
stack; the gradient loop runs, for t = T_eff - 1 .. 0, an inner gradient
loop of N(t, row) iterations in reverse, popping them.  Each ponder step's
gradient is the LSTM step's; dy_t enters at the last ponder state; x_t is
read by every ponder step, so dx_t sums the ponder steps' dz_k W_x^T; dW
sums [x_t, h^{k-1}]^T dz_k over steps and ponder steps; db sums dz_k.

The bias argument is [4H + H + 1] = [b (4H), w_p (H), b_p]; dbias has the same
length with zeros in the halting part.  M is `ponder_max` (>= 1).

Decision precision: the inner trip count is an integer decided by floating
point, so the oracle decides it in float32, the precision of the kernel:
s = sum(op(h) * op(w_p)) in float32 plus b_p, p = sigmoid(s) in float32, P
summed in float32, halting when P >= float32(1 - eps); op is the matrix-core
operand form (bfloat16 rounding in "bf16" mode, the identity otherwise).  The
tape keeps |P - (1 - eps)| of every decision so that a test can check that
no decision sits closer to the threshold than the two sides' summation
orders and activation functions could move it.
"""
from __future__ import annotations

import numpy as np

from .lstm import bf16_round, sigmoid

__all__ = ["act_forward_literal", "act_forward", "act_backward",
           "stacked_act_forward", "stacked_act_backward", "ACT_EPS"]

ACT_EPS = 0.01


def _dtype(precision):
    if precision not in ("fp64", "fp32", "bf16"):
        raise ValueError(f"unknown precision {precision!r}")
    return np.float32 if precision == "fp32" else np.float64


def _operand(v, precision):
    return bf16_round(v) if precision == "bf16" else v


def _split_bias(bias, H):
    bias = np.asarray(bias)
    if bias.shape[0] != 5 * H + 1:
        raise ValueError("bias must be [4H + H + 1] = [b (4H), w_p (H), b_p]")
    return bias[:4 * H], bias[4 * H:5 * H], float(bias[-1])


def _halt_prob(h_op, wp_op, bp):
    """float32 halting probability of each row from its (operand-form) state."""
    s = (np.asarray(h_op, np.float32) @ np.asarray(wp_op, np.float32)) + np.float32(bp)
    return (np.float32(1.0) / (np.float32(1.0) + np.exp(-s.astype(np.float32)))).astype(np.float32)


def _lstm_step(xt, h_op, c, Wx, Wh, b, H):
    z = xt @ Wx + h_op @ Wh + b
    i = sigmoid(z[..., 0:H])
    f = sigmoid(z[..., H:2 * H])
    g = np.tanh(z[..., 2 * H:3 * H])
    o = sigmoid(z[..., 3 * H:4 * H])
    c_new = f * c + i * g
    return i, f, g, o, c_new, o * np.tanh(c_new)


def act_forward_literal(x, seq_len, W, bias, h0=None, c0=None, precision="fp64", ponder_max=4,
                        eps=ACT_EPS):
    """One sequence at a time; both loops are Python while loops.
    Returns y [T_max,B,H], hT, cT [B,H], trips [T_max,B] (0 past the length)."""
    x = np.asarray(x, np.float64)
    W = np.asarray(W, np.float64)
    T_max, B, I = x.shape
    H = W.shape[1] // 4
    b, wp, bp = _split_bias(np.asarray(bias, np.float64), H)
    wp_op = _operand(wp, precision)
    thr = np.float32(1.0 - eps)
    y = np.zeros((T_max, B, H))
    hT = np.zeros((B, H))
    cT = np.zeros((B, H))
    trips = np.zeros((T_max, B), np.int64)
    for r in range(B):
        h = np.zeros(H) if h0 is None else np.array(h0[r], np.float64)
        c = np.zeros(H) if c0 is None else np.array(c0[r], np.float64)
        t = 0
        while t < int(seq_len[r]):
            P = np.float32(0.0)
            n = 0
            while True:                                   # the nested loop
                _, _, _, _, c, h = _lstm_step(x[t, r], _operand(h, precision), c, W[:I], W[I:], b, H)
                n += 1
                if n == ponder_max:
                    break
                P = np.float32(P + _halt_prob(_operand(h, precision), wp_op, bp))
                if P >= thr:
                    break
            y[t, r] = h
            trips[t, r] = n
            t += 1
        hT[r] = h
        cT[r] = c
    return y, hT, cT, trips


def act_forward(x, seq_len, W, bias, h0=None, c0=None, precision="fp64", ponder_max=4, eps=ACT_EPS):
    """Forward while-loop over the batch, the nested loop masked per row.
    Returns (y, hT, cT, tape)."""
    if ponder_max < 1:
        raise ValueError("ponder_max must be >= 1")
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
    b, wp, bp = _split_bias(np.asarray(bias, dt), H)
    wp_op = _operand(wp, precision)
    thr = np.float32(1.0 - eps)
    Wx, Wh = W[:I], W[I:]
    h = np.zeros((B, H), dt) if h0 is None else np.array(h0, dt)
    c = np.zeros((B, H), dt) if c0 is None else np.array(c0, dt)
    y = np.zeros((T_max, B, H), dt)
    trips = np.zeros((T_max, B), np.int64)
    margins = []
    row_margin = np.full(B, np.inf)    # per row: the closest of its decisions
    T_eff = int(seq_len.max()) if B else 0
    stack = []          # one entry per outer step: that step's ponder steps
    t = 0
    while t < T_eff:
        valid = t < seq_len
        running = valid.copy()
        P = np.zeros(B, np.float32)
        n = np.zeros(B, np.int64)
        steps = []
        while running.any():                 # the nested loop: while some row ponders
            h_op = _operand(h, precision)
            i, f, g, o, c_new, h_new = _lstm_step(x[t], h_op, c, Wx, Wh, b, H)
            run = running.copy()[:, None]      # (running changes below)
            steps.append(dict(i=i, f=f, g=g, o=o, c_prev=c, c=c_new, h_op=h_op, guard=run))
            c = np.where(run, c_new, c)
            h = np.where(run, h_new, h)
            n += running
            stop = running & (n == ponder_max)
            cont = running & ~stop
            if cont.any():
                P_new = (P + _halt_prob(_operand(h, precision), wp_op, bp)).astype(np.float32)
                P = np.where(cont, P_new, P)
                dist = np.abs(P_new - thr).astype(np.float64)
                margins.append(dist[cont])
                row_margin = np.where(cont, np.minimum(row_margin, dist), row_margin)
                stop |= cont & (P_new >= thr)
            running &= ~stop
        stack.append(dict(steps=steps, valid=valid[:, None], trips=n.copy()))
        y[t] = np.where(valid[:, None], h, 0.0)
        trips[t] = n
        t += 1
    m = np.concatenate(margins) if margins else np.zeros(0)
    tape = dict(stack=stack, T_eff=T_eff, x=x, W=W, precision=precision, I=I, H=H, trips=trips,
                min_margin=float(m.min()) if m.size else np.inf, row_margin=row_margin)
    return y, h, c, tape


def act_backward(tape, dy=None, dhT=None, dcT=None):
    """Gradient while-loop with a nested gradient loop per step: pops the
    inner trip counts and each ponder step's values.
    Returns dict(dx, dW [I+H,4H], dbias [5H+1], dh0, dc0)."""
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
        entry = stack.pop()
        valid = entry["valid"]
        if dy is not None:
            dh = dh + np.where(valid, np.asarray(dy[t], dt), 0.0)
        steps = list(entry["steps"])
        while steps:                          # the nested gradient loop, in reverse
            s = steps.pop()
            run = s["guard"]
            i, f, g, o = s["i"], s["f"], s["g"], s["o"]
            tc = np.tanh(s["c"])
            dc_tot = dc + dh * o * (1.0 - tc * tc)
            dz = np.concatenate([dc_tot * g * i * (1.0 - i), dc_tot * s["c_prev"] * f * (1.0 - f),
                                 dc_tot * i * (1.0 - g * g), dh * tc * o * (1.0 - o)], axis=1)
            dz = np.where(run, dz, 0.0)
            dz_op = _operand(dz, precision)
            dx[t] += dz_op @ Wx.T
            dWx += np.where(run, x[t], 0.0).T @ dz_op
            dWh += s["h_op"].T @ dz_op
            db += dz.sum(axis=0)
            dh = np.where(run, dz_op @ Wh.T, dh)
            dc = np.where(run, dc_tot * f, dc)
    assert not stack
    dbias = np.concatenate([db, np.zeros(H + 1, dt)])
    return dict(dx=dx, dW=np.concatenate([dWx, dWh], axis=0), dbias=dbias, dh0=dh, dc0=dc)


def stacked_act_forward(x, seq_len, Ws, biases, h0=None, c0=None, precision="fp64", ponder_max=4,
                        eps=ACT_EPS):
    tapes, hTs, cTs = [], [], []
    inp = x
    y = None
    for l, (Wl, bl) in enumerate(zip(Ws, biases)):
        y, hT, cT, tape = act_forward(inp, seq_len, Wl, bl, None if h0 is None else h0[l],
                                      None if c0 is None else c0[l], precision, ponder_max, eps)
        tapes.append(tape)
        hTs.append(hT)
        cTs.append(cT)
        inp = _operand(y, precision)
    return y, np.stack(hTs), np.stack(cTs), tapes


def stacked_act_backward(tapes, dy=None, dhT=None, dcT=None):
    L = len(tapes)
    g_out = dy
    dWs, dbs, dh0s, dc0s = [None] * L, [None] * L, [None] * L, [None] * L
    for l in reversed(range(L)):
        r = act_backward(tapes[l], g_out, None if dhT is None else dhT[l],
                         None if dcT is None else dcT[l])
        dWs[l], dbs[l], dh0s[l], dc0s[l] = r["dW"], r["dbias"], r["dh0"], r["dc0"]
        g_out = r["dx"]
    return dict(dx=g_out, dW=dWs, dbias=dbs, dh0=np.stack(dh0s), dc0=np.stack(dc0s))
