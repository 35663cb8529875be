"""CPU oracle for the device-side LSTM while-loop and its gradient loop.

TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the
benchmark's CPU-baseline leg may import this module; the product path never
does.  It shares no code with the HIP library: it is a plain, slow NumPy
restatement of what the method computes, written for checking by eye.

What is computed (Dynamic Control Flow in Large-Scale Machine Learning,
Sections 2.1, 4.2, 5.1, 5.2 and 6.2):

* ``while_loop(pred, body, inits)`` runs ``body`` while ``pred`` holds and
  returns the final loop variables; if the predicate is false at entry the
  inits are returned unchanged (Section 4.2, the Exit of a loop that never
  iterates).  Here the loop variables are (t, h, c), the loop constants are
  x, W and bias, and the predicate is ``t < max_b seq_len[b]``; the number of
  iterations is recorded so that the gradient loop can run the same count
  in reverse (Section 5.1, first feature of the loop gradient).
* The body is one step of an LSTM cell (the paper cites Hochreiter and
  Schmidhuber without equations; the textbook cell with a forget gate is
  used): z = [x_t, h_{t-1}] W + b split into gate blocks (i, f, g, o),
  i, f, o = sigmoid, g = tanh, c_t = f*c_{t-1} + i*g, h_t = o*tanh(c_t).
  Rows whose sequence has ended keep their state; their output is 0
  (the dynamic_rnn workload of Section 6.2 over variable-length sequences).
* Values the gradient needs are pushed on a stack by the forward loop and
  popped in reverse by the gradient loop (Section 5.1, stack figure).
* Gradients of loop variables are loop variables of the gradient loop,
  initialised with the gradient of the loop outputs; gradients of loop
  constants (W, bias) are sums over iterations, accumulated eagerly
  (Section 5.1, second and third features, and its remark on eager
  accumulation).  The per-step products follow the matmul gradient
  g_x = g_z y^T, g_y = x^T g_z (Section 5.1).
* Reading x_t from a TensorArray has as gradient a write of dx_t into the
  gradient TensorArray (Section 5.2).

Precision modes
  "fp64": every value in float64 (reference for float32 GPU runs).
  "bf16": float64 arithmetic, with bfloat16 rounding (nearest, ties to even)
          exactly where the bfloat16 kernels round a matrix-core operand:
          h_{t-1} before the recurrent product; dz before the products that
          give dx, dh_{t-1} and dW; h_{t-1} before the dW product.  x and W
          are expected bfloat16-representable already.  db sums unrounded dz.
  "fp32": the "fp64" algorithm in float32 arrays (CPU timing baseline only).
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "bf16_round", "sigmoid", "lstm_forward_literal", "lstm_forward",
    "lstm_backward", "stacked_forward", "stacked_backward",
    "matmul_chain_grad",
]


# --------------------------------------------------------------------------
# bfloat16 rounding, from the number format: bfloat16 keeps the float32
# exponent range and 8 significant bits.  Round to nearest, ties to even.
# --------------------------------------------------------------------------
def bf16_round(a):
    """Round float64 values to the nearest bfloat16 value (ties to even).

    Normal range: keep 8 significant bits.  Below 2^-126 the spacing is the
    fixed subnormal quantum 2^-133.  Overflow past the largest finite value
    (rounding boundary 2^128 * (1 - 2^-9)) gives infinity.
    """
    a = np.asarray(a, dtype=np.float64)
    out = np.empty_like(a)
    finite = np.isfinite(a)
    out[~finite] = a[~finite]
    v = a[finite]
    mant, expo = np.frexp(v)                 # v = mant * 2^expo, |mant| in [0.5, 1)
    normal = np.abs(v) >= 2.0 ** -126
    r = np.empty_like(v)
    # 8 significant bits: mant * 2^8 is in [128, 256); np.rint rounds half to even
    r[normal] = np.ldexp(np.rint(np.ldexp(mant[normal], 8)), expo[normal] - 8)
    q = 2.0 ** -133
    r[~normal] = np.rint(v[~normal] / q) * q
    big = np.abs(v) >= 2.0 ** 128 * (1.0 - 2.0 ** -9)
    r[big] = np.copysign(np.inf, v[big])
    out[finite] = r
    return out


def sigmoid(u):
    return 1.0 / (1.0 + np.exp(-u))


def _dtype(precision):
    if precision not in ("fp64", "fp32", "bf16"):
        raise ValueError(f"unknown precision {precision!r}")
    return np.float32 if precision == "fp32" else np.float64


def _operand(v, precision):
    """Matrix-core operand form of an activation (see module docstring)."""
    return bf16_round(v) if precision == "bf16" else v


# --------------------------------------------------------------------------
# Literal form: each sequence alone, a Python loop over its own length.
# --------------------------------------------------------------------------
def lstm_forward_literal(x, seq_len, W, bias, h0=None, c0=None):
    """float64, one sequence at a time: the plain definition of the result.

    x [T_max,B,I], seq_len [B], W [I+H,4H] (rows: x part then h part;
    gate column blocks i,f,g,o), bias [4H], h0/c0 [B,H] or None.
    Returns y [T_max,B,H] (0 at t >= seq_len[b]), hT [B,H], cT [B,H].
    """
    x = np.asarray(x, np.float64)
    W = np.asarray(W, np.float64)
    bias = np.asarray(bias, np.float64)
    T_max, B, I = x.shape
    H = W.shape[1] // 4
    y = np.zeros((T_max, B, H))
    hT = np.zeros((B, H))
    cT = np.zeros((B, H))
    for b in range(B):
        h = np.zeros(H) if h0 is None else np.array(h0[b], np.float64)
        c = np.zeros(H) if c0 is None else np.array(c0[b], np.float64)
        for t in range(int(seq_len[b])):
            z = np.concatenate([x[t, b], h]) @ W + bias
            i = sigmoid(z[0:H])
            f = sigmoid(z[H:2 * H])
            g = np.tanh(z[2 * H:3 * H])
            o = sigmoid(z[3 * H:4 * H])
            c = f * c + i * g
            h = o * np.tanh(c)
            y[t, b] = h
        hT[b] = h
        cT[b] = c
    return y, hT, cT


# --------------------------------------------------------------------------
# Batched, masked form: the while-loop over t with a per-row validity mask.
# --------------------------------------------------------------------------
def lstm_forward(x, seq_len, W, bias, h0=None, c0=None, precision="fp64"):
    """Forward while-loop over the batch.  Returns (y, hT, cT, tape).

    The tape is the stack of Section 5.1: one entry per iteration, pushed in
    order, holding what the gradient loop pops.  tape["T_eff"] is the loop
    counter the forward records (Section 5.1, first feature).
    """
    dt = _dtype(precision)
    seq_len = np.asarray(seq_len, np.int64)
    x = np.asarray(x, dt)
    W = np.asarray(W, dt)
    bias = np.asarray(bias, dt)
    T_max, B, I = x.shape
    H = W.shape[1] // 4
    if W.shape[0] != I + H:
        raise ValueError("W must have I+H rows")
    if (seq_len < 0).any() or (seq_len > T_max).any():
        raise ValueError("seq_len outside [0, T_max]")
    Wx, Wh = W[:I], W[I:]
    h = np.zeros((B, H), dt) if h0 is None else np.array(h0, dt)
    c = np.zeros((B, H), dt) if c0 is None else np.array(c0, dt)
    y = np.zeros((T_max, B, H), dt)
    T_eff = int(seq_len.max()) if B else 0        # loop predicate: t < T_eff
    stack = []
    t = 0
    while t < T_eff:
        valid = (t < seq_len)[:, None]
        h_op = _operand(h, precision)
        z = x[t] @ Wx + h_op @ Wh + bias
        i = sigmoid(z[:, 0:H])
        f = sigmoid(z[:, H:2 * H])
        g = np.tanh(z[:, 2 * H:3 * H])
        o = sigmoid(z[:, 3 * H:4 * H])
        c_new = f * c + i * g
        h_new = o * np.tanh(c_new)
        stack.append(dict(i=i, f=f, g=g, o=o, c_prev=c, c=c_new, h_op=h_op,
                          valid=valid))
        c = np.where(valid, c_new, c)
        h = np.where(valid, h_new, h)
        y[t] = np.where(valid, h_new, 0.0)
        t += 1
    tape = dict(stack=stack, T_eff=T_eff, seq_len=seq_len, x=x, W=W,
                precision=precision, I=I, H=H)
    return y, h, c, tape


def lstm_backward(tape, dy=None, dhT=None, dcT=None):
    """Gradient while-loop: same trip count as the forward, in reverse.

    dy [T_max,B,H] or None, dhT/dcT [B,H] or None (zeros).
    Returns dict(dx [T_max,B,I], dW [I+H,4H], dbias [4H], dh0 [B,H], dc0 [B,H]).
    """
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
    while t > 0:                               # same number of iterations
        t -= 1
        s = stack.pop()                         # pop in reverse order
        valid = s["valid"]
        i, f, g, o = s["i"], s["f"], s["g"], s["o"]
        dh_tot = dh + (np.where(valid, np.asarray(dy[t], dt), 0.0)
                       if dy is not None else 0.0)
        tc = np.tanh(s["c"])
        do = dh_tot * tc
        dc_tot = dc + dh_tot * o * (1.0 - tc * tc)
        di = dc_tot * g
        df = dc_tot * s["c_prev"]
        dg = dc_tot * i
        dz = np.concatenate([di * i * (1.0 - i), df * f * (1.0 - f),
                             dg * (1.0 - g * g), do * o * (1.0 - o)], axis=1)
        dz = np.where(valid, dz, 0.0)
        dz_op = _operand(dz, precision)
        x_t = np.where(valid, x[t], 0.0)        # padding never enters a product
        dx[t] = dz_op @ Wx.T                    # TensorArray read -> write of dx_t
        dWx += x_t.T @ dz_op                    # loop constants: sum over iterations
        dWh += s["h_op"].T @ dz_op
        db += dz.sum(axis=0)
        dh_prev = dz_op @ Wh.T
        dc_prev = dc_tot * f
        dh = np.where(valid, dh_prev, dh)       # finished rows pass gradients through
        dc = np.where(valid, dc_prev, dc)
    assert not stack
    return dict(dx=dx, dW=np.concatenate([dWx, dWh], axis=0), dbias=db,
                dh0=dh, dc0=dc)


# --------------------------------------------------------------------------
# Two stacked layers: layer 2 reads layer 1's output sequence.
# --------------------------------------------------------------------------
def stacked_forward(x, seq_len, Ws, biases, h0=None, c0=None, precision="fp64"):
    """L layers; layer l+1 takes layer l's y (bfloat16-rounded in "bf16" mode,
    the operand form of the next layer's input).  h0/c0 are [L,B,H] or None.
    Returns (y_top, hT [L,B,H], cT [L,B,H], tapes)."""
    tapes, hTs, cTs = [], [], []
    inp = x
    y = None
    for l, (Wl, bl) in enumerate(zip(Ws, biases)):
        y, hT, cT, tape = lstm_forward(inp, seq_len, Wl, bl,
                                       None if h0 is None else h0[l],
                                       None if c0 is None else c0[l], precision)
        tapes.append(tape)
        hTs.append(hT)
        cTs.append(cT)
        inp = _operand(y, precision)
    return y, np.stack(hTs), np.stack(cTs), tapes


def stacked_backward(tapes, dy=None, dhT=None, dcT=None):
    """Backward through L stacked layers; the gradient reaching layer l's
    output is layer l+1's dx (rounding of the inter-layer activation is
    passed straight through).  Returns dict with dx, dW [list], dbias [list],
    dh0 [L,B,H], dc0 [L,B,H]."""
    L = len(tapes)
    g_out = dy
    dWs, dbs, dh0s, dc0s = [None] * L, [None] * L, [None] * L, [None] * L
    for l in reversed(range(L)):
        r = lstm_backward(tapes[l], g_out,
                          None if dhT is None else dhT[l],
                          None if dcT is None else dcT[l])
        dWs[l], dbs[l], dh0s[l], dc0s[l] = r["dW"], r["dbias"], r["dh0"], r["dc0"]
        g_out = r["dx"]
    return dict(dx=g_out, dW=dWs, dbias=dbs, dh0=np.stack(dh0s),
                dc0=np.stack(dc0s))


# --------------------------------------------------------------------------
# The loop-gradient scaffolding on the paper's own small example
# (Section 5.1, "computing the gradient of a loop by unrolling"):
# a_{k+1} = a_k w for k < n, y = sum(a_n); gradient w.r.t. w.
# --------------------------------------------------------------------------
def matmul_chain_grad(x, w, n):
    """Gradient of y = sum(a_n), a_0 = x, a_{k+1} = a_k @ w, w.r.t. w, computed
    with the three loop-gradient rules: a forward loop that pushes a_k and
    counts iterations, a reverse loop of the same count whose loop variable
    is g_a, and g_w summed over iterations.  Returns (y, g_w)."""
    x = np.asarray(x, np.float64)
    w = np.asarray(w, np.float64)
    stack = []
    a = x
    k = 0
    while k < n:
        stack.append(a)
        a = a @ w
        k += 1
    y = a.sum()
    g_a = np.ones_like(a)                       # gradient of reduce_sum
    g_w = np.zeros_like(w)
    while k > 0:
        k -= 1
        a_k = stack.pop()
        g_w += a_k.T @ g_a                      # MatMulGrad, y-side
        g_a = g_a @ w.T                         # MatMulGrad, x-side
    return y, g_w
