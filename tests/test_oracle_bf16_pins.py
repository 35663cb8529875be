"""Pins for the oracles' bfloat16 mode: where it rounds.

The "bf16" precision mode of every oracle computes in float64 and rounds to
bfloat16 exactly where the bfloat16 kernels round a matrix-core operand
(h_{t-1} before the recurrent product; dz before the products that give dx,
dh_{t-1} and dW; the layer below's y as the next layer's input; the
predicate / halting weights), while the state, the cell arithmetic and the
bias sums stay unrounded.

Independent implementation here: torch autograd (CPU, float64) run one
sequence at a time in Python loops, with the cell's nonlinear part taken from
torch.nn.LSTMCell / torch.nn.RNNCell (input weights the identity, recurrent
weights zero, so the library cell applies its gates to the pre-activations it
is given) and the rounding points as two small autograd functions built on
torch's float -> bfloat16 conversion:
- RoundOperand: forward rounds, backward passes the gradient through;
- RoundGradProduct: forward a @ w, backward rounds the incoming gradient
  before the two products (grad_a = bf16(g) w^T, grad_w = a^T bf16(g)).
The GRU's cell (no library cell can take its reset-gated recurrent part from
outside) is written with torch operations and first checked against
torch.nn.GRUCell in float64.

Each test also removes one rounding point at a time from the torch side and
checks that the results then move well beyond the tolerance, so every
rounding point is exercised.
"""
import numpy as np
import pytest
import torch

import oracle

TOL = dict(rtol=1e-10, atol=1e-12)


def t_round(a):
    return a.to(torch.bfloat16).to(torch.float64)


class RoundOperand(torch.autograd.Function):
    @staticmethod
    def forward(ctx, a):
        return t_round(a)

    @staticmethod
    def backward(ctx, g):
        return g


class RoundGradProduct(torch.autograd.Function):
    @staticmethod
    def forward(ctx, a, w):
        ctx.save_for_backward(a, w)
        return a @ w

    @staticmethod
    def backward(ctx, g):
        a, w = ctx.saved_tensors
        gr = t_round(g)
        return gr @ w.T, a.T @ gr


class Rounding:
    """The rounding points of the torch side; each can be switched off."""

    def __init__(self, h=True, dz=True, inp=True):
        self.h, self.dz, self.inp = h, dz, inp

    def op(self, a):          # a recurrent-product operand
        return RoundOperand.apply(a) if self.h else a

    def layer_input(self, a):  # the layer below's y as the next layer's input
        return RoundOperand.apply(a) if self.inp else a

    def prod(self, a, w):
        return RoundGradProduct.apply(a, w) if self.dz else a @ w


def _bf16_case(rng, T, B, I, H, G, lens, scale=0.6):
    x = oracle.bf16_round(rng.standard_normal((T, B, I)))
    W = oracle.bf16_round(rng.uniform(-scale, scale, (I + H, G * H)))
    h0 = 0.5 * rng.standard_normal((B, H))
    c0 = 0.5 * rng.standard_normal((B, H))
    dy = rng.standard_normal((T, B, H))
    dhT = rng.standard_normal((B, H))
    dcT = rng.standard_normal((B, H))
    return x, np.asarray(lens, np.int64), W, h0, c0, dy, dhT, dcT


def _lstm_cell(H):
    cell = torch.nn.LSTMCell(4 * H, H).double()
    with torch.no_grad():
        cell.weight_ih.copy_(torch.eye(4 * H, dtype=torch.float64))
        cell.weight_hh.zero_()
        cell.bias_ih.zero_()
        cell.bias_hh.zero_()
    cell.requires_grad_(False)
    return cell


def _leaf(a):
    return torch.from_numpy(np.array(a, np.float64)).requires_grad_(True)


def _grad(t, like):
    return t.grad.numpy() if t.grad is not None else np.zeros_like(like)


def _max_rel(a, b):
    a, b = np.asarray(a), np.asarray(b)
    s = max(np.abs(b).max(), 1e-300)
    return np.abs(a - b).max() / s


# ------------------------------------------------------------------ LSTM
def _torch_lstm(x, lens, Ws, bs, h0, c0, dy, dhT, dcT, rnd):
    """L stacked LSTM layers, torch autograd per sequence.  h0/c0/dhT/dcT
    [L,B,H]; returns forward outputs and every gradient."""
    T, B, I = x.shape
    L = len(Ws)
    H = Ws[0].shape[1] // 4
    cell = _lstm_cell(H)
    xs = _leaf(x)
    Wt = [_leaf(W) for W in Ws]
    bt = [_leaf(b) for b in bs]
    h0t, c0t = _leaf(h0), _leaf(c0)
    y = np.zeros((T, B, H))
    hT, cT = np.zeros((L, B, H)), np.zeros((L, B, H))
    loss = 0.0
    for r in range(B):
        n = int(lens[r])
        inp = [xs[t, r:r + 1] for t in range(n)]
        for l in range(L):
            Il = Ws[l].shape[0] - H
            Wx, Wh = Wt[l][:Il], Wt[l][Il:]
            h, c = h0t[l, r:r + 1], c0t[l, r:r + 1]
            outs = []
            for t in range(n):
                pre = rnd.prod(inp[t], Wx) + rnd.prod(rnd.op(h), Wh) + bt[l]
                h, c = cell(pre, (h, c))
                outs.append(h)
            loss = loss + (h * torch.from_numpy(dhT[l, r:r + 1])).sum() + (c * torch.from_numpy(dcT[l, r:r + 1])).sum()
            hT[l, r], cT[l, r] = h.detach().numpy()[0], c.detach().numpy()[0]
            inp = [rnd.layer_input(o) for o in outs]
        for t in range(n):
            loss = loss + (outs[t] * torch.from_numpy(dy[t, r:r + 1])).sum()
            y[t, r] = outs[t].detach().numpy()[0]
    loss.backward()
    return dict(y=y, hT=hT, cT=cT, dx=_grad(xs, x), dW=[_grad(w, W) for w, W in zip(Wt, Ws)],
                db=[_grad(b, bb) for b, bb in zip(bt, bs)], dh0=_grad(h0t, h0), dc0=_grad(c0t, c0))


def _oracle_lstm(x, lens, Ws, bs, h0, c0, dy, dhT, dcT):
    y, hT, cT, tapes = oracle.stacked_forward(x, lens, Ws, bs, h0, c0, precision="bf16")
    g = oracle.stacked_backward(tapes, dy, dhT, dcT)
    return dict(y=y, hT=hT, cT=cT, dx=g["dx"], dW=g["dW"], db=g["dbias"], dh0=g["dh0"], dc0=g["dc0"])


def _compare(got, ref, keys):
    for k in keys:
        a, b = got[k], ref[k]
        if isinstance(a, list):
            for i, (ai, bi) in enumerate(zip(a, b)):
                np.testing.assert_allclose(ai, bi, err_msg=f"{k}[{i}]", **TOL)
        else:
            np.testing.assert_allclose(a, b, err_msg=k, **TOL)


def _spread(got, ref, keys):
    """Largest max-normalised difference over the outputs."""
    out = 0.0
    for k in keys:
        a, b = got[k], ref[k]
        pairs = zip(a, b) if isinstance(a, list) else [(a, b)]
        for ai, bi in pairs:
            if np.abs(bi).max() > 0:
                out = max(out, _max_rel(ai, bi))
    return out


LSTM_KEYS = ("y", "hT", "cT", "dx", "dW", "db", "dh0", "dc0")


@pytest.mark.parametrize("layers", [1, 2])
def test_lstm_bf16_mode_rounds_where_the_kernels_do(layers):
    rng = np.random.default_rng(9100 + layers)
    T, B, I, H = 6, 4, 5, 3
    x, lens, W1, h0, c0, dy, dhT, dcT = _bf16_case(rng, T, B, I, H, 4, [6, 3, 0, 5])
    Ws = [W1] + [oracle.bf16_round(rng.uniform(-0.6, 0.6, (2 * H, 4 * H))) for _ in range(layers - 1)]
    bs = [rng.uniform(-0.6, 0.6, 4 * H) for _ in range(layers)]
    h0 = 0.5 * rng.standard_normal((layers, B, H))
    c0 = 0.5 * rng.standard_normal((layers, B, H))
    dhT = rng.standard_normal((layers, B, H))
    dcT = rng.standard_normal((layers, B, H))
    ref = _oracle_lstm(x, lens, Ws, bs, h0, c0, dy, dhT, dcT)
    _compare(_torch_lstm(x, lens, Ws, bs, h0, c0, dy, dhT, dcT, Rounding()), ref, LSTM_KEYS)
    # every rounding point matters: without it the results move far beyond the tolerance
    points = [dict(h=False), dict(dz=False)] + ([dict(inp=False)] if layers > 1 else [])
    for off in points:
        moved = _spread(_torch_lstm(x, lens, Ws, bs, h0, c0, dy, dhT, dcT, Rounding(**off)), ref, LSTM_KEYS)
        assert moved > 1e-5, off


# ------------------------------------------------------------------ RNN
def _torch_rnn(x, lens, W, b, h0, dy, dhT, rnd):
    T, B, I = x.shape
    H = W.shape[1]
    cell = torch.nn.RNNCell(H, H, nonlinearity="tanh").double()
    with torch.no_grad():
        cell.weight_ih.copy_(torch.eye(H, dtype=torch.float64))
        cell.weight_hh.zero_()
        cell.bias_ih.zero_()
        cell.bias_hh.zero_()
    cell.requires_grad_(False)
    xs, Wt, bt, h0t = _leaf(x), _leaf(W), _leaf(b), _leaf(h0)
    y, hT = np.zeros((T, B, H)), np.zeros((B, H))
    loss = 0.0
    for r in range(B):
        h = h0t[r:r + 1]
        for t in range(int(lens[r])):
            pre = rnd.prod(xs[t, r:r + 1], Wt[:I]) + rnd.prod(rnd.op(h), Wt[I:]) + bt
            h = cell(pre, h)
            loss = loss + (h * torch.from_numpy(dy[t, r:r + 1])).sum()
            y[t, r] = h.detach().numpy()[0]
        loss = loss + (h * torch.from_numpy(dhT[r:r + 1])).sum()
        hT[r] = h.detach().numpy()[0]
    loss.backward()
    return dict(y=y, hT=hT, dx=_grad(xs, x), dW=_grad(Wt, W), db=_grad(bt, b), dh0=_grad(h0t, h0))


def test_rnn_bf16_mode_rounds_where_the_kernels_do():
    rng = np.random.default_rng(9200)
    T, B, I, H = 7, 4, 3, 5
    x, lens, W, h0, _, dy, dhT, _ = _bf16_case(rng, T, B, I, H, 1, [7, 2, 0, 6])
    b = rng.uniform(-0.6, 0.6, H)
    y, hT, tape = oracle.rnn_forward(x, lens, W, b, h0, precision="bf16")
    g = oracle.rnn_backward(tape, dy, dhT)
    ref = dict(y=y, hT=hT, dx=g["dx"], dW=g["dW"], db=g["dbias"], dh0=g["dh0"])
    keys = ("y", "hT", "dx", "dW", "db", "dh0")
    _compare(_torch_rnn(x, lens, W, b, h0, dy, dhT, Rounding()), ref, keys)
    for off in (dict(h=False), dict(dz=False)):
        assert _spread(_torch_rnn(x, lens, W, b, h0, dy, dhT, Rounding(**off)), ref, keys) > 1e-5, off


# ------------------------------------------------------------------ GRU
def _gru_step(xt, h, Wx, Wh, bx, bhn, rnd, H):
    """GRU with the reset gate after the recurrent product (gates r, u, n)."""
    zx = rnd.prod(xt, Wx) + bx
    zh = rnd.prod(rnd.op(h), Wh)
    r = torch.sigmoid(zx[:, :H] + zh[:, :H])
    u = torch.sigmoid(zx[:, H:2 * H] + zh[:, H:2 * H])
    n = torch.tanh(zx[:, 2 * H:] + r * (zh[:, 2 * H:] + bhn))
    return (1.0 - u) * n + u * h


def test_gru_step_formula_is_torch_gru_cell():
    """The GRU step used below, without rounding, against torch.nn.GRUCell."""
    rng = np.random.default_rng(9300)
    B, I, H = 4, 3, 5
    x = torch.from_numpy(rng.standard_normal((B, I)))
    h = torch.from_numpy(rng.standard_normal((B, H)))
    W = torch.from_numpy(rng.uniform(-0.6, 0.6, (I + H, 3 * H)))
    b = torch.from_numpy(rng.uniform(-0.6, 0.6, 4 * H))
    cell = torch.nn.GRUCell(I, H).double()
    with torch.no_grad():
        cell.weight_ih.copy_(W[:I].T)
        cell.weight_hh.copy_(W[I:].T)
        cell.bias_ih.copy_(b[:3 * H])
        cell.bias_hh.zero_()
        cell.bias_hh[2 * H:] = b[3 * H:]
    got = _gru_step(x, h, W[:I], W[I:], b[:3 * H], b[3 * H:], Rounding(h=False, dz=False), H)
    np.testing.assert_allclose(got.numpy(), cell(x, h).detach().numpy(), rtol=0, atol=1e-14)


def _torch_gru(x, lens, W, b, h0, dy, dhT, rnd):
    T, B, I = x.shape
    H = W.shape[1] // 3
    xs, Wt, bt, h0t = _leaf(x), _leaf(W), _leaf(b), _leaf(h0)
    y, hT = np.zeros((T, B, H)), np.zeros((B, H))
    loss = 0.0
    for r in range(B):
        h = h0t[r:r + 1]
        for t in range(int(lens[r])):
            h = _gru_step(xs[t, r:r + 1], h, Wt[:I], Wt[I:], bt[:3 * H], bt[3 * H:], rnd, H)
            loss = loss + (h * torch.from_numpy(dy[t, r:r + 1])).sum()
            y[t, r] = h.detach().numpy()[0]
        loss = loss + (h * torch.from_numpy(dhT[r:r + 1])).sum()
        hT[r] = h.detach().numpy()[0]
    loss.backward()
    return dict(y=y, hT=hT, dx=_grad(xs, x), dW=_grad(Wt, W), db=_grad(bt, b), dh0=_grad(h0t, h0))


def test_gru_bf16_mode_rounds_where_the_kernels_do():
    rng = np.random.default_rng(9301)
    T, B, I, H = 6, 4, 3, 4
    x, lens, W, h0, _, dy, dhT, _ = _bf16_case(rng, T, B, I, H, 3, [6, 1, 0, 4])
    b = rng.uniform(-0.6, 0.6, 4 * H)
    y, hT, tape = oracle.gru_forward(x, lens, W, b, h0, precision="bf16")
    g = oracle.gru_backward(tape, dy, dhT)
    ref = dict(y=y, hT=hT, dx=g["dx"], dW=g["dW"], db=g["dbias"], dh0=g["dh0"])
    keys = ("y", "hT", "dx", "dW", "db", "dh0")
    _compare(_torch_gru(x, lens, W, b, h0, dy, dhT, Rounding()), ref, keys)
    for off in (dict(h=False), dict(dz=False)):
        assert _spread(_torch_gru(x, lens, W, b, h0, dy, dhT, Rounding(**off)), ref, keys) > 1e-5, off


# ------------------------------------------------------------------ cond body
def _skip_guard(xt, h, wp, bp):
    """The predicate in float32 on the operand forms (the oracle's decision
    rule): s = (x.w_px + op(h).w_ph) + b_p with w_p rounded."""
    I = xt.shape[0]
    wpr = oracle.bf16_round(wp)
    sx = np.asarray(xt, np.float32) @ np.asarray(wpr[:I], np.float32)
    sh = np.asarray(oracle.bf16_round(h), np.float32) @ np.asarray(wpr[I:], np.float32)
    return float((sx + sh) + np.float32(bp)) > 0


def _torch_skip(x, lens, W, bias, h0, c0, dy, dhT, dcT, rnd):
    """The cond body; each guard decided along this trajectory by the same
    float32 rule.  Returns outputs, gradients and the guards taken."""
    T, B, I = x.shape
    H = W.shape[1] // 4
    wp, bp = bias[4 * H:-1], bias[-1]
    cell = _lstm_cell(H)
    xs, Wt, h0t, c0t = _leaf(x), _leaf(W), _leaf(h0), _leaf(c0)
    bt = _leaf(bias[:4 * H])
    y, hT, cT = np.zeros((T, B, H)), np.zeros((B, H)), np.zeros((B, H))
    guards = np.zeros((T, B), bool)
    loss = 0.0
    for r in range(B):
        h, c = h0t[r:r + 1], c0t[r:r + 1]
        for t in range(int(lens[r])):
            guards[t, r] = _skip_guard(x[t, r], h.detach().numpy()[0], wp, bp)
            if guards[t, r]:
                pre = rnd.prod(xs[t, r:r + 1], Wt[:I]) + rnd.prod(rnd.op(h), Wt[I:]) + bt
                h, c = cell(pre, (h, c))
            loss = loss + (h * torch.from_numpy(dy[t, r:r + 1])).sum()
            y[t, r] = h.detach().numpy()[0]
        loss = loss + (h * torch.from_numpy(dhT[r:r + 1])).sum() + (c * torch.from_numpy(dcT[r:r + 1])).sum()
        hT[r], cT[r] = h.detach().numpy()[0], c.detach().numpy()[0]
    loss.backward()
    return dict(y=y, hT=hT, cT=cT, dx=_grad(xs, x), dW=_grad(Wt, W), db=_grad(bt, bias[:4 * H]),
                dh0=_grad(h0t, h0), dc0=_grad(c0t, c0), guards=guards)


SKIP_KEYS = ("y", "hT", "cT", "dx", "dW", "db", "dh0", "dc0")


def test_cond_body_bf16_mode_rounds_where_the_kernels_do():
    rng = np.random.default_rng(9400)
    T, B, I, H = 8, 5, 4, 3
    x, lens, W, h0, c0, dy, dhT, dcT = _bf16_case(rng, T, B, I, H, 4, [8, 4, 0, 7, 2])
    bias = np.concatenate([rng.uniform(-0.6, 0.6, 4 * H), rng.uniform(-1.5, 1.5, I + H), [0.0]])
    y, hT, cT, tape = oracle.skip_forward(x, lens, W, bias, h0, c0, precision="bf16")
    g = oracle.skip_backward(tape, dy, dhT, dcT)
    valid = np.arange(T)[:, None] < lens[None, :]
    assert tape["guards"][valid].any() and not tape["guards"][valid].all()   # both branches taken
    assert tape["min_margin"] > 1e-6
    ref = dict(y=y, hT=hT, cT=cT, dx=g["dx"], dW=g["dW"], db=g["dbias"][:4 * H], dh0=g["dh0"], dc0=g["dc0"])
    got = _torch_skip(x, lens, W, bias, h0, c0, dy, dhT, dcT, Rounding())
    np.testing.assert_array_equal(got["guards"][valid], tape["guards"][valid])
    _compare(got, ref, SKIP_KEYS)
    assert not g["dbias"][4 * H:].any()
    for off in (dict(h=False), dict(dz=False)):
        other = _torch_skip(x, lens, W, bias, h0, c0, dy, dhT, dcT, Rounding(**off))
        assert _spread(other, ref, SKIP_KEYS) > 1e-5, off


# ------------------------------------------------------------------ nested loop (ACT)
def _act_halt(h, wp, bp):
    """Halting probability in float32 on the operand forms (the oracle's rule)."""
    s = np.float32(np.asarray(oracle.bf16_round(h), np.float32) @ np.asarray(oracle.bf16_round(wp), np.float32))
    s = s + np.float32(bp)
    return np.float32(1.0) / (np.float32(1.0) + np.exp(-np.float32(s)))


def _torch_act(x, lens, W, bias, h0, c0, dy, dhT, dcT, M, rnd):
    """The nested loop, both loops in Python, trip counts decided along this
    trajectory by the same float32 rule."""
    T, B, I = x.shape
    H = W.shape[1] // 4
    wp, bp = bias[4 * H:5 * H], bias[-1]
    eps = np.float32(1.0 - oracle.ACT_EPS)
    cell = _lstm_cell(H)
    xs, Wt, h0t, c0t = _leaf(x), _leaf(W), _leaf(h0), _leaf(c0)
    bt = _leaf(bias[:4 * H])
    y, hT, cT = np.zeros((T, B, H)), np.zeros((B, H)), np.zeros((B, H))
    trips = np.zeros((T, B), np.int64)
    loss = 0.0
    for r in range(B):
        h, c = h0t[r:r + 1], c0t[r:r + 1]
        for t in range(int(lens[r])):
            P, n = np.float32(0.0), 0
            while True:
                pre = rnd.prod(xs[t, r:r + 1], Wt[:I]) + rnd.prod(rnd.op(h), Wt[I:]) + bt
                h, c = cell(pre, (h, c))
                n += 1
                if n == M:
                    break
                P = np.float32(P + _act_halt(h.detach().numpy()[0], wp, bp))
                if P >= eps:
                    break
            trips[t, r] = n
            loss = loss + (h * torch.from_numpy(dy[t, r:r + 1])).sum()
            y[t, r] = h.detach().numpy()[0]
        loss = loss + (h * torch.from_numpy(dhT[r:r + 1])).sum() + (c * torch.from_numpy(dcT[r:r + 1])).sum()
        hT[r], cT[r] = h.detach().numpy()[0], c.detach().numpy()[0]
    loss.backward()
    return dict(y=y, hT=hT, cT=cT, dx=_grad(xs, x), dW=_grad(Wt, W), db=_grad(bt, bias[:4 * H]),
                dh0=_grad(h0t, h0), dc0=_grad(c0t, c0), trips=trips)


def test_nested_loop_bf16_mode_rounds_where_the_kernels_do():
    rng = np.random.default_rng(9500)
    T, B, I, H, M = 6, 5, 4, 3, 4
    x, lens, W, h0, c0, dy, dhT, dcT = _bf16_case(rng, T, B, I, H, 4, [6, 3, 0, 5, 1])
    bias = np.concatenate([rng.uniform(-0.6, 0.6, 4 * H), rng.uniform(-1.5, 1.5, H), [0.0]])
    y, hT, cT, tape = oracle.act_forward(x, lens, W, bias, h0, c0, precision="bf16", ponder_max=M)
    g = oracle.act_backward(tape, dy, dhT, dcT)
    valid = np.arange(T)[:, None] < lens[None, :]
    assert len(np.unique(tape["trips"][valid])) >= 2   # the nested loop really varies
    assert tape["min_margin"] > 1e-6
    ref = dict(y=y, hT=hT, cT=cT, dx=g["dx"], dW=g["dW"], db=g["dbias"][:4 * H], dh0=g["dh0"], dc0=g["dc0"])
    got = _torch_act(x, lens, W, bias, h0, c0, dy, dhT, dcT, M, Rounding())
    np.testing.assert_array_equal(got["trips"], tape["trips"])
    _compare(got, ref, SKIP_KEYS)
    assert not g["dbias"][4 * H:].any()
    for off in (dict(h=False), dict(dz=False)):
        other = _torch_act(x, lens, W, bias, h0, c0, dy, dhT, dcT, M, Rounding(**off))
        assert _spread(other, ref, SKIP_KEYS) > 1e-5, off
