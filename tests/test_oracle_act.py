"""Pins for the oracle of the loop whose LSTM body holds a nested while-loop
(ACT's halting rule decides how many times the body ponders each input).

- torch (CPU, float64): torch.nn.LSTMCell inside two Python while loops,
  the inner trip count decided by the halting rule in float32, autograd
  through the nested data-dependent loops, sequence by sequence: an
  independent implementation of the ponder steps and of the nested
  gradient's bookkeeping.
- closed forms against the LSTM oracle (itself pinned against
  torch.nn.LSTM): at most one ponder step, or a halting unit that always
  halts at once, is the plain LSTM loop; a halting unit that never halts
  gives M ponder steps of every input, i.e. the LSTM loop over x with every
  x_t repeated M times (y_t its last ponder state, dx_t the sum of the
  repeats' dx).
- central finite differences in float64 (no decision near the threshold).
- the batched form equals the per-sequence literal form (float64 and
  bfloat16 modes); the trip counts lie in [1, M]; zero trip count.
"""
import numpy as np
import pytest
import torch

import oracle

EPS = oracle.ACT_EPS


def _case(rng, T=6, B=5, I=3, H=4, lens=None, scale=0.6, wp_scale=1.5, bp=0.0):
    x = rng.standard_normal((T, B, I))
    W = rng.uniform(-scale, scale, (I + H, 4 * H))
    b = rng.uniform(-scale, scale, 4 * H)
    wp = rng.uniform(-wp_scale, wp_scale, H)
    bias = np.concatenate([b, wp, [bp]])
    if lens is None:
        lens = rng.integers(0, T + 1, B)
    h0 = 0.5 * rng.standard_normal((B, H))
    c0 = 0.5 * rng.standard_normal((B, H))
    return x, np.asarray(lens, np.int64), W, bias, h0, c0


def _halt(h, wp, bp):
    """float32 halting probability (the rule's precision)."""
    s = np.float32(np.asarray(h, np.float32) @ np.asarray(wp, np.float32)) + np.float32(bp)
    return np.float32(1.0) / (np.float32(1.0) + np.exp(-np.float32(s)))


def _torch_reference(x, lens, W, bias, h0, c0, dy, dhT, dcT, M):
    """Forward outputs and gradients from torch autograd, one sequence at a time."""
    T, B, I = x.shape
    H = W.shape[1] // 4
    wp, bp = bias[4 * H:5 * H], bias[-1]
    cell = torch.nn.LSTMCell(I, H).double()
    with torch.no_grad():
        cell.weight_ih.copy_(torch.from_numpy(W[:I].T.copy()))
        cell.weight_hh.copy_(torch.from_numpy(W[I:].T.copy()))
        cell.bias_ih.copy_(torch.from_numpy(bias[:4 * H].copy()))
        cell.bias_hh.zero_()
    xs = torch.from_numpy(x).requires_grad_(True)
    hs0 = torch.from_numpy(h0).requires_grad_(True)
    cs0 = torch.from_numpy(c0).requires_grad_(True)
    y = torch.zeros(T, B, H, dtype=torch.float64)
    hT, cT, trips = [], [], np.zeros((T, B), np.int64)
    loss = 0.0
    for r in range(B):
        h, c = hs0[r:r + 1], cs0[r:r + 1]
        t = 0
        while t < lens[r]:
            P, n = np.float32(0.0), 0
            while True:
                h, c = cell(xs[t, r:r + 1], (h, c))
                n += 1
                if n == M:
                    break
                P = np.float32(P + _halt(h.detach().numpy()[0], wp, bp))
                if P >= np.float32(1.0 - EPS):
                    break
            trips[t, r] = n
            loss = loss + (h[0] * torch.from_numpy(dy[t, r])).sum()
            y[t, r] = h[0].detach()
            t += 1
        loss = loss + (h[0] * torch.from_numpy(dhT[r])).sum() + (c[0] * torch.from_numpy(dcT[r])).sum()
        hT.append(h[0].detach().numpy())
        cT.append(c[0].detach().numpy())
    loss.backward()
    dW = np.concatenate([cell.weight_ih.grad.numpy().T, cell.weight_hh.grad.numpy().T])
    return dict(y=y.numpy(), hT=np.array(hT), cT=np.array(cT), trips=trips, dx=xs.grad.numpy(),
                dW=dW, db=cell.bias_ih.grad.numpy(), dh0=hs0.grad.numpy(), dc0=cs0.grad.numpy())


@pytest.mark.parametrize("M", [1, 3, 5])
def test_forward_backward_match_torch_per_sequence(M):
    rng = np.random.default_rng(71 + M)
    T, B, I, H = 7, 5, 4, 3
    x, _, W, bias, h0, c0 = _case(rng, T, B, I, H)
    lens = np.array([7, 3, 0, 6, 1])
    dy = rng.standard_normal((T, B, H))
    dhT = rng.standard_normal((B, H))
    dcT = rng.standard_normal((B, H))
    y, hT, cT, tape = oracle.act_forward(x, lens, W, bias, h0, c0, ponder_max=M)
    assert tape["min_margin"] > 1e-6
    g = oracle.act_backward(tape, dy, dhT, dcT)
    ref = _torch_reference(x, lens, W, bias, h0, c0, dy, dhT, dcT, M)
    np.testing.assert_array_equal(tape["trips"], ref["trips"])
    valid = np.arange(T)[:, None] < lens[None, :]
    if M > 2:   # the nested loop really varies: several trip counts occur
        assert len(np.unique(tape["trips"][valid])) >= 2
    for k, v in (("y", y), ("hT", hT), ("cT", cT), ("dx", g["dx"]), ("dW", g["dW"]),
                 ("db", g["dbias"][:4 * H]), ("dh0", g["dh0"]), ("dc0", g["dc0"])):
        np.testing.assert_allclose(v, ref[k], rtol=1e-10, atol=1e-12, err_msg=k)
    assert not g["dbias"][4 * H:].any()


def test_one_ponder_step_is_the_lstm_loop():
    rng = np.random.default_rng(81)
    x, lens, W, bias, h0, c0 = _case(rng, 8, 6, 3, 5)
    H = 5
    dy = rng.standard_normal((8, 6, H))
    for M, bp in ((1, 0.0), (4, 40.0)):      # at most one step; or halting at once
        b2 = bias.copy()
        b2[-1] = bp
        b2[4 * H:5 * H] = 0.0 if bp else b2[4 * H:5 * H]
        y, hT, cT, tape = oracle.act_forward(x, lens, W, b2, h0, c0, ponder_max=M)
        g = oracle.act_backward(tape, dy, hT * 0 + 1, cT * 0)
        yl, hl, cl, tl = oracle.lstm_forward(x, lens, W, b2[:4 * H], h0, c0)
        gl = oracle.lstm_backward(tl, dy, hl * 0 + 1, cl * 0)
        valid = np.arange(8)[:, None] < lens[None, :]
        assert (tape["trips"][valid] == 1).all()
        for a, r in ((y, yl), (hT, hl), (cT, cl), (g["dx"], gl["dx"]), (g["dW"], gl["dW"]),
                     (g["dbias"][:4 * H], gl["dbias"]), (g["dh0"], gl["dh0"]), (g["dc0"], gl["dc0"])):
            np.testing.assert_allclose(a, r, rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("M", [2, 3])
def test_never_halting_is_the_lstm_loop_over_repeated_inputs(M):
    """w_p = 0, b_p = -40: the summed halting probability never reaches
    1 - eps, so every input is pondered M times."""
    rng = np.random.default_rng(91 + M)
    T, B, I, H = 5, 4, 3, 4
    x, lens, W, bias, h0, c0 = _case(rng, T, B, I, H)
    bias[4 * H:5 * H] = 0.0
    bias[-1] = -40.0
    dy = rng.standard_normal((T, B, H))
    dhT = rng.standard_normal((B, H))
    dcT = rng.standard_normal((B, H))
    y, hT, cT, tape = oracle.act_forward(x, lens, W, bias, h0, c0, ponder_max=M)
    g = oracle.act_backward(tape, dy, dhT, dcT)
    valid = np.arange(T)[:, None] < lens[None, :]
    assert (tape["trips"][valid] == M).all()
    xr = np.repeat(x, M, axis=0)                       # x_t at steps M t .. M t + M - 1
    dyr = np.zeros((T * M, B, H))
    dyr[M - 1::M] = dy                                  # y_t is the last ponder state
    yl, hl, cl, tl = oracle.lstm_forward(xr, lens * M, W, bias[:4 * H], h0, c0)
    gl = oracle.lstm_backward(tl, dyr, dhT, dcT)
    np.testing.assert_allclose(y, yl[M - 1::M], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(hT, hl, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(cT, cl, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(g["dx"], gl["dx"].reshape(T, M, B, I).sum(axis=1), rtol=1e-10, atol=1e-12)
    for a, r in ((g["dW"], gl["dW"]), (g["dbias"][:4 * H], gl["dbias"]), (g["dh0"], gl["dh0"]),
                 (g["dc0"], gl["dc0"])):
        np.testing.assert_allclose(a, r, rtol=1e-10, atol=1e-12)


def test_gradients_match_central_differences():
    rng = np.random.default_rng(101)
    T, B, I, H, M = 5, 3, 3, 3, 4
    x, lens, W, bias, h0, c0 = _case(rng, T, B, I, H, lens=[5, 2, 4])
    dy = rng.standard_normal((T, B, H))
    dhT = rng.standard_normal((B, H))
    dcT = rng.standard_normal((B, H))

    def loss(x_, W_, b_, h0_, c0_):
        y, hT, cT, tape = oracle.act_forward(x_, lens, W_, b_, h0_, c0_, ponder_max=M)
        return (y * dy).sum() + (hT * dhT).sum() + (cT * dcT).sum(), tape

    base, tape = loss(x, W, bias, h0, c0)
    assert tape["min_margin"] > 1e-4
    assert len(np.unique(tape["trips"][np.arange(T)[:, None] < lens[None, :]])) >= 2
    g = oracle.act_backward(tape, dy, dhT, dcT)
    e = 1e-6
    checks = [("x", x, (2, 1, 0), g["dx"]), ("W", W, (1, 5), g["dW"]), ("W", W, (4, 2), g["dW"]),
              ("b", bias, (7,), g["dbias"]), ("h0", h0, (0, 2), g["dh0"]), ("c0", c0, (2, 1), g["dc0"])]
    for name, arr, idx, grad in checks:
        plus, minus = arr.copy(), arr.copy()
        plus[idx] += e
        minus[idx] -= e
        args = {"x": (x, W, bias, h0, c0)}
        def call(a):
            return loss(*[a if n == name else v for n, v in
                          zip(("x", "W", "b", "h0", "c0"), (x, W, bias, h0, c0))])[0]
        fd = (call(plus) - call(minus)) / (2 * e)
        assert abs(fd - grad[idx]) <= 1e-6 * max(1.0, abs(fd)), (name, idx, fd, grad[idx])


@pytest.mark.parametrize("precision", ["fp64", "bf16"])
def test_batched_equals_literal(precision):
    rng = np.random.default_rng(111)
    x, lens, W, bias, h0, c0 = _case(rng, 9, 7, 4, 5)
    if precision == "bf16":
        x = oracle.bf16_round(x)
        W = oracle.bf16_round(W)
    y, hT, cT, tape = oracle.act_forward(x, lens, W, bias, h0, c0, precision, ponder_max=4)
    yl, hl, cl, trips = oracle.act_forward_literal(x, lens, W, bias, h0, c0, precision, ponder_max=4)
    np.testing.assert_array_equal(tape["trips"], trips)
    valid = np.arange(9)[:, None] < lens[None, :]
    assert ((trips[valid] >= 1) & (trips[valid] <= 4)).all() and not trips[~valid].any()
    for a, r in ((y, yl), (hT, hl), (cT, cl)):
        np.testing.assert_allclose(a, r, rtol=1e-12, atol=1e-14)


def test_zero_trip_count_returns_the_inits():
    rng = np.random.default_rng(121)
    x, _, W, bias, h0, c0 = _case(rng, 4, 3, 3, 4)
    lens = np.zeros(3, np.int64)
    dhT = rng.standard_normal((3, 4))
    dcT = rng.standard_normal((3, 4))
    y, hT, cT, tape = oracle.act_forward(x, lens, W, bias, h0, c0, ponder_max=3)
    g = oracle.act_backward(tape, rng.standard_normal((4, 3, 4)), dhT, dcT)
    assert tape["T_eff"] == 0 and not y.any()
    np.testing.assert_array_equal(hT, h0)
    np.testing.assert_array_equal(cT, c0)
    np.testing.assert_array_equal(g["dh0"], dhT)
    np.testing.assert_array_equal(g["dc0"], dcT)
    assert not g["dW"].any() and not g["dx"].any() and not g["dbias"].any()
