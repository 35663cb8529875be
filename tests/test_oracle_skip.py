"""Pins for the oracle of the loop whose LSTM body holds a data-dependent cond
(a row runs the cell or keeps its state, decided from x_t and h_{t-1} every
step).

- torch (CPU, float64): torch.nn.LSTMCell for the true branch, a Python
  branch on the predicate, autograd through the data-dependent control flow,
  sequence by sequence at its own length: an independent implementation of
  the step and of the cond gradient's bookkeeping.
- closed forms: a predicate that always holds gives the plain LSTM loop
  (the LSTM oracle, itself pinned against torch.nn.LSTM); one that never
  holds keeps the initial state, with dh0 = dhT + the sum of dy over the
  valid steps, dc0 = dcT and zero dW, db, dx.
- central finite differences in float64 (cases whose decisions all sit far
  from the threshold, so no perturbation flips one).
- the batched form equals the per-sequence literal form; zero trip count.
"""
import numpy as np
import pytest
import torch

import oracle


def _case(rng, T=6, B=5, I=3, H=4, lens=None, scale=0.6, bp=0.0):
    x = rng.standard_normal((T, B, I))
    W = rng.uniform(-scale, scale, (I + H, 4 * H))
    b = rng.uniform(-scale, scale, 4 * H)
    wp = rng.standard_normal(I + H)
    bias = np.concatenate([b, wp, [bp]])
    if lens is None:
        lens = rng.integers(0, T + 1, B)
    h0 = 0.5 * rng.standard_normal((B, H))
    c0 = 0.5 * rng.standard_normal((B, H))
    return x, np.asarray(lens, np.int64), W, bias, h0, c0


def _guard(xt, h, wp, bp):
    # the predicate in float32, as the oracle and the kernel decide it
    I = len(xt)
    sx = np.asarray(xt, np.float32) @ np.asarray(wp[:I], np.float32)
    sh = np.asarray(h, np.float32) @ np.asarray(wp[I:], np.float32)
    return float((sx + sh) + np.float32(bp)) > 0


def test_forward_backward_match_torch_per_sequence():
    rng = np.random.default_rng(61)
    T, B, I, H = 9, 5, 4, 3
    x, _, W, bias, h0, c0 = _case(rng, T, B, I, H)
    lens = np.array([9, 4, 0, 7, 1])
    dy = rng.standard_normal((T, B, H))
    dhT = rng.standard_normal((B, H))
    dcT = rng.standard_normal((B, H))
    y, hT, cT, tape = oracle.skip_forward(x, lens, W, bias, h0, c0)
    assert tape["min_margin"] > 1e-6
    valid = np.arange(T)[:, None] < lens[None, :]
    assert tape["guards"][valid].any() and not tape["guards"][valid].all()   # both branches taken
    g = oracle.skip_backward(tape, dy, dhT, dcT)
    wp, bp = bias[4 * H:-1], bias[-1]
    dW = np.zeros_like(W)
    db = np.zeros(4 * H)
    for r in range(B):
        n = int(lens[r])
        cell = torch.nn.LSTMCell(I, H).double()
        with torch.no_grad():
            cell.weight_ih.copy_(torch.from_numpy(W[:I].T))
            cell.weight_hh.copy_(torch.from_numpy(W[I:].T))
            cell.bias_ih.copy_(torch.from_numpy(bias[:4 * H]))
            cell.bias_hh.zero_()
        xt = torch.from_numpy(x[:, r].copy()).requires_grad_(True)
        h = h0t = torch.from_numpy(h0[r].copy()).requires_grad_(True)
        c = c0t = torch.from_numpy(c0[r].copy()).requires_grad_(True)
        loss = 0.0
        for t in range(n):
            run = _guard(x[t, r], h.detach().numpy(), wp, bp)
            assert run == bool(tape["guards"][t, r])
            if run:
                h, c = cell(xt[t][None], (h[None], c[None]))
                h, c = h[0], c[0]
            loss = loss + (h * torch.from_numpy(dy[t, r])).sum()
            np.testing.assert_allclose(y[t, r], h.detach().numpy(), rtol=0, atol=1e-13)
        assert not y[n:, r].any()
        np.testing.assert_allclose(hT[r], h.detach().numpy(), rtol=0, atol=1e-13)
        np.testing.assert_allclose(cT[r], c.detach().numpy(), rtol=0, atol=1e-13)
        loss = loss + (h * torch.from_numpy(dhT[r])).sum() + (c * torch.from_numpy(dcT[r])).sum()
        loss.backward()
        gx = xt.grad.numpy() if xt.grad is not None else np.zeros_like(x[:, r])
        np.testing.assert_allclose(g["dx"][:, r], gx, rtol=0, atol=1e-12)
        np.testing.assert_allclose(g["dh0"][r], h0t.grad.numpy(), rtol=0, atol=1e-12)
        np.testing.assert_allclose(g["dc0"][r], c0t.grad.numpy(), rtol=0, atol=1e-12)
        if cell.weight_ih.grad is not None:
            dW[:I] += cell.weight_ih.grad.numpy().T
            dW[I:] += cell.weight_hh.grad.numpy().T
            db += cell.bias_ih.grad.numpy()
    np.testing.assert_allclose(g["dW"], dW, rtol=0, atol=1e-12)
    np.testing.assert_allclose(g["dbias"][:4 * H], db, rtol=0, atol=1e-12)
    assert not g["dbias"][4 * H:].any()


def test_always_true_predicate_is_the_plain_lstm_loop():
    rng = np.random.default_rng(62)
    x, lens, W, bias, h0, c0 = _case(rng, T=7, B=6, I=4, H=5)
    H = 5
    bias[4 * H:-1] = 0.0
    bias[-1] = 1.0                        # s = 1 > 0 for every row and step
    dy = rng.standard_normal((7, 6, H))
    for precision in ("fp64", "bf16"):
        y, hT, cT, tape = oracle.skip_forward(x, lens, W, bias, h0, c0, precision)
        y2, hT2, cT2, tape2 = oracle.lstm_forward(x, lens, W, bias[:4 * H], h0, c0, precision)
        for a, b_ in ((y, y2), (hT, hT2), (cT, cT2)):
            np.testing.assert_allclose(a, b_, rtol=0, atol=1e-14)
        g = oracle.skip_backward(tape, dy)
        g2 = oracle.lstm_backward(tape2, dy)
        for k in ("dx", "dW", "dh0", "dc0"):
            np.testing.assert_allclose(g[k], g2[k], rtol=0, atol=1e-13, err_msg=k)
        np.testing.assert_allclose(g["dbias"][:4 * H], g2["dbias"], rtol=0, atol=1e-13)


def test_never_true_predicate_keeps_the_state():
    rng = np.random.default_rng(63)
    T, B, H = 6, 5, 4
    x, lens, W, bias, h0, c0 = _case(rng, T=T, B=B, I=3, H=H, lens=[6, 3, 0, 1, 5])
    bias[4 * H:-1] = 0.0
    bias[-1] = -1.0
    dy = rng.standard_normal((T, B, H))
    dhT = rng.standard_normal((B, H))
    dcT = rng.standard_normal((B, H))
    y, hT, cT, tape = oracle.skip_forward(x, lens, W, bias, h0, c0)
    assert not tape["guards"].any()
    valid = np.arange(T)[:, None] < lens[None, :]
    np.testing.assert_array_equal(y, np.where(valid[:, :, None], h0[None], 0.0))
    np.testing.assert_array_equal(hT, h0)
    np.testing.assert_array_equal(cT, c0)
    g = oracle.skip_backward(tape, dy, dhT, dcT)
    assert not g["dW"].any() and not g["dbias"].any() and not g["dx"].any()
    np.testing.assert_allclose(g["dh0"], dhT + (dy * valid[:, :, None]).sum(axis=0), rtol=0, atol=1e-14)
    np.testing.assert_array_equal(g["dc0"], dcT)


def test_batched_equals_literal():
    rng = np.random.default_rng(64)
    x, lens, W, bias, h0, c0 = _case(rng, T=8, B=7, I=4, H=6)
    for precision in ("fp64", "bf16"):
        y, hT, cT, _ = oracle.skip_forward(x, lens, W, bias, h0, c0, precision)
        y_l, hT_l, cT_l = oracle.skip_forward_literal(x, lens, W, bias, h0, c0, precision)
        for a, b_ in ((y, y_l), (hT, hT_l), (cT, cT_l)):
            np.testing.assert_allclose(a, b_, rtol=0, atol=1e-14)


def test_zero_trip_returns_inits_and_passes_gradients():
    rng = np.random.default_rng(65)
    x, _, W, bias, h0, c0 = _case(rng, T=4, B=3, I=2, H=3, lens=[0, 0, 0])
    y, hT, cT, tape = oracle.skip_forward(x, np.zeros(3, np.int64), W, bias, h0, c0)
    assert tape["T_eff"] == 0 and not y.any()
    np.testing.assert_array_equal(hT, h0)
    np.testing.assert_array_equal(cT, c0)
    dhT = rng.standard_normal((3, 3))
    dcT = rng.standard_normal((3, 3))
    g = oracle.skip_backward(tape, rng.standard_normal((4, 3, 3)), dhT, dcT)
    np.testing.assert_array_equal(g["dh0"], dhT)
    np.testing.assert_array_equal(g["dc0"], dcT)
    assert not g["dW"].any() and not g["dbias"].any() and not g["dx"].any()


def _loss(x, lens, W, bias, h0, c0, dy, dhT, dcT):
    y, hT, cT, _ = oracle.skip_forward(x, lens, W, bias, h0, c0)
    return float((y * dy).sum() + (hT * dhT).sum() + (cT * dcT).sum())


@pytest.mark.parametrize("seed", [71, 72])
def test_gradients_match_central_differences(seed):
    rng = np.random.default_rng(seed)
    T, B, H = 5, 3, 2
    x, _, W, bias, h0, c0 = _case(rng, T=T, B=B, I=3, H=H)
    lens = np.array([5, 3, 0])
    dy = rng.standard_normal((T, B, H))
    dhT = rng.standard_normal((B, H))
    dcT = rng.standard_normal((B, H))
    _, _, _, tape = oracle.skip_forward(x, lens, W, bias, h0, c0)
    assert tape["min_margin"] > 1e-3      # no perturbation below flips a decision
    g = oracle.skip_backward(tape, dy, dhT, dcT)
    eps = 1e-6
    args = dict(x=x, W=W, bias=bias, h0=h0, c0=c0)
    names = dict(x="dx", W="dW", bias="dbias", h0="dh0", c0="dc0")
    for key, arr in args.items():
        num = np.zeros_like(arr)
        it = np.nditer(arr, flags=["multi_index"])
        for _ in it:
            idx = it.multi_index
            a_p = {k: v.copy() for k, v in args.items()}
            a_m = {k: v.copy() for k, v in args.items()}
            a_p[key][idx] += eps
            a_m[key][idx] -= eps
            lp = _loss(a_p["x"], lens, a_p["W"], a_p["bias"], a_p["h0"], a_p["c0"], dy, dhT, dcT)
            lm = _loss(a_m["x"], lens, a_m["W"], a_m["bias"], a_m["h0"], a_m["c0"], dy, dhT, dcT)
            num[idx] = (lp - lm) / (2 * eps)
        np.testing.assert_allclose(g[names[key]], num, rtol=1e-6, atol=1e-8, err_msg=key)


def test_bf16_mode_rounds_and_stays_close():
    rng = np.random.default_rng(66)
    x, lens, W, bias, h0, c0 = _case(rng, T=6, B=5, I=4, H=8, scale=0.3)
    x = oracle.bf16_round(x)
    W = oracle.bf16_round(W)
    y64, _, _, t64 = oracle.skip_forward(x, lens, W, bias, h0, c0)
    y16, _, _, t16 = oracle.skip_forward(x, lens, W, bias, h0, c0, precision="bf16")
    np.testing.assert_array_equal(t64["guards"], t16["guards"])
    err = np.abs(y16 - y64).max()
    assert 0 < err < 2e-2
