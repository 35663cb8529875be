"""Pins for the GRU-cell oracle (the while-loop with a GRU body, reset gate
applied after the recurrent product).

- torch.nn.GRU (CPU, float64) forward and autograd backward, per sequence:
  an independent implementation of the same cell (gate order r, z, n;
  weight_ih = W[:I].T, weight_hh = W[I:].T, bias_ih = bias[:3H],
  bias_hh = [0, 0, bias[3H:]]).
- central finite differences in float64 for every gradient output.
- closed form: zero weights give h_t = n + u^t (h0 - n) with the constant
  gates u = sigmoid(b_u), n = tanh(b_n + sigmoid(b_r) b_hn).
- the loop semantics: zero trip count returns the inits and passes dhT
  through; the batched form equals the per-sequence literal form.
"""
import numpy as np
import pytest
import torch

import oracle


def _case(rng, T=6, B=5, I=3, H=4, lens=None, scale=0.6):
    x = rng.standard_normal((T, B, I))
    W = rng.uniform(-scale, scale, (I + H, 3 * H))
    b = rng.uniform(-scale, scale, 4 * H)
    if lens is None:
        lens = rng.integers(0, T + 1, B)
    h0 = 0.5 * rng.standard_normal((B, H))
    return x, np.asarray(lens, np.int64), W, b, h0


def _torch_gru_one(x_seq, W, b, h0, I):
    H = W.shape[1] // 3
    m = torch.nn.GRU(I, H, batch_first=False).double()
    with torch.no_grad():
        m.weight_ih_l0.copy_(torch.from_numpy(W[:I].T))
        m.weight_hh_l0.copy_(torch.from_numpy(W[I:].T))
        m.bias_ih_l0.copy_(torch.from_numpy(b[:3 * H]))
        m.bias_hh_l0.zero_()
        m.bias_hh_l0[2 * H:] = torch.from_numpy(b[3 * H:])
    xt = torch.from_numpy(x_seq[:, None, :].copy()).requires_grad_(True)
    h0t = torch.from_numpy(h0[None, None, :].copy()).requires_grad_(True)
    y, hn = m(xt, h0t)
    return m, xt, h0t, y[:, 0], hn[0, 0]


def test_forward_backward_match_torch_gru_per_sequence():
    rng = np.random.default_rng(51)
    T, B, I, H = 7, 4, 5, 3
    x, _, W, b, h0 = _case(rng, T, B, I, H)
    lens = np.array([7, 3, 1, 5])
    dy = rng.standard_normal((T, B, H))
    dhT = rng.standard_normal((B, H))
    y, hT, tape = oracle.gru_forward(x, lens, W, b, h0)
    g = oracle.gru_backward(tape, dy, dhT)
    dW = np.zeros_like(W)
    db = np.zeros_like(b)
    for r in range(B):
        n = int(lens[r])
        m, xt, h0t, yr, hn = _torch_gru_one(x[:n, r], W, b, h0[r], I)
        np.testing.assert_allclose(y[:n, r], yr.detach().numpy(), rtol=0, atol=1e-13)
        assert not y[n:, r].any()
        np.testing.assert_allclose(hT[r], hn.detach().numpy(), rtol=0, atol=1e-13)
        loss = (yr * torch.from_numpy(dy[:n, r])).sum() + (hn * torch.from_numpy(dhT[r])).sum()
        loss.backward()
        np.testing.assert_allclose(g["dx"][:n, r], xt.grad[:, 0].numpy(), rtol=0, atol=1e-12)
        assert not g["dx"][n:, r].any()
        np.testing.assert_allclose(g["dh0"][r], h0t.grad[0, 0].numpy(), rtol=0, atol=1e-12)
        dW[:I] += m.weight_ih_l0.grad.numpy().T
        dW[I:] += m.weight_hh_l0.grad.numpy().T
        db[:3 * H] += m.bias_ih_l0.grad.numpy()
        db[3 * H:] += m.bias_hh_l0.grad.numpy()[2 * H:]
    np.testing.assert_allclose(g["dW"], dW, rtol=0, atol=1e-12)
    np.testing.assert_allclose(g["dbias"], db, rtol=0, atol=1e-12)


def test_batched_equals_literal():
    rng = np.random.default_rng(52)
    x, lens, W, b, h0 = _case(rng, T=8, B=6, I=4, H=5)
    y, hT, _ = oracle.gru_forward(x, lens, W, b, h0)
    y_l, hT_l = oracle.gru_forward_literal(x, lens, W, b, h0)
    np.testing.assert_allclose(y, y_l, rtol=0, atol=1e-14)
    np.testing.assert_allclose(hT, hT_l, rtol=0, atol=1e-14)


def test_zero_weights_closed_form():
    rng = np.random.default_rng(53)
    H = 2
    x, lens, _, b, h0 = _case(rng, T=5, B=4, I=3, H=H, lens=[5, 2, 0, 1])
    W = np.zeros((3 + H, 3 * H))
    y, hT, _ = oracle.gru_forward(x, lens, W, b, h0)
    r_ = 1 / (1 + np.exp(-b[:H]))
    u_ = 1 / (1 + np.exp(-b[H:2 * H]))
    n_ = np.tanh(b[2 * H:3 * H] + r_ * b[3 * H:])
    for r in range(4):
        k = int(lens[r])
        for t in range(5):
            want = n_ + u_ ** (t + 1) * (h0[r] - n_) if t < k else np.zeros(H)
            np.testing.assert_allclose(y[t, r], want, rtol=0, atol=1e-14)
        want_T = n_ + u_ ** k * (h0[r] - n_)
        np.testing.assert_allclose(hT[r], want_T, rtol=0, atol=1e-14)


def test_zero_trip_returns_inits_and_passes_gradients():
    rng = np.random.default_rng(54)
    x, _, W, b, h0 = _case(rng, T=4, B=3, I=2, H=3)
    lens = np.zeros(3, np.int64)
    y, hT, tape = oracle.gru_forward(x, lens, W, b, h0)
    assert tape["T_eff"] == 0 and not y.any()
    np.testing.assert_array_equal(hT, h0)
    dhT = rng.standard_normal((3, 3))
    g = oracle.gru_backward(tape, rng.standard_normal((4, 3, 3)), dhT)
    np.testing.assert_array_equal(g["dh0"], dhT)
    assert not g["dW"].any() and not g["dbias"].any() and not g["dx"].any()


def _loss(x, lens, W, b, h0, dy, dhT):
    y, hT, _ = oracle.gru_forward(x, lens, W, b, h0)
    return float((y * dy).sum() + (hT * dhT).sum())


@pytest.mark.parametrize("seed", [61, 62])
def test_gradients_match_central_differences(seed):
    rng = np.random.default_rng(seed)
    x, _, W, b, h0 = _case(rng, T=5, B=3, I=3, H=2)
    lens = np.array([5, 2, 0])
    dy = rng.standard_normal((5, 3, 2))
    dhT = rng.standard_normal((3, 2))
    _, _, tape = oracle.gru_forward(x, lens, W, b, h0)
    g = oracle.gru_backward(tape, dy, dhT)
    eps = 1e-6
    args = dict(x=x, W=W, b=b, h0=h0)
    names = dict(x="dx", W="dW", b="dbias", h0="dh0")
    for key, arr in args.items():
        num = np.zeros_like(arr)
        it = np.nditer(arr, flags=["multi_index"])
        for _ in it:
            idx = it.multi_index
            a_p = {k: v.copy() for k, v in args.items()}
            a_m = {k: v.copy() for k, v in args.items()}
            a_p[key][idx] += eps
            a_m[key][idx] -= eps
            lp = _loss(a_p["x"], lens, a_p["W"], a_p["b"], a_p["h0"], dy, dhT)
            lm = _loss(a_m["x"], lens, a_m["W"], a_m["b"], a_m["h0"], dy, dhT)
            num[idx] = (lp - lm) / (2 * eps)
        np.testing.assert_allclose(g[names[key]], num, rtol=1e-6, atol=1e-8, err_msg=key)


def test_bf16_mode_rounds_and_stays_close():
    rng = np.random.default_rng(56)
    x, lens, W, b, h0 = _case(rng, T=6, B=5, I=4, H=8, scale=0.3)
    x = oracle.bf16_round(x)
    W = oracle.bf16_round(W)
    y64, _, t64 = oracle.gru_forward(x, lens, W, b, h0)
    y16, _, t16 = oracle.gru_forward(x, lens, W, b, h0, precision="bf16")
    err = np.abs(y16 - y64).max()
    assert 0 < err < 2e-2
    dy = rng.standard_normal(y64.shape)
    g64 = oracle.gru_backward(t64, dy)
    g16 = oracle.gru_backward(t16, dy)
    assert 0 < np.abs(g16["dW"] - g64["dW"]).max() < 2e-2 * np.abs(g64["dW"]).max()
