"""The loop kernels' activation functions against float64 (through the C ABI
diagnostic ll_eval_activations, which runs the kernels' own device functions).

Bounds, from the operations each form uses (float ulp u = 2^-23):
- sigmoid(v) = 1 / (1 + e^-v): the rounding of the exponent's argument gives
  a relative error of about |v| 2^-24 in e^-v, plus the exponential, the sum
  and the reciprocal, each within one ulp: relative error <= (|v| + 8) u.
- tanh(v) = 1 - 2 / (1 + e^{2v}) for |v| >= 1/8: the same terms in q =
  2 / (1 + e^{2v}) <= 0.9, made relative to |tanh(v)| >= 0.124:
  relative error <= (8 |v| + 16) u; below 1/8 the Taylor form: <= 8 u.
Relative error is taken where the float64 value is a normal float32.
"""
import numpy as np
import pytest
import torch

from paper_1805_01772_amd.lstmloop import LL_EINVAL, ll_eval_activations, load_library

pytestmark = pytest.mark.gpu

U = 2.0 ** -23


def _inputs():
    rng = np.random.default_rng(5)
    mags = np.concatenate([10.0 ** rng.uniform(-30, 2, 200000), rng.uniform(0, 0.25, 100000),
                           rng.uniform(0, 90, 100000), [0.0, 0.125, 0.12499999, 1e-38, 1e-45]])
    v = np.concatenate([mags, -mags]).astype(np.float32)
    return v


def _rel(got, ref):
    return np.abs(got.astype(np.float64) - ref) / np.abs(ref)


def test_sigmoid_against_float64():
    v = _inputs()
    got = ll_eval_activations(torch.from_numpy(v).cuda(), "sigmoid").cpu().numpy()
    ref = 1.0 / (1.0 + np.exp(-v.astype(np.float64)))
    ok = ref >= np.finfo(np.float32).tiny
    rel = _rel(got[ok], ref[ok])
    bound = (np.abs(v[ok]).astype(np.float64) + 8.0) * U
    worst = int(np.argmax(rel / bound))
    print(f"sigmoid: max rel err {rel.max():.3e}; worst vs bound at v={v[ok][worst]:.4g}: "
          f"{rel[worst]:.3e} <= {bound[worst]:.3e}")
    assert (rel <= bound).all()
    assert np.all(got[v > 90] == 1.0) and np.all(np.isfinite(got))
    assert np.all((got >= 0) & (got <= 1))


def test_tanh_against_float64():
    v = _inputs()
    got = ll_eval_activations(torch.from_numpy(v).cuda(), "tanh").cpu().numpy()
    ref = np.tanh(v.astype(np.float64))
    ok = np.abs(ref) >= np.finfo(np.float32).tiny
    rel = _rel(got[ok], ref[ok])
    a = np.abs(v[ok]).astype(np.float64)
    bound = np.where(a < 0.125, 8.0 * U, (8.0 * a + 16.0) * U)
    worst = int(np.argmax(rel / bound))
    print(f"tanh: max rel err {rel.max():.3e}; worst vs bound at v={v[ok][worst]:.4g}: "
          f"{rel[worst]:.3e} <= {bound[worst]:.3e}")
    assert (rel <= bound).all()
    assert np.all(got[v == 0] == 0.0)
    np.testing.assert_array_equal(got[v > 20], 1.0)
    np.testing.assert_array_equal(got[v < -20], -1.0)
    # the Taylor form is odd bit for bit
    pos = (v > 0) & (v < 0.125)
    neg = ll_eval_activations(torch.from_numpy(-v[pos]).cuda(), "tanh").cpu().numpy()
    np.testing.assert_array_equal(neg, -got[pos])


def test_bad_function_code():
    x = torch.zeros(4, device="cuda")
    lib = load_library()
    assert lib.ll_eval_activations(0, x.data_ptr(), x.data_ptr(), 4, 2) == LL_EINVAL
    assert lib.ll_eval_activations(0, x.data_ptr(), x.data_ptr(), -1, 0) == LL_EINVAL
