"""The inference forward that allocates nothing (lstm_loop_fwd_noalloc)
against the plan-based lstm_loop_fwd(save_for_backward = 0): two calls in a
row, the second on a smaller input (the scratch array keeps the first call's
contents), each bitwise equal to the plan's forward on the same inputs and
within the parity tolerance of the oracle; the limits and the device error
word through the same call."""
import numpy as np
import pytest
import torch

from paper_1805_01772_amd import lstmloop as ll
from paper_1805_01772_amd import workloads as wl
from paper_1805_01772_amd.runner import DeviceCase
from _helpers import TOL, compare, oracle_reference, say

pytestmark = pytest.mark.gpu

W = wl.Workload
CASES = [
    # larger first, then smaller: the second call must not see the first's leftovers
    W("noalloc_bf16_b64_i512_h512_t50", B=64, I=512, H=512, T_max=50, dtype="bf16", len_lo=0,
      len_hi=50, random_state=True, seed=301),
    W("noalloc_f32_b20_i24_h64_t13", B=20, I=24, H=64, T_max=13, dtype="f32", len_lo=0, len_hi=13,
      w_scale=0.3, random_state=True, seed=302),
]
FWD_KEYS = ("y", "hT", "cT")


def _desc(w):
    cell = {"lstm": ll.LL_CELL_LSTM, "rnn": ll.LL_CELL_RNN, "gru": ll.LL_CELL_GRU,
            "skip": ll.LL_CELL_LSTM_SKIP}[w.cell]
    return ll.make_desc(w.T_max, w.B, w.I, w.H, w.layers, w.dtype, cell=cell)


def _noalloc(dc, w):
    err = torch.full((4,), -1, dtype=torch.int32, device=dc.dev)
    for t in (dc.y, dc.hT, dc.cT):
        t.fill_(float("nan"))
    dc.trip.fill_(-1)
    ll.lstm_loop_fwd_noalloc(_desc(w), dc.x, dc.seq_len, dc.W, dc.bias, dc.h0, dc.c0, dc.y, dc.hT,
                             dc.cT, dc.trip, err)
    torch.cuda.synchronize()
    return {k: getattr(dc, k).cpu().numpy().astype(np.float64) for k in FWD_KEYS}, \
        int(dc.trip.item()), int(err[0].item())


def _plan_fwd(dc):
    plan = dc.plan()
    dc.fwd(plan, save=False)
    assert plan.status_sync() == 0
    plan.close()
    torch.cuda.synchronize()
    return {k: getattr(dc, k).cpu().numpy().astype(np.float64) for k in FWD_KEYS}, int(dc.trip.item())


def test_noalloc_forward_matches_the_plan_forward_twice():
    for w in CASES:
        say(f"[noalloc] {w.name}")
        inp = wl.generate(w)
        dc = DeviceCase(inp, w.H, w.I, w.layers, w.dtype)
        got, trip, derr = _noalloc(dc, w)
        ref, trip_ref = _plan_fwd(dc)
        assert derr == 0 and trip == trip_ref == int(inp["seq_len"].max())
        for k in FWD_KEYS:
            np.testing.assert_array_equal(got[k], ref[k], err_msg=k)
        o = oracle_reference(inp, w.layers, w.dtype)
        errs, bad = compare(got, o, TOL[w.dtype], keys=FWD_KEYS)
        say(f"    errors vs oracle {errs}")
        assert not bad, bad


def test_noalloc_limits_and_device_error():
    w = CASES[1]
    inp = wl.generate(w)
    dc = DeviceCase(inp, w.H, w.I, w.layers, w.dtype)
    # beyond the scratch array: the H = 1024 benchmark shape
    big = ll.make_desc(200, 128, 1024, 1024, 1, "bf16")
    with pytest.raises(ll.LoopError) as e:
        ll.lstm_loop_fwd_noalloc(big, dc.x, dc.seq_len, dc.W, dc.bias, None, None, dc.y, dc.hT, dc.cT)
    assert e.value.status == ll.LL_EUNSUPPORTED and "scratch" in str(e.value)
    with pytest.raises(ll.LoopError) as e:
        ll.lstm_loop_fwd_noalloc(ll.make_desc(w.T_max, w.B, w.I, w.H, spill=1), dc.x, dc.seq_len,
                                 dc.W, dc.bias, None, None, dc.y, dc.hT, dc.cT)
    assert e.value.status == ll.LL_EUNSUPPORTED
    # a length outside [0, T_max]: zero iterations, the error word set, the
    # state returned unchanged; the next call is clean again
    bad = inp["seq_len"].copy()
    bad[5] = w.T_max + 1
    dc.seq_len.copy_(torch.from_numpy(bad))
    got, trip, derr = _noalloc(dc, w)
    assert derr & ll.LL_DEVERR_SEQ_LEN and trip == 0
    np.testing.assert_array_equal(got["hT"][0], inp["h0"][0])
    assert not got["y"].any()
    dc.seq_len.copy_(torch.from_numpy(inp["seq_len"]))
    got, trip, derr = _noalloc(dc, w)
    assert derr == 0 and trip == int(inp["seq_len"].max())
