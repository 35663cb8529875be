"""GPU parity: the HIP loops (through the C ABI) against the CPU oracle.

Tolerance (per output tensor, max |gpu - oracle| / max |oracle|): 1e-5 for
float32 runs against the float64 oracle, 2e-2 for bfloat16-operand runs
against the bfloat16-emulating oracle.  Invariants that the method fixes
exactly (finished rows, zero-trip loops, per-row independence) are checked
bitwise between GPU runs.
"""
import numpy as np
import pytest
import torch

from paper_1805_01772_amd import workloads as wl
from paper_1805_01772_amd.lstmloop import LL_DEVERR_SEQ_LEN, LL_ESTATE, LoopError
from paper_1805_01772_amd.runner import DeviceCase
from _helpers import TOL, compare, oracle_reference, rel_err, say

pytestmark = pytest.mark.gpu

W = wl.Workload
SMALL = [
    wl.TINY,
    wl.TINY.with_(name="tiny_random_state_dy", random_state=True, with_dy=True, seed=7),
    W("f32_b37_i48_h64_t23", B=37, I=48, H=64, T_max=23, dtype="f32", len_lo=0, len_hi=23,
      w_scale=0.3, random_state=True, seed=11),
    W("bf16_b50_i64_h96_t19", B=50, I=64, H=96, T_max=19, dtype="bf16", len_lo=0, len_hi=19,
      w_scale=0.3, random_state=True, seed=12),
    W("f32_b1_i4_h32_t1", B=1, I=4, H=32, T_max=1, dtype="f32", len_lo=1, len_hi=1,
      random_state=True, seed=13),
    W("f32_b100_i32_h512_t9_mrt2", B=100, I=32, H=512, T_max=9, dtype="f32", len_lo=0,
      len_hi=9, random_state=True, seed=14),
    W("bf16_b200_i64_h1024_t6_mrt4", B=200, I=64, H=1024, T_max=6, dtype="bf16", len_lo=1,
      len_hi=6, random_state=True, seed=15),
    W("bf16_b250_i64_h2048_t3_mrt16", B=250, I=64, H=2048, T_max=3, dtype="bf16", len_lo=0,
      len_hi=3, random_state=True, seed=16),
    W("f32_2layer_b21_i40_h32_t11", B=21, I=40, H=32, T_max=11, dtype="f32", layers=2,
      len_lo=1, len_hi=11, w_scale=0.3, random_state=True, seed=17),
    W("bf16_2layer_b33_i32_h64_t9", B=33, I=32, H=64, T_max=9, dtype="bf16", layers=2,
      len_lo=0, len_hi=9, w_scale=0.3, random_state=True, seed=18),
    W("f32_b300_i16_h64_t5_ragged", B=300, I=16, H=64, T_max=5, dtype="f32", len_lo=0,
      len_hi=5, random_state=True, seed=19),
]


def run_case(w, inp, save=True, backward=True, with_dy=True, geometry=None):
    dc = DeviceCase(inp, w.H, w.I, w.layers, w.dtype)
    plan = dc.plan()
    geom = plan.geometry()
    say(f"    {w.name}: loops {geom}")
    if geometry is not None:
        geometry.update(geom)
    dc.fwd(plan, save=save)
    if backward:
        dc.bwd(plan, with_dy=with_dy)
    err = plan.status_sync()
    res = dc.results()
    plan.close()
    return res, err


@pytest.fixture(params=["auto", "grid"])
def loop_mode(request, monkeypatch):
    """auto: the library's choice (XCD-local loops where the shape allows);
    grid: the grid-barrier loops, forced through LSTMLOOP_LOOPS."""
    if request.param == "grid":
        monkeypatch.setenv("LSTMLOOP_LOOPS", "grid")
    else:
        monkeypatch.delenv("LSTMLOOP_LOOPS", raising=False)
    return request.param


@pytest.mark.parametrize("w", SMALL, ids=[w.name for w in SMALL])
def test_small_parity(w, loop_mode):
    inp = wl.generate(w)
    dc = DeviceCase(inp, w.H, w.I, w.layers, w.dtype)
    plan = dc.plan()
    geom = plan.geometry()
    plan.close()
    say(f"[parity] {w.name} mode={loop_mode} geometry={geom}")
    if loop_mode == "grid":
        assert not geom["xcd_local"]
    res, err = run_case(w, inp)
    assert err == 0
    ref = oracle_reference(inp, w.layers, w.dtype)
    assert res["T_eff"] == ref["T_eff"] == int(inp["seq_len"].max())
    errs, bad = compare(res, ref, TOL[w.dtype])
    say(f"    errors {errs}")
    assert not bad, bad


MAX_BATCH = [
    W("f32_b4096_i8_h32_t4_maxbatch", B=4096, I=8, H=32, T_max=4, dtype="f32", len_lo=0, len_hi=4,
      w_scale=0.3, random_state=True, seed=61),
    W("bf16_b4096_i16_h64_t3_maxbatch", B=4096, I=16, H=64, T_max=3, dtype="bf16", len_lo=0,
      len_hi=3, random_state=True, seed=62),
]


@pytest.mark.parametrize("w", MAX_BATCH, ids=[w.name for w in MAX_BATCH])
def test_maximum_batch_parity(w):
    """The largest batch a plan accepts (4096 rows: 256 row tiles, beyond the
    XCD-local loops' row tiles, so the library's own choice of loops), with
    zero-length rows among them, against the oracle."""
    inp = wl.generate(w)
    say(f"[maxbatch] {w.name}")
    res, err = run_case(w, inp)
    assert err == 0
    ref = oracle_reference(inp, w.layers, w.dtype)
    assert res["T_eff"] == ref["T_eff"] == int(inp["seq_len"].max())
    errs, bad = compare(res, ref, TOL[w.dtype])
    say(f"    errors {errs}")
    assert not bad, bad


# Shapes whose recurrent weights need more than one XCD: the chip-wide form
# (bf16 H = 2048, f32 H = 1024), one row tile to all 16, ragged lengths, two
# layers; against the oracle in that form and in the grid-barrier form.
CHIP = [
    W("chip_bf16_b37_i64_h2048_t7", B=37, I=64, H=2048, T_max=7, dtype="bf16", len_lo=0,
      len_hi=7, random_state=True, seed=41),
    W("chip_f32_b50_i32_h1024_t9", B=50, I=32, H=1024, T_max=9, dtype="f32", len_lo=1,
      len_hi=9, random_state=True, seed=42),
    W("chip_bf16_b256_i32_h2048_t4_mrt16", B=256, I=32, H=2048, T_max=4, dtype="bf16",
      len_lo=0, len_hi=4, random_state=True, seed=43),
    W("chip_f32_b9_i8_h1024_t12", B=9, I=8, H=1024, T_max=12, dtype="f32", len_lo=0,
      len_hi=12, random_state=True, seed=44),
    W("chip_f32_2layer_b20_i16_h1024_t6", B=20, I=16, H=1024, T_max=6, dtype="f32", layers=2,
      len_lo=0, len_hi=6, random_state=True, seed=45),
]


@pytest.mark.parametrize("w", CHIP, ids=[w.name for w in CHIP])
def test_chip_loops_parity(w, loop_mode):
    say(f"[chip] {w.name} mode={loop_mode}")
    inp = wl.generate(w)
    geom = {}
    res, err = run_case(w, inp, geometry=geom)
    assert geom["loops"] == ("grid" if loop_mode == "grid" else "chip"), geom
    assert err == 0
    ref = oracle_reference(inp, w.layers, w.dtype)
    assert res["T_eff"] == ref["T_eff"]
    errs, bad = compare(res, ref, TOL[w.dtype])
    say(f"    errors {errs}")
    assert not bad, bad


def test_zero_trip_loop_returns_inits_bitwise():
    w = wl.TINY.with_(name="all_zero", random_state=True, with_dy=True, seed=21)
    inp = wl.generate(w)
    inp["seq_len"][:] = 0
    say("[edge] all lengths zero")
    res, err = run_case(w, inp)
    assert err == 0 and res["T_eff"] == 0
    assert (res["y"] == 0).all() and (res["dx"] == 0).all()
    np.testing.assert_array_equal(res["hT"], inp["h0"])
    np.testing.assert_array_equal(res["cT"], inp["c0"])
    np.testing.assert_array_equal(res["dh0"], inp["dhT"])
    np.testing.assert_array_equal(res["dc0"], inp["dcT"])
    assert all((d == 0).all() for d in res["dW"]) and all((d == 0).all() for d in res["dbias"])


def test_finished_rows_and_nan_padding():
    w = W("nanpad", B=19, I=24, H=64, T_max=13, dtype="f32", len_lo=0, len_hi=13,
          random_state=True, seed=22)
    inp = wl.generate(w)
    say("[edge] NaN padding")
    clean, _ = run_case(w, inp)
    inp_nan = wl.generate(w, nan_padding=True)
    dirty, err = run_case(w, inp_nan)
    assert err == 0
    for k in ("y", "hT", "cT", "dx", "dh0", "dc0"):
        np.testing.assert_array_equal(dirty[k], clean[k], err_msg=k)
    for a, b in zip(dirty["dW"] + dirty["dbias"], clean["dW"] + clean["dbias"]):
        np.testing.assert_array_equal(a, b)
    L = inp["seq_len"]
    for b in range(w.B):
        assert (clean["y"][L[b]:, b] == 0).all() and (clean["dx"][L[b]:, b] == 0).all()
        if L[b] > 0:
            np.testing.assert_array_equal(clean["hT"][0, b], clean["y"][L[b] - 1, b])
        else:
            np.testing.assert_array_equal(clean["hT"][0, b], inp["h0"][0, b])


def test_rows_are_independent_and_permutation_equivariant():
    w = W("perm", B=40, I=32, H=128, T_max=10, dtype="bf16", len_lo=0, len_hi=10,
          random_state=True, seed=23)
    inp = wl.generate(w)
    say("[edge] permutation")
    full, _ = run_case(w, inp)
    p = np.random.default_rng(0).permutation(w.B)
    pin = dict(inp)
    pin["x"] = inp["x"][:, p].copy()
    pin["dy"] = inp["dy"][:, p].copy()
    pin["seq_len"] = inp["seq_len"][p].copy()
    for k in ("h0", "c0", "dhT", "dcT"):
        pin[k] = inp[k][:, p].copy()
    perm, _ = run_case(w, pin)
    for k in ("y", "dx"):
        np.testing.assert_array_equal(perm[k], full[k][:, p], err_msg=k)
    for k in ("hT", "cT", "dh0", "dc0"):
        np.testing.assert_array_equal(perm[k], full[k][:, p], err_msg=k)
    for a, b in zip(perm["dW"] + perm["dbias"], full["dW"] + full["dbias"]):
        assert np.abs(a - b).max() <= 1e-5 * np.abs(b).max()
    say("[edge] one row alone")
    for b in (0, 7, 33):
        one = {k: (v[:, b:b + 1].copy() if k in ("x", "dy", "h0", "c0", "dhT", "dcT") else v)
               for k, v in inp.items()}
        one["seq_len"] = inp["seq_len"][b:b + 1].copy()
        res, _ = run_case(w.with_(B=1), one)
        for k in ("y", "dx"):
            np.testing.assert_array_equal(res[k][:, 0], full[k][:, b], err_msg=k)
        for k in ("hT", "cT", "dh0", "dc0"):
            np.testing.assert_array_equal(res[k][:, 0], full[k][:, b], err_msg=k)


def test_tmax_padding_changes_nothing():
    w = W("tpad", B=24, I=32, H=64, T_max=8, dtype="f32", len_lo=0, len_hi=8,
          random_state=True, seed=24)
    inp = wl.generate(w)
    say("[edge] T_max padding")
    a, _ = run_case(w, inp)
    big = dict(inp)
    rng = np.random.default_rng(1)
    big["x"] = np.concatenate([inp["x"], rng.standard_normal((5, 24, 32), dtype=np.float32)])
    big["dy"] = np.concatenate([inp["dy"], rng.standard_normal((5, 24, 64), dtype=np.float32)])
    b, _ = run_case(w.with_(T_max=13), big)
    for k in ("hT", "cT", "dh0", "dc0"):
        np.testing.assert_array_equal(b[k], a[k], err_msg=k)
    np.testing.assert_array_equal(b["y"][:8], a["y"])
    np.testing.assert_array_equal(b["dx"][:8], a["dx"])
    assert (b["y"][8:] == 0).all() and (b["dx"][8:] == 0).all()
    for u, v in zip(b["dW"] + b["dbias"], a["dW"] + a["dbias"]):
        assert np.abs(u - v).max() <= 1e-6 * np.abs(v).max()


def test_repeat_calls_are_deterministic():
    w = W("det", B=64, I=64, H=256, T_max=12, dtype="bf16", len_lo=1, len_hi=12,
          random_state=True, seed=25)
    inp = wl.generate(w)
    say("[edge] determinism")
    dc = DeviceCase(inp, w.H, w.I, w.layers, w.dtype)
    plan = dc.plan()
    outs = []
    for _ in range(3):
        dc.fwd(plan)
        dc.bwd(plan)
        outs.append(dc.results())
    plan.close()
    for o in outs[1:]:
        for k in ("y", "hT", "cT", "dx", "dh0", "dc0"):
            np.testing.assert_array_equal(o[k], outs[0][k])
        for u, v in zip(o["dW"] + o["dbias"], outs[0]["dW"] + outs[0]["dbias"]):
            np.testing.assert_array_equal(u, v)


@pytest.mark.parametrize("dtype,layers", [("bf16", 1), ("f32", 1), ("bf16", 2)])
def test_inference_forward_between_saved_forwards_changes_nothing(dtype, layers):
    """A saved forward prepares part of the gradient pass's set-up (flags,
    row maps, permuted weights) in its own launches; an inference forward in
    between, and the saved forward it replaces, leave the next saved
    forward's gradient pass bitwise unchanged."""
    w = W("interleave", B=64, I=64, H=256, T_max=12, dtype=dtype, layers=layers, len_lo=0,
          len_hi=12, random_state=True, seed=31)
    inp = wl.generate(w)
    say(f"[edge] saved / inference / saved forwards, {dtype}, {layers} layer(s)")
    dc = DeviceCase(inp, w.H, w.I, w.layers, w.dtype)
    plan = dc.plan()
    dc.fwd(plan)
    dc.bwd(plan)
    ref = dc.results()
    dc.fwd(plan)
    dc.fwd(plan, save=False)
    dc.fwd(plan)
    dc.bwd(plan)
    got = dc.results()
    plan.close()
    for k in ("y", "hT", "cT", "dx", "dh0", "dc0"):
        np.testing.assert_array_equal(got[k], ref[k])
    for u, v in zip(got["dW"] + got["dbias"], ref["dW"] + ref["dbias"]):
        np.testing.assert_array_equal(u, v)


@pytest.mark.parametrize("dtype,layers,B,I,H,loops", [
    ("bf16", 1, 48, 64, 128, "auto"), ("f32", 1, 48, 64, 128, "auto"), ("bf16", 2, 48, 64, 128, "auto"),
    ("bf16", 1, 128, 1024, 1024, "auto"), ("bf16", 1, 64, 64, 2048, "auto"), ("f32", 1, 64, 64, 1024, "auto"),
    ("f32", 1, 48, 64, 128, "grid")])
def test_plan_reused_with_new_lengths_matches_a_fresh_plan(dtype, layers, B, I, H, loops, monkeypatch):
    """Everything a call derives from the lengths (trip count, order, compact
    offsets, row maps, loop flags, barrier counters) is rebuilt on the device
    by each call: a plan reused with other lengths in the same seq_len
    buffer gives the results of a fresh plan bitwise, also when the new trip
    count is shorter or zero (XCD-local loops, the benchmark's widths, the
    chip-wide loops of bf16 H = 2048 and f32 H = 1024, the grid-barrier
    loops)."""
    if loops == "grid":
        monkeypatch.setenv("LSTMLOOP_LOOPS", "grid")
    else:
        monkeypatch.delenv("LSTMLOOP_LOOPS", raising=False)
    w = W("new_lengths", B=B, I=I, H=H, T_max=15, dtype=dtype, layers=layers, len_lo=0,
          len_hi=15, random_state=True, with_dy=True, seed=33)
    _check_reuse_with_new_lengths(w, "lstm")


@pytest.mark.parametrize("cell", ["gru", "rnn", "skip", "act"])
def test_other_cells_plan_reused_with_new_lengths(cell):
    """As above for the other bodies (the cond body's guards, the nested
    loop's ponder slots and inner trip counts are per call too)."""
    w = W("new_lengths_" + cell, B=48, I=64, H=128, T_max=15, dtype="bf16", len_lo=0, len_hi=15,
          random_state=True, with_dy=True, cell=cell, seed=35)
    _check_reuse_with_new_lengths(w, cell)


def _check_reuse_with_new_lengths(w, cell):
    pm = w.ponder_max if cell == "act" else 0
    say(f"[edge] plan reuse with new lengths, {cell}, {w.dtype}, {w.layers} layer(s), H={w.H}")
    inp = wl.generate(w)
    dc = DeviceCase(inp, w.H, w.I, w.layers, w.dtype, cell=cell, ponder_max=pm)
    plan = dc.plan()
    say(f"    loops {plan.geometry()}")
    dc.fwd(plan)
    dc.bwd(plan)
    rng = np.random.default_rng(34)
    for new_len in (rng.integers(0, 8, size=w.B).astype(np.int32),      # shorter trip count
                    rng.integers(3, 16, size=w.B).astype(np.int32),     # longer again
                    np.zeros(w.B, dtype=np.int32)):                     # zero trip
        inp2 = dict(inp, seq_len=new_len)
        dc.seq_len.copy_(torch.from_numpy(new_len))
        dc.fwd(plan)
        dc.bwd(plan)
        assert plan.status_sync() == 0
        got = dc.results()
        fresh = DeviceCase(inp2, w.H, w.I, w.layers, w.dtype, cell=cell, ponder_max=pm)
        plan2 = fresh.plan()
        fresh.fwd(plan2)
        fresh.bwd(plan2)
        assert plan2.status_sync() == 0
        ref = fresh.results()
        plan2.close()
        for k in ("y", "hT", "cT", "dx", "dh0", "dc0"):
            np.testing.assert_array_equal(got[k], ref[k])
        for u, v in zip(got["dW"] + got["dbias"], ref["dW"] + ref["dbias"]):
            np.testing.assert_array_equal(u, v)
    plan.close()


def test_plans_on_two_streams_match_one_stream():
    """Two plans whose calls alternate between two streams: the loop launches
    stay ordered across streams (the first one from the second stream
    synchronises the device, later ones wait on the previous launch's
    event), and every output equals, bitwise, the same calls on one stream."""
    w = W("streams", B=24, I=32, H=64, T_max=9, dtype="f32", len_lo=0, len_hi=9,
          random_state=True, seed=41)
    inp = wl.generate(w)
    say("[edge] two streams")
    ref, err = run_case(w, inp)
    assert err == 0
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    dcs = [DeviceCase(inp, w.H, w.I, w.layers, w.dtype) for _ in streams]
    plans = [dc.plan() for dc in dcs]
    torch.cuda.synchronize()
    for _ in range(3):
        for dc, plan, st in zip(dcs, plans, streams):
            with torch.cuda.stream(st):
                dc.fwd(plan)
                dc.bwd(plan)
    torch.cuda.synchronize()
    for dc, plan in zip(dcs, plans):
        assert plan.status_sync() == 0
        res = dc.results()
        plan.close()
        for k in ("y", "hT", "cT", "dx", "dh0", "dc0"):
            np.testing.assert_array_equal(res[k], ref[k], err_msg=k)
        for u, v in zip(res["dW"] + res["dbias"], ref["dW"] + ref["dbias"]):
            np.testing.assert_array_equal(u, v)


def test_two_layers_equal_two_single_layer_calls(monkeypatch):
    # layer by layer, the two-layer plan makes the same calls as two plans
    monkeypatch.setenv("LSTMLOOP_WAVEFRONT", "off")
    w = W("stack2", B=45, I=64, H=64, T_max=10, dtype="bf16", layers=2, len_lo=0, len_hi=10,
          random_state=True, seed=26)
    inp = wl.generate(w)
    say("[edge] two layers vs two calls")
    geom = {}
    both, _ = run_case(w, inp, geometry=geom)
    assert not geom["wavefront"]
    w1 = w.with_(layers=1)
    l1 = dict(inp, W=[inp["W"][0]], bias=[inp["bias"][0]], h0=inp["h0"][:1], c0=inp["c0"][:1],
              dhT=inp["dhT"][:1], dcT=inp["dcT"][:1])
    # forward of layer 1, then layer 2 on bf16(y1); backward in reverse order
    dc1 = DeviceCase(l1, w.H, w.I, 1, "bf16")
    p1 = dc1.plan()
    dc1.fwd(p1)
    y1 = dc1.y.detach().clone()
    l2 = dict(inp, x=y1.to(torch.bfloat16).float().cpu().numpy(), W=[inp["W"][1]],
              bias=[inp["bias"][1]], h0=inp["h0"][1:], c0=inp["c0"][1:], dhT=inp["dhT"][1:],
              dcT=inp["dcT"][1:])
    dc2 = DeviceCase(l2, w.H, w.H, 1, "bf16")
    p2 = dc2.plan()
    dc2.fwd(p2)
    dc2.bwd(p2)
    r2 = dc2.results()
    dc1.dy = dc2.dx.detach().clone()
    dc1.bwd(p1)
    r1 = dc1.results()
    p1.close()
    p2.close()
    np.testing.assert_array_equal(both["y"], r2["y"])
    np.testing.assert_array_equal(both["hT"], np.concatenate([r1["hT"], r2["hT"]]))
    np.testing.assert_array_equal(both["cT"], np.concatenate([r1["cT"], r2["cT"]]))
    np.testing.assert_array_equal(both["dx"], r1["dx"])
    np.testing.assert_array_equal(both["dh0"], np.concatenate([r1["dh0"], r2["dh0"]]))
    np.testing.assert_array_equal(both["dW"][0], r1["dW"][0])
    np.testing.assert_array_equal(both["dW"][1], r2["dW"][0])
    np.testing.assert_array_equal(both["dbias"][1], r2["dbias"][0])


# ------------------------------------------------ two-layer wavefront
# Shapes where one launch runs both layers (2 H / units per work-group <= 32),
# covering one and several row tiles per XCD, both forward k-step classes and
# tiles that start or finish at different steps.
TWO_LAYER_WAVE = [
    W("wave_bf16_b150_i64_h512_t12", B=150, I=64, H=512, T_max=12, dtype="bf16", layers=2,
      len_lo=0, len_hi=12, random_state=True, seed=31),
    W("wave_f32_b40_i24_h256_t15", B=40, I=24, H=256, T_max=15, dtype="f32", layers=2,
      len_lo=1, len_hi=15, random_state=True, seed=32),
    W("wave_bf16_b300_i32_h128_t10_mrt3", B=300, I=32, H=128, T_max=10, dtype="bf16",
      layers=2, len_lo=0, len_hi=10, w_scale=0.3, random_state=True, seed=33),
    W("wave_f32_b9_i8_h96_t20", B=9, I=8, H=96, T_max=20, dtype="f32", layers=2, len_lo=0,
      len_hi=20, w_scale=0.3, random_state=True, seed=34),
]


@pytest.fixture(params=["wavefront", "layerwise"])
def layer_schedule(request, monkeypatch):
    """wavefront: the library's choice for these shapes; layerwise: one launch
    per layer, forced through LSTMLOOP_WAVEFRONT."""
    if request.param == "layerwise":
        monkeypatch.setenv("LSTMLOOP_WAVEFRONT", "off")
    else:
        monkeypatch.delenv("LSTMLOOP_WAVEFRONT", raising=False)
    monkeypatch.delenv("LSTMLOOP_LOOPS", raising=False)
    return request.param


@pytest.mark.parametrize("w", TWO_LAYER_WAVE, ids=[w.name for w in TWO_LAYER_WAVE])
def test_two_layer_wavefront_parity(w, layer_schedule):
    say(f"[wave] {w.name} {layer_schedule}")
    inp = wl.generate(w)
    geom = {}
    res, err = run_case(w, inp, geometry=geom)
    assert geom["xcd_local"] and geom["wavefront"] == (layer_schedule == "wavefront"), geom
    assert err == 0
    ref = oracle_reference(inp, w.layers, w.dtype)
    assert res["T_eff"] == ref["T_eff"]
    errs, bad = compare(res, ref, TOL[w.dtype])
    say(f"    errors {errs}")
    assert not bad, bad


def test_two_layer_wavefront_zero_trip_and_finished_rows():
    w = TWO_LAYER_WAVE[3]
    inp = wl.generate(w)
    say("[wave] all lengths zero")
    zero = dict(inp, seq_len=np.zeros_like(inp["seq_len"]))
    geom = {}
    res, err = run_case(w, zero, geometry=geom)
    assert geom["wavefront"] and err == 0 and res["T_eff"] == 0
    assert (res["y"] == 0).all() and (res["dx"] == 0).all()
    np.testing.assert_array_equal(res["hT"], inp["h0"])
    np.testing.assert_array_equal(res["cT"], inp["c0"])
    np.testing.assert_array_equal(res["dh0"], inp["dhT"])
    np.testing.assert_array_equal(res["dc0"], inp["dcT"])
    assert all((d == 0).all() for d in res["dW"]) and all((d == 0).all() for d in res["dbias"])
    say("[wave] finished rows")
    res, err = run_case(w, inp)
    L = inp["seq_len"]
    for b in range(w.B):
        assert (res["y"][L[b]:, b] == 0).all() and (res["dx"][L[b]:, b] == 0).all()
        if L[b] > 0:
            np.testing.assert_array_equal(res["hT"][1, b], res["y"][L[b] - 1, b])
        else:
            np.testing.assert_array_equal(res["hT"][:, b], inp["h0"][:, b])


def test_invalid_lengths_raise_device_error_and_recover():
    w = W("badlen", B=8, I=32, H=32, T_max=6, dtype="f32", len_lo=1, len_hi=6,
          random_state=True, seed=27)
    inp = wl.generate(w)
    say("[edge] invalid seq_len")
    bad = dict(inp, seq_len=inp["seq_len"].copy())
    bad["seq_len"][3] = 7
    res, err = run_case(w, bad)
    assert err & LL_DEVERR_SEQ_LEN
    assert res["T_eff"] == 0 and (res["y"] == 0).all() and (res["dx"] == 0).all()
    np.testing.assert_array_equal(res["hT"], inp["h0"])
    good, err2 = run_case(w, inp)
    assert err2 == 0 and good["T_eff"] == int(inp["seq_len"].max())


def test_backward_without_forward_is_a_state_error():
    w = wl.TINY
    inp = wl.generate(w)
    dc = DeviceCase(inp, w.H, w.I, 1, w.dtype)
    plan = dc.plan()
    with pytest.raises(LoopError) as e:
        dc.bwd(plan)
    assert e.value.status == LL_ESTATE
    dc.fwd(plan, save=False)                 # inference saves nothing
    with pytest.raises(LoopError):
        dc.bwd(plan)
    dc.fwd(plan, save=True)
    dc.bwd(plan)
    with pytest.raises(LoopError):           # the stack was consumed
        dc.bwd(plan)
    plan.close()


# ----------------------------------------------------------- full sizes
@pytest.mark.parametrize("w", [wl.FIXED_H512, wl.VAR_H1024], ids=lambda w: w.name)
def test_full_size_parity(w):
    say(f"[full] {w.name}")
    inp = wl.generate(w)
    geom = {}
    res, err = run_case(w, inp, geometry=geom)
    assert err == 0
    # the launch configuration the benchmark times: XCD-local loops
    assert geom["xcd_local"], geom
    say("    oracle running")
    ref = oracle_reference(inp, w.layers, w.dtype)
    errs, bad = compare(res, ref, TOL[w.dtype])
    say(f"    errors {errs}")
    assert not bad, bad


@pytest.mark.parametrize("w", [wl.RNN_VAR_H1024, wl.GRU_VAR_H1024], ids=lambda w: w.name)
def test_other_cells_full_size_parity(w):
    """The benchmark's RNN and GRU workloads at full size, every output."""
    say(f"[full] {w.name}")
    inp = wl.generate(w)
    dc = DeviceCase(inp, w.H, w.I, w.layers, w.dtype, cell=w.cell)
    plan = dc.plan()
    assert plan.geometry()["xcd_local"]
    dc.fwd(plan)
    dc.bwd(plan)
    err = plan.status_sync()
    res = dc.results()
    plan.close()
    assert err == 0
    say("    oracle running")
    ref = oracle_reference(inp, w.layers, w.dtype, cell=w.cell)
    errs, bad = compare(res, ref, TOL[w.dtype])
    say(f"    errors {errs}")
    assert not bad, bad


def _clear_skip_margins(inp, w, margin, max_rounds=12):
    """Redraw x_t of the (step, row) pairs whose decision sits within
    `margin` of the threshold in the oracle, until no valid decision does
    (each redraw changes that row's trajectory from t on, so it can move a
    later decision of the same row; a few rounds settle it).  Only the oracle
    decides; the returned inputs feed both sides."""
    inp = dict(inp, x=inp["x"].copy())
    rng = np.random.default_rng(4242)
    for _ in range(max_rounds):
        ref = oracle_reference(inp, w.layers, w.dtype, cell="skip")
        close = np.zeros(inp["x"].shape[:2], bool)
        for m in ref["margin"]:
            close |= m <= margin
        if not close.any():
            return inp, ref
        ts, bs = np.nonzero(close)
        say(f"    redrawing x at {len(ts)} close decisions")
        fresh = rng.standard_normal((len(ts), w.I), dtype=np.float32)
        inp["x"][ts, bs] = wl.round_to_bf16(fresh) if w.dtype == "bf16" else fresh
    raise AssertionError("decisions did not clear the margin")


def test_skip_full_size_all_outputs():
    """The cond-body workload at full size with every decision at least 1e-3
    from the threshold in the oracle (x redrawn at the few close decisions,
    chosen by the oracle alone), so every output, dW and db included, is
    compared with the oracle."""
    w = wl.SKIP_VAR_H1024
    say(f"[full] {w.name} (all decisions clear)")
    inp, ref = _clear_skip_margins(wl.generate(w), w, 1e-3)
    assert min(float(m.min()) for m in ref["margin"]) > 1e-3
    dc = DeviceCase(inp, w.H, w.I, w.layers, w.dtype, cell="skip")
    plan = dc.plan()
    assert plan.geometry()["xcd_local"]
    dc.fwd(plan)
    dc.bwd(plan)
    err = plan.status_sync()
    res = dc.results()
    plan.close()
    assert err == 0
    errs, bad = compare(res, ref, TOL[w.dtype])
    say(f"    errors {errs}")
    assert not bad, bad


def test_skip_full_size_parity():
    """The benchmark's cond-body workload at full size, inputs as generated.
    Its ~2.6e4 decisions include some within the two sides' float32 rounding
    of the threshold, and a row that decides differently follows another
    trajectory, so the comparison is per row: every row whose decisions all
    sit at least 1e-3 from the threshold in the oracle must match it within
    the tolerance (rows do not interact in the loop).  At least 75% of the
    rows must qualify.  (dW and db over every row: the test above.)"""
    w = wl.SKIP_VAR_H1024
    say(f"[full] {w.name}")
    inp = wl.generate(w)
    dc = DeviceCase(inp, w.H, w.I, w.layers, w.dtype, cell="skip")
    plan = dc.plan()
    assert plan.geometry()["xcd_local"]
    dc.fwd(plan)
    dc.bwd(plan)
    err = plan.status_sync()
    res = dc.results()
    plan.close()
    assert err == 0
    say("    oracle running")
    ref = oracle_reference(inp, w.layers, w.dtype, cell="skip")
    good = (ref["margin"][0] > 1e-3).all(axis=0)       # [B]
    say(f"    rows with clear decisions: {int(good.sum())} of {w.B}")
    assert good.mean() >= 0.75
    tol = TOL[w.dtype]
    for key in ("y", "dx"):
        e = rel_err(res[key][:, good], ref[key][:, good])
        assert e <= tol, (key, e)
    for key in ("hT", "cT", "dh0", "dc0"):
        e = rel_err(res[key][:, good], ref[key][:, good])
        assert e <= tol, (key, e)


# The two-layer H = 2048 workload's shape (bf16, I = H = 2048: chip-wide
# loops, and dW through the gather-transposes and the split-K NT product,
# which the plan's cost model picks for these long reductions) at batches the
# oracle finishes in seconds; every output, dW and db of both layers included.
TWO_LAYER_H2048_REDUCED = [
    W("lstm2_b24_h2048_t6_bf16", B=24, I=2048, H=2048, T_max=6, dtype="bf16", layers=2,
      len_lo=0, len_hi=6, random_state=True, seed=1105),
    W("lstm2_b64_h2048_t4_bf16", B=64, I=2048, H=2048, T_max=4, dtype="bf16", layers=2,
      len_lo=1, len_hi=4, seed=1205),
]


@pytest.mark.parametrize("w", TWO_LAYER_H2048_REDUCED, ids=[w.name for w in TWO_LAYER_H2048_REDUCED])
def test_two_layer_h2048_reduced_batch_every_output(w):
    say(f"[h2048] {w.name}")
    inp = wl.generate(w)
    geom = {}
    res, err = run_case(w, inp, geometry=geom)
    assert geom["loops"] == "chip", geom
    assert err == 0
    say("    oracle running")
    ref = oracle_reference(inp, w.layers, w.dtype)
    assert res["T_eff"] == ref["T_eff"]
    errs, bad = compare(res, ref, TOL[w.dtype])
    say(f"    errors {errs}")
    assert not bad, bad


def test_two_layer_full_size_sampled_rows():
    w = wl.TWO_LAYER
    say(f"[full] {w.name} (sampled rows)")
    inp = wl.generate(w)
    res, err = run_case(w, inp)
    assert err == 0
    rows = [int(np.argmax(inp["seq_len"])), int(np.argmin(inp["seq_len"])), 101]
    sub = {k: (v[:, rows].copy() if k in ("x", "dy", "h0", "c0", "dhT", "dcT") else v)
           for k, v in inp.items()}
    sub["seq_len"] = inp["seq_len"][rows].copy()
    ref = oracle_reference(sub, w.layers, w.dtype)
    got = {k: res[k][:, rows] for k in ("y", "hT", "cT", "dx", "dh0", "dc0")}
    errs, bad = compare(got, ref, TOL[w.dtype], keys=("y", "hT", "cT", "dx", "dh0", "dc0"))
    say(f"    errors {errs}")
    assert not bad, bad


# ----------------------------------------------------------- stack spill
def _run_plan(w, inp, **plan_kw):
    dc = DeviceCase(inp, w.H, w.I, w.layers, w.dtype)
    plan = dc.plan(**plan_kw)
    dev_bytes, host_bytes = plan.stack_bytes()
    dc.fwd(plan)
    dc.bwd(plan)
    err = plan.status_sync()
    res = dc.results()
    plan.close()
    return res, err, dev_bytes, host_bytes


SPILL_CASES = [
    # (workload, chunk steps, ring slots)
    (W("spill_f32_b20_i24_h64_t50", B=20, I=24, H=64, T_max=50, dtype="f32", len_lo=0, len_hi=50,
       w_scale=0.3, random_state=True, seed=21), 8, 3),
    (W("spill_bf16_b40_i32_h128_t37", B=40, I=32, H=128, T_max=37, dtype="bf16", len_lo=1, len_hi=37,
       w_scale=0.3, random_state=True, seed=22), 5, 4),
    (W("spill_f32_2layer_b17_i16_h32_t29", B=17, I=16, H=32, T_max=29, dtype="f32", layers=2,
       len_lo=0, len_hi=29, w_scale=0.3, random_state=True, seed=23), 4, 3),
    (W("spill_f32_resident_b9_i8_h32_t12", B=9, I=8, H=32, T_max=12, dtype="f32", len_lo=0,
       len_hi=12, w_scale=0.3, random_state=True, seed=24), 6, 3),
]


@pytest.mark.parametrize("w,C,R", SPILL_CASES, ids=[c[0].name for c in SPILL_CASES])
def test_spill_matches_resident_stack_bitwise(w, C, R, monkeypatch):
    """Swapping the stack to host memory in chunks changes no result bit
    (against the resident stack with the same layer-by-layer schedule: a
    spilling plan runs its layers one after the other)."""
    monkeypatch.setenv("LSTMLOOP_WAVEFRONT", "off")
    say(f"[spill] {w.name} C={C} R={R}")
    inp = wl.generate(w)
    ref, err0, dev0, host0 = _run_plan(w, inp)
    slot_bytes = C * w.B * 5 * w.H * 4
    got, err1, dev1, host1 = _run_plan(w, inp, spill=1, spill_chunk_steps=C,
                                       device_stack_budget_bytes=R * slot_bytes)
    assert err0 == 0 and err1 == 0
    # only the chunks a later chunk evicts from the ring of R slots (at least
    # 3) go to host memory; a budget that holds every chunk moves nothing
    nch = -(-w.T_max // C)
    nslots = max(3, min(R, nch))
    assert host0 == 0
    assert host1 == w.layers * max(0, nch - nslots) * slot_bytes
    for k in ("y", "hT", "cT", "dx", "dh0", "dc0"):
        assert np.array_equal(got[k], ref[k]), k
    for a, b in zip(got["dW"] + got["dbias"], ref["dW"] + ref["dbias"]):
        assert np.array_equal(a, b)
    # and the resident run is right
    errs, bad = compare(ref, oracle_reference(inp, w.layers, w.dtype), TOL[w.dtype])
    assert not bad, bad


@pytest.mark.parametrize("dtype,mode", [("f32", "spill"), ("bf16", "spill"), ("f32", "recompute")])
def test_memory_policy_repeat_calls_bitwise(dtype, mode, monkeypatch):
    """Consecutive training steps on one plan that swaps the stack (device
    ring, host stack, copy events) or recomputes the gates (chunk buffers)
    reuse its state; every step's results equal the first's bitwise, and a
    forward-only call in between changes nothing."""
    monkeypatch.setenv("LSTMLOOP_WAVEFRONT", "off")
    w = W("policy_repeat", B=24, I=32, H=64, T_max=41, dtype=dtype, len_lo=0, len_hi=41,
          w_scale=0.3, random_state=True, seed=26)
    say(f"[{mode}] repeat calls, {dtype}")
    inp = wl.generate(w)
    C, R = 6, 3
    dc = DeviceCase(inp, w.H, w.I, w.layers, w.dtype)
    if mode == "spill":
        plan = dc.plan(spill=1, spill_chunk_steps=C, device_stack_budget_bytes=R * C * w.B * 5 * w.H * 4)
    else:
        plan = dc.plan(recompute=1, spill_chunk_steps=C)
    outs = []
    for k in range(3):
        dc.fwd(plan)
        dc.bwd(plan)
        assert plan.status_sync() == 0
        outs.append(dc.results())
        if k == 0:
            dc.fwd(plan, save=False)
    plan.close()
    for o in outs[1:]:
        for key in ("y", "hT", "cT", "dx", "dh0", "dc0"):
            np.testing.assert_array_equal(o[key], outs[0][key])
        for u, v in zip(o["dW"] + o["dbias"], outs[0]["dW"] + outs[0]["dbias"]):
            np.testing.assert_array_equal(u, v)


def test_spill_long_sequences():
    """2000-step sequences, the stack swapped through a ring of 4 chunks."""
    w = wl.LONG_SPILL
    say(f"[spill] {w.name}")
    inp = wl.generate(w)
    C = 32
    slot_bytes = C * w.B * 5 * w.H * 4
    got, err1, dev1, host1 = _run_plan(w, inp, spill=1, spill_chunk_steps=C,
                                       device_stack_budget_bytes=4 * slot_bytes)
    assert err1 == 0
    ref, err0, dev0, _ = _run_plan(w, inp)
    assert err0 == 0
    say(f"    device stack bytes {dev1} (resident {dev0}), host {host1}")
    nch = -(-w.T_max // C)
    assert dev1 < dev0 and host1 == (nch - 4) * slot_bytes
    for k in ("y", "hT", "cT", "dx", "dh0", "dc0"):
        assert np.array_equal(got[k], ref[k]), k
    assert all(np.array_equal(a, b) for a, b in zip(got["dW"], ref["dW"]))
    # sampled rows against the oracle
    rows = [0, 31, 63]
    sub = {k: (v[:, rows].copy() if k in ("x", "dy", "h0", "c0", "dhT", "dcT") else v)
           for k, v in inp.items()}
    sub["seq_len"] = inp["seq_len"][rows].copy()
    ref_o = oracle_reference(sub, w.layers, w.dtype)
    gsub = {k: got[k][:, rows] for k in ("y", "hT", "cT", "dx", "dh0", "dc0")}
    errs, bad = compare(gsub, ref_o, TOL[w.dtype], keys=("y", "hT", "cT", "dx", "dh0", "dc0"))
    say(f"    errors {errs}")
    assert not bad, bad


def test_spill_h512_every_output_against_the_oracle():
    """The spill workload's shape (f32, I = H = 512, B = 64, every length T)
    at T = 96 with chunks of 16 steps and a ring of 4 (two chunks swapped out
    and back): every output, dW and db included, against the oracle."""
    w = W("spill_f32_b64_h512_t96", B=64, I=512, H=512, T_max=96, dtype="f32", len_lo=96,
          len_hi=96, spill=True, seed=1304)
    say(f"[spill] {w.name}")
    inp = wl.generate(w)
    C = 16
    slot_bytes = C * w.B * 5 * w.H * 4
    got, err, dev, host = _run_plan(w, inp, spill=1, spill_chunk_steps=C,
                                    device_stack_budget_bytes=4 * slot_bytes)
    assert err == 0 and host == 2 * slot_bytes
    say("    oracle running")
    errs, bad = compare(got, oracle_reference(inp, w.layers, w.dtype), TOL[w.dtype])
    say(f"    errors {errs}")
    assert not bad, bad


RECOMPUTE_CASES = [
    # (workload, chunk steps)
    (W("rc_f32_b20_i24_h64_t50", B=20, I=24, H=64, T_max=50, dtype="f32", len_lo=0, len_hi=50,
       w_scale=0.3, random_state=True, seed=31), 8),
    (W("rc_bf16_b40_i32_h128_t37", B=40, I=32, H=128, T_max=37, dtype="bf16", len_lo=1, len_hi=37,
       w_scale=0.3, random_state=True, seed=32), 5),
    (W("rc_f32_2layer_b17_i16_h32_t29", B=17, I=16, H=32, T_max=29, dtype="f32", layers=2,
       len_lo=0, len_hi=29, w_scale=0.3, random_state=True, seed=33), 4),
    (W("rc_bf16_2layer_b70_i64_h128_t21", B=70, I=64, H=128, T_max=21, dtype="bf16", layers=2,
       len_lo=0, len_hi=21, w_scale=0.3, random_state=True, seed=34), 32),
    (W("rc_f32_b9_i8_h32_t12_short", B=9, I=8, H=32, T_max=12, dtype="f32", len_lo=0, len_hi=5,
       w_scale=0.3, random_state=True, seed=35), 3),
]


@pytest.mark.parametrize("w,C", RECOMPUTE_CASES, ids=[c[0].name for c in RECOMPUTE_CASES])
def test_recompute_parity(w, C):
    """Gates recomputed per chunk in the gradient pass (only c_t pushed):
    every output within the tolerance of the oracle, and of the plan that
    saves the gates; the device stack is smaller."""
    say(f"[recompute] {w.name} C={C}")
    inp = wl.generate(w)
    got, err1, dev1, host1 = _run_plan(w, inp, recompute=1, spill_chunk_steps=C)
    ref, err0, dev0, _ = _run_plan(w, inp)
    assert err0 == 0 and err1 == 0
    assert host1 == 0 and dev1 < dev0
    errs, bad = compare(got, oracle_reference(inp, w.layers, w.dtype), TOL[w.dtype])
    say(f"    errors vs oracle {errs}")
    assert not bad, bad
    errs, bad = compare(got, ref, TOL[w.dtype])
    say(f"    errors vs saved gates {errs}")
    assert not bad, bad


def test_recompute_zero_trip():
    """All lengths zero: no iteration, no recomputation; outputs are the
    initial state and the incoming gradients."""
    w = W("rc_zero_b6_i8_h32_t9", B=6, I=8, H=32, T_max=9, dtype="f32", len_lo=0, len_hi=0,
          w_scale=0.3, random_state=True, seed=36)
    inp = wl.generate(w)
    got, err, _, _ = _run_plan(w, inp, recompute=1, spill_chunk_steps=4)
    assert err == 0
    assert np.array_equal(got["hT"][0], inp["h0"][0]) and np.array_equal(got["cT"][0], inp["c0"][0])
    assert np.array_equal(got["dh0"][0], inp["dhT"][0]) and np.array_equal(got["dc0"][0], inp["dcT"][0])
    assert not np.any(got["dW"][0]) and not np.any(got["dx"])


RNN_CASES = [
    # (bf16 cases use the default U(+-1/sqrt(H)) weights: with larger ones the
    # tanh recurrence is expanding, and bf16 rounding differences of one ulp
    # in h grow step by step, the oracle's accumulation order being fp64)
    W("rnn_f32_b20_i24_h64_t30", B=20, I=24, H=64, T_max=30, dtype="f32", len_lo=0, len_hi=30,
      w_scale=0.3, random_state=True, cell="rnn", seed=41),
    W("rnn_bf16_b40_i32_h128_t37", B=40, I=32, H=128, T_max=37, dtype="bf16", len_lo=1, len_hi=37,
      random_state=True, cell="rnn", seed=42),
    W("rnn_bf16_b130_i64_h256_t21", B=130, I=64, H=256, T_max=21, dtype="bf16", len_lo=0,
      len_hi=21, random_state=True, cell="rnn", seed=43),
    W("rnn_f32_2layer_b17_i16_h32_t29", B=17, I=16, H=32, T_max=29, dtype="f32", layers=2,
      len_lo=0, len_hi=29, w_scale=0.3, random_state=True, cell="rnn", seed=44),
    W("rnn_bf16_b9_i8_h1024_t12", B=9, I=8, H=1024, T_max=12, dtype="bf16", len_lo=0, len_hi=12,
      random_state=True, cell="rnn", seed=45),
]


@pytest.mark.parametrize("w", RNN_CASES, ids=[w.name for w in RNN_CASES])
def test_rnn_cell_parity(w):
    """The same loop engine with the Elman RNN body: every output within the
    tolerance of the RNN oracle; cT and dc0 are written as zeros."""
    say(f"[rnn] {w.name}")
    inp = wl.generate(w)
    dc = DeviceCase(inp, w.H, w.I, w.layers, w.dtype, cell="rnn")
    plan = dc.plan()
    geom = plan.geometry()
    assert geom["xcd_local"], geom
    dc.fwd(plan)
    dc.bwd(plan)
    err = plan.status_sync()
    res = dc.results()
    plan.close()
    assert err == 0
    ref = oracle_reference(inp, w.layers, w.dtype, cell="rnn")
    assert res["T_eff"] == ref["T_eff"] == int(inp["seq_len"].max())
    errs, bad = compare(res, ref, TOL[w.dtype])
    say(f"    errors {errs}")
    assert not bad, bad


GRU_CASES = [
    W("gru_f32_b20_i24_h64_t30", B=20, I=24, H=64, T_max=30, dtype="f32", len_lo=0, len_hi=30,
      w_scale=0.3, random_state=True, cell="gru", seed=51),
    W("gru_bf16_b40_i32_h128_t37", B=40, I=32, H=128, T_max=37, dtype="bf16", len_lo=1, len_hi=37,
      random_state=True, cell="gru", seed=52),
    W("gru_bf16_b130_i64_h256_t21", B=130, I=64, H=256, T_max=21, dtype="bf16", len_lo=0,
      len_hi=21, random_state=True, cell="gru", seed=53),
    W("gru_f32_2layer_b17_i16_h32_t29", B=17, I=16, H=32, T_max=29, dtype="f32", layers=2,
      len_lo=0, len_hi=29, w_scale=0.3, random_state=True, cell="gru", seed=54),
    W("gru_f32_b33_i20_h512_t9", B=33, I=20, H=512, T_max=9, dtype="f32", len_lo=0, len_hi=9,
      random_state=True, cell="gru", seed=55),
    W("gru_bf16_b9_i8_h1024_t12", B=9, I=8, H=1024, T_max=12, dtype="bf16", len_lo=0, len_hi=12,
      random_state=True, cell="gru", seed=56),
]


@pytest.mark.parametrize("w", GRU_CASES, ids=[w.name for w in GRU_CASES])
def test_gru_cell_parity(w):
    """The loop engine with the GRU body (three gate blocks; the candidate
    block's two sides differ in the gradient): every output within the
    tolerance of the GRU oracle; cT and dc0 are written as zeros."""
    say(f"[gru] {w.name}")
    inp = wl.generate(w)
    dc = DeviceCase(inp, w.H, w.I, w.layers, w.dtype, cell="gru")
    plan = dc.plan()
    geom = plan.geometry()
    assert geom["xcd_local"], geom
    dc.fwd(plan)
    dc.bwd(plan)
    err = plan.status_sync()
    res = dc.results()
    plan.close()
    assert err == 0
    ref = oracle_reference(inp, w.layers, w.dtype, cell="gru")
    assert res["T_eff"] == ref["T_eff"] == int(inp["seq_len"].max())
    errs, bad = compare(res, ref, TOL[w.dtype])
    say(f"    errors {errs}")
    assert not bad, bad


# The LSTM body with a data-dependent cond.  The predicate is an integer
# decided by floating point on both sides (float32 sums in different orders,
# and the bf16 runs' trajectories differ within the tolerance), so every case
# uses a seed whose decisions all sit at least MARGIN from the threshold in
# the oracle; both branches occur in each.
SKIP_CASES = [
    (W("skip_f32_b20_i24_h64_t30", B=20, I=24, H=64, T_max=30, dtype="f32", len_lo=0, len_hi=30,
       w_scale=0.3, random_state=True, cell="skip", seed=89), 1e-3),
    (W("skip_bf16_b40_i32_h128_t37", B=40, I=32, H=128, T_max=37, dtype="bf16", len_lo=1, len_hi=37,
       random_state=True, cell="skip", seed=86), 5e-4),
    (W("skip_bf16_b130_i64_h256_t21", B=130, I=64, H=256, T_max=21, dtype="bf16", len_lo=0,
       len_hi=21, random_state=True, cell="skip", seed=89), 5e-4),
    (W("skip_f32_2layer_b17_i16_h32_t29", B=17, I=16, H=32, T_max=29, dtype="f32", layers=2,
       len_lo=0, len_hi=29, w_scale=0.3, random_state=True, cell="skip", seed=98), 1e-3),
    (W("skip_f32_b33_i20_h512_t9", B=33, I=20, H=512, T_max=9, dtype="f32", len_lo=0, len_hi=9,
       random_state=True, cell="skip", seed=81), 1e-3),
    (W("skip_bf16_b9_i8_h1024_t12", B=9, I=8, H=1024, T_max=12, dtype="bf16", len_lo=0, len_hi=12,
       random_state=True, cell="skip", seed=87), 5e-4),
]


@pytest.mark.parametrize("w,margin", SKIP_CASES, ids=[c[0].name for c in SKIP_CASES])
def test_skip_cell_parity(w, margin):
    """The loop engine with the cond body: guards pushed in the forward and
    popped in the gradient loop; every output within the tolerance of the
    cond-body oracle, dbias zero in the predicate part."""
    say(f"[skip] {w.name}")
    inp = wl.generate(w)
    ref = oracle_reference(inp, w.layers, w.dtype, cell="skip")
    assert ref["min_margin"] > margin, "ill-conditioned case: a decision sits at the threshold"
    for l, gd in enumerate(ref["guards"]):
        valid = np.arange(w.T_max)[:, None] < inp["seq_len"][None, :]
        assert gd[valid].any() and not gd[valid].all(), f"layer {l}: one branch only"
    dc = DeviceCase(inp, w.H, w.I, w.layers, w.dtype, cell="skip")
    plan = dc.plan()
    geom = plan.geometry()
    assert geom["xcd_local"], geom
    dc.fwd(plan)
    dc.bwd(plan)
    err = plan.status_sync()
    res = dc.results()
    plan.close()
    assert err == 0
    assert res["T_eff"] == ref["T_eff"] == int(inp["seq_len"].max())
    errs, bad = compare(res, ref, TOL[w.dtype])
    say(f"    errors {errs}")
    assert not bad, bad
    for l in range(w.layers):
        I_l = w.I if l == 0 else w.H
        assert not res["dbias"][l][4 * w.H:].any() and res["dbias"][l].shape[0] == 4 * w.H + I_l + w.H + 1


@pytest.mark.parametrize("cell", ["rnn", "gru", "skip"])
def test_other_cells_zero_trip(cell):
    """Every length 0: the loop runs no iteration with any body, returns its
    inits (hT = h0; the LSTM-state cT = c0 for the cond body, zeros for the
    one-state cells) and passes the state gradients through; dW, db, dx are
    zero (bitwise)."""
    w = W(f"{cell}_zero_trip", B=20, I=16, H=64, T_max=5, dtype="bf16", len_lo=0, len_hi=0,
          random_state=True, cell=cell, seed=71)
    inp = wl.generate(w)
    assert not inp["seq_len"].any()
    dc = DeviceCase(inp, w.H, w.I, w.layers, w.dtype, cell=cell)
    plan = dc.plan()
    dc.fwd(plan)
    dc.bwd(plan)
    err = plan.status_sync()
    res = dc.results()
    plan.close()
    assert err == 0 and res["T_eff"] == 0
    np.testing.assert_array_equal(res["hT"], inp["h0"])
    np.testing.assert_array_equal(res["cT"], inp["c0"] if cell == "skip" else 0 * inp["c0"])
    np.testing.assert_array_equal(res["dh0"], inp["dhT"])
    np.testing.assert_array_equal(res["dc0"], inp["dcT"] if cell == "skip" else 0 * inp["dcT"])
    for k in ("y", "dx"):
        assert not res[k].any(), k
    assert not any(d.any() for d in res["dW"]) and not any(b.any() for b in res["dbias"])


# ------------------------------------------------------------ ABI contract
def test_bwd_rejects_operands_other_than_the_saved_forwards():
    """lstm_loop_bwd with an x, seq_len or W other than the saved forward's:
    LL_EINVAL, nothing enqueued, the saved stack kept for the right call."""
    from paper_1805_01772_amd.lstmloop import LL_EINVAL
    w = wl.TINY.with_(random_state=True, with_dy=True, seed=77)
    inp = wl.generate(w)
    dc = DeviceCase(inp, w.H, w.I, 1, w.dtype)
    plan = dc.plan()
    dc.fwd(plan)
    other_x = dc.x.clone()
    other_len = dc.seq_len.clone()
    other_W = [t.clone() for t in dc.W]
    for args in ((other_x, dc.seq_len, dc.W), (dc.x, other_len, dc.W), (dc.x, dc.seq_len, other_W)):
        with pytest.raises(LoopError) as e:
            plan.bwd(*args, dc.dy, dc.dhT, dc.dcT, dc.dx, dc.dW, dc.dbias, dc.dh0, dc.dc0)
        assert e.value.status == LL_EINVAL
    dc.bwd(plan)
    assert plan.status_sync() == 0
    res = dc.results()
    plan.close()
    ref = oracle_reference(inp, 1, w.dtype)
    errs, bad = compare(res, ref, TOL[w.dtype])
    assert not bad, bad


def _offset_copy(t, elems):
    """A contiguous copy of t whose data starts `elems` elements into a larger
    allocation (for alignment tests)."""
    flat = torch.empty(t.numel() + elems, dtype=t.dtype, device=t.device)
    v = flat[elems:].view(t.shape)
    v.copy_(t)
    return v


def test_misaligned_arrays_rejected_before_anything_is_enqueued():
    """An array that is not 16-byte aligned (here x, then dx) gives LL_EINVAL
    before anything is enqueued; the plan then runs normally."""
    from paper_1805_01772_amd.lstmloop import LL_EINVAL
    w = W("align_bf16_b16_i1024_h1024_t5", B=16, I=1024, H=1024, T_max=5, dtype="bf16",
          len_lo=0, len_hi=5, random_state=True, seed=78)
    inp = wl.generate(w)
    dc = DeviceCase(inp, w.H, w.I, 1, w.dtype)
    plan = dc.plan()
    assert plan.geometry()["dw_in_place"] == [True]
    x_al = dc.x
    dc.x = _offset_copy(x_al, 1)                 # 2 bytes off
    assert dc.x.data_ptr() % 16 != 0
    for save in (True, False):
        with pytest.raises(LoopError) as e:
            dc.fwd(plan, save=save)
        assert e.value.status == LL_EINVAL
    dc.x = x_al
    dc.fwd(plan)
    dx_al = dc.dx
    dc.dx = _offset_copy(dx_al, 2)               # 8 bytes off
    with pytest.raises(LoopError) as e:
        dc.bwd(plan)
    assert e.value.status == LL_EINVAL
    dc.dx = dx_al
    dc.bwd(plan)                                 # the saved stack was kept
    assert plan.status_sync() == 0
    res = dc.results()
    plan.close()
    errs, bad = compare(res, oracle_reference(inp, 1, w.dtype), TOL[w.dtype])
    assert not bad, bad


def test_dw_split_halves_summed_in_place():
    """bf16 I = H = 1024, B = 128: the dW product over rows runs as two
    split-K halves per 256x256 tile that meet on the tile's counter (the
    first stores its sums, the second adds them and writes dW); few steps
    keep the oracle quick.  Every output against the oracle, and a second
    call bitwise equal to the first (the counters reset themselves)."""
    w = W("dwsplit_bf16_b128_i1024_h1024_t6", B=128, I=1024, H=1024, T_max=6, dtype="bf16",
          len_lo=1, len_hi=6, random_state=True, seed=83)
    inp = wl.generate(w)
    say(f"[dw] {w.name}")
    dc = DeviceCase(inp, w.H, w.I, 1, w.dtype)
    plan = dc.plan()
    assert plan.geometry()["dw_in_place"] == [True]
    outs = []
    for _ in range(2):
        dc.fwd(plan)
        dc.bwd(plan)
        outs.append(dc.results())
    assert plan.status_sync() == 0
    plan.close()
    for u, v in zip(outs[1]["dW"] + outs[1]["dbias"], outs[0]["dW"] + outs[0]["dbias"]):
        np.testing.assert_array_equal(u, v)
    errs, bad = compare(outs[0], oracle_reference(inp, 1, w.dtype), TOL[w.dtype])
    say(f"    errors {errs}")
    assert not bad, bad


def test_dw_operands_past_two_gib_take_the_transposes():
    """bf16 I = H = 1024, B = 128, T_max = 2048: the dz rows of the row
    capacity reach 2 GiB, past the 32-bit offsets of the dW product over rows,
    so the plan takes the gather-transposes instead (the same shape at
    T_max = 200 reads in place); short lengths keep the oracle quick.  Every
    output against the oracle."""
    w = W("big_bf16_b128_i1024_h1024_t2048", B=128, I=1024, H=1024, T_max=2048, dtype="bf16",
          len_lo=0, len_hi=5, random_state=True, seed=79)
    inp = wl.generate(w)
    say(f"[abi] {w.name}")
    dc = DeviceCase(inp, w.H, w.I, 1, w.dtype)
    plan = dc.plan()
    assert plan.geometry()["dw_in_place"] == [False]
    dc.fwd(plan)
    dc.bwd(plan)
    assert plan.status_sync() == 0
    res = dc.results()
    plan.close()
    small = wl.Workload("b128_t200", B=128, I=1024, H=1024, T_max=200, dtype="bf16", len_lo=0,
                        len_hi=5)
    with DeviceCase(wl.generate(small), small.H, small.I, 1, small.dtype).plan() as p2:
        assert p2.geometry()["dw_in_place"] == [True]
    say("    oracle running")
    errs, bad = compare(res, oracle_reference(inp, 1, w.dtype), TOL[w.dtype])
    say(f"    errors {errs}")
    assert not bad, bad


# The LSTM body with a nested loop (ACT's halting rule).  The inner trip
# count is an integer decided by floating point on both sides (float32 sums
# in different orders, the kernel's sigmoid against the oracle's, and the
# bf16 runs' trajectories differ within the tolerance), so every case uses a
# seed whose decisions all sit at least MARGIN from the threshold in the
# oracle, with several trip counts occurring.  (case, margin, post-processing
# of the drawn inputs: halting bias and weight scale, or None)
ACT_CASES = [
    (W("act_f32_b20_i24_h64_t12_m3", B=20, I=24, H=64, T_max=12, dtype="f32", len_lo=0, len_hi=12,
       w_scale=0.3, random_state=True, cell="act", ponder_max=3, seed=200), 1e-4, None),
    (W("act_bf16_b40_i32_h128_t10_m4", B=40, I=32, H=128, T_max=10, dtype="bf16", len_lo=1, len_hi=10,
       w_scale=0.2, random_state=True, cell="act", ponder_max=4, seed=220), 2e-3, None),
    (W("act_bf16_b130_i64_h256_t8_m3", B=130, I=64, H=256, T_max=8, dtype="bf16", len_lo=0, len_hi=8,
       w_scale=0.15, random_state=True, cell="act", ponder_max=3, seed=272), 2e-3, None),
    (W("act_f32_b33_i20_h512_t6_m2", B=33, I=20, H=512, T_max=6, dtype="f32", len_lo=0, len_hi=6,
       random_state=True, cell="act", ponder_max=2, seed=209), 1e-4, (4.6, 8.0)),
    (W("act_bf16_b9_i8_h1024_t6_m4", B=9, I=8, H=1024, T_max=6, dtype="bf16", len_lo=0, len_hi=6,
       random_state=True, cell="act", ponder_max=4, seed=200), 2e-3, None),
    (W("act_f32_b5_i8_h32_t9_m1", B=5, I=8, H=32, T_max=9, dtype="f32", len_lo=0, len_hi=9,
       w_scale=0.3, random_state=True, cell="act", ponder_max=1, seed=200), 1e-4, None),
]


def _act_inputs(w, post):
    inp = wl.generate(w)
    if post is not None:
        bp, wscale = post
        inp["bias"][0][-1] = bp
        inp["bias"][0][4 * w.H:5 * w.H] *= wscale
    return inp


def _act_run(w, inp):
    dc = DeviceCase(inp, w.H, w.I, w.layers, w.dtype, cell="act", ponder_max=w.ponder_max)
    plan = dc.plan()
    geom = plan.geometry()
    assert geom["xcd_local"], geom
    dc.fwd(plan)
    dc.bwd(plan)
    err = plan.status_sync()
    res = dc.results()
    plan.close()
    return res, err


@pytest.mark.parametrize("w,margin,post", ACT_CASES, ids=[c[0].name for c in ACT_CASES])
def test_act_cell_parity(w, margin, post):
    """The loop engine with a nested loop in the body: inner trip counts
    decided on the device, pushed with every ponder step, popped by the
    nested gradient loop; every output within the tolerance of the oracle,
    dbias zero in the halting part."""
    say(f"[act] {w.name}")
    inp = _act_inputs(w, post)
    ref = oracle_reference(inp, w.layers, w.dtype, cell="act", ponder_max=w.ponder_max)
    assert ref["min_margin"] > margin, "ill-conditioned case: a decision sits at the threshold"
    valid = np.arange(w.T_max)[:, None] < inp["seq_len"][None, :]
    trips = ref["trips"][0][valid]
    assert trips.min() >= 1 and trips.max() <= w.ponder_max
    if w.ponder_max > 1:
        assert len(np.unique(trips)) >= 2, "one inner trip count only"
    res, err = _act_run(w, inp)
    assert err == 0
    assert res["T_eff"] == ref["T_eff"] == int(inp["seq_len"].max())
    errs, bad = compare(res, ref, TOL[w.dtype])
    say(f"    trips {np.unique(trips, return_counts=True)} errors {errs}")
    assert not bad, bad
    assert not res["dbias"][0][4 * w.H:].any() and res["dbias"][0].shape[0] == 5 * w.H + 1


def test_act_cell_zero_trip():
    """Every length 0: no iteration of either loop; inits returned, state
    gradients passed through, dW, db, dx zero (bitwise)."""
    w = W("act_zero_trip", B=20, I=16, H=64, T_max=5, dtype="bf16", len_lo=0, len_hi=0,
          random_state=True, cell="act", ponder_max=3, seed=71)
    inp = wl.generate(w)
    res, err = _act_run(w, inp)
    assert err == 0 and res["T_eff"] == 0
    np.testing.assert_array_equal(res["hT"], inp["h0"])
    np.testing.assert_array_equal(res["cT"], inp["c0"])
    np.testing.assert_array_equal(res["dh0"], inp["dhT"])
    np.testing.assert_array_equal(res["dc0"], inp["dcT"])
    for k in ("y", "dx"):
        assert not res[k].any(), k
    assert not any(d.any() for d in res["dW"]) and not any(b.any() for b in res["dbias"])


def test_act_cell_inference_matches_training_forward():
    """The nested-loop forward without a saved stack (inference) gives the
    same outputs bitwise as the forward that pushes it."""
    w, margin, post = ACT_CASES[1]
    inp = _act_inputs(w, post)
    dc = DeviceCase(inp, w.H, w.I, w.layers, w.dtype, cell="act", ponder_max=w.ponder_max)
    plan = dc.plan()
    dc.fwd(plan, save=True)
    a = dc.results()
    dc.fwd(plan, save=False)
    b = dc.results()
    assert plan.status_sync() == 0
    plan.close()
    for k in ("y", "hT", "cT"):
        np.testing.assert_array_equal(a[k], b[k], err_msg=k)


def test_act_full_size_rows_with_clear_decisions():
    """The nested-loop workload at full size (B = 128, I = H = 1024,
    T_max = 200, bf16, at most 4 ponder steps).  Its ~4e4 halting decisions
    include many within the two sides' differing float32 sums and bf16
    trajectories of the threshold, and a row that decides differently follows
    another trajectory, so the comparison is per row (rows do not interact):
    every row whose decisions all sit at least 1e-3 from the threshold in the
    oracle must match it within the tolerance in y, dx, hT, cT, dh0 and dc0;
    at least 10 rows must qualify."""
    w = wl.ACT_VAR_H1024
    say(f"[full] {w.name}")
    inp = wl.generate(w)
    res, err = _act_run(w, inp)
    assert err == 0
    say("    oracle running")
    import oracle as orc
    x = inp["x"].astype(np.float64)
    y, hT, cT, tape = orc.act_forward(x, inp["seq_len"], inp["W"][0].astype(np.float64),
                                      inp["bias"][0].astype(np.float64), inp["h0"][0].astype(np.float64),
                                      inp["c0"][0].astype(np.float64), "bf16", w.ponder_max)
    g = orc.act_backward(tape, inp["dy"].astype(np.float64), inp["dhT"][0].astype(np.float64),
                         inp["dcT"][0].astype(np.float64))
    good = tape["row_margin"] >= 1e-3
    say(f"    rows with clear decisions: {int(good.sum())} of {w.B}")
    assert good.sum() >= 10
    tol = TOL[w.dtype]
    ref = dict(y=y, dx=g["dx"], hT=hT[None], cT=cT[None], dh0=g["dh0"][None], dc0=g["dc0"][None])
    for key in ("y", "dx", "hT", "cT", "dh0", "dc0"):
        e = rel_err(res[key][:, good], ref[key][:, good])
        say(f"    {key}: {e:.3e}")
        assert e <= tol, (key, e)

