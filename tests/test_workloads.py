"""Host-side checks of the seeded input generators (no method arithmetic)."""
import numpy as np

from paper_1805_01772_amd import workloads as wl


def test_shapes_per_cell():
    base = dict(B=3, I=16, H=8, T_max=5, dtype="f32", len_lo=0, len_hi=5, layers=2, seed=7)
    for cell, G, blen0, blen1 in (("lstm", 4, 32, 32), ("rnn", 1, 8, 8), ("gru", 3, 32, 32),
                                  ("skip", 4, 4 * 8 + 16 + 8 + 1, 4 * 8 + 8 + 8 + 1)):
        w = wl.Workload("t", cell=cell, **base)
        inp = wl.generate(w)
        assert w.gates == G
        assert [a.shape for a in inp["W"]] == [(16 + 8, G * 8), (8 + 8, G * 8)]
        assert [a.shape[0] for a in inp["bias"]] == [blen0, blen1] == [w.bias_len(0), w.bias_len(1)]
        assert inp["x"].shape == (5, 3, 16) and inp["dy"].shape == (5, 3, 8)
        assert ((inp["seq_len"] >= 0) & (inp["seq_len"] <= 5)).all()


def test_seeded_and_bf16_representable():
    w = wl.GRU_VAR_H1024.with_(B=4, T_max=6, I=16, H=32, len_lo=1, len_hi=6)
    a, b = wl.generate(w), wl.generate(w)
    for k in ("x", "seq_len"):
        np.testing.assert_array_equal(a[k], b[k])
    np.testing.assert_array_equal(wl.round_to_bf16(a["x"]), a["x"])
    np.testing.assert_array_equal(wl.round_to_bf16(a["W"][0]), a["W"][0])


def test_flops_count_valid_steps_only():
    w = wl.Workload("t", B=2, I=4, H=2, T_max=3, dtype="f32", len_lo=0, len_hi=3, cell="gru")
    assert wl.algorithmic_flops(w, np.array([3, 1])) == 6.0 * 3 * 2 * (4 + 2) * 4
