"""ctypes binding of liblstmloop.so: argument marshalling only.

Every computation happens in the HIP library; this module turns torch
tensors into device pointers and the current torch stream into a hipStream_t.
The function names follow the C ABI of include/lstmloop.h.
If the library has not been built, every call raises; there is no fallback.
"""
from __future__ import annotations

import atexit
import ctypes
import os
import weakref
from typing import Optional, Sequence

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "liblstmloop.so")

LL_OK, LL_EINVAL, LL_ENOMEM, LL_EHIP, LL_ESTATE, LL_EUNSUPPORTED = range(6)
LL_F32, LL_BF16 = 0, 1
LL_DEVERR_SEQ_LEN, LL_DEVERR_BARRIER = 1, 2
LL_LOOPS_GRID, LL_LOOPS_XCD, LL_LOOPS_CHIP = 0, 1, 2
LL_CELL_LSTM, LL_CELL_RNN, LL_CELL_GRU, LL_CELL_LSTM_SKIP, LL_CELL_LSTM_ACT = 0, 1, 2, 3, 4
LL_ACT_EPS = 0.01
LL_ACT_PONDER_MAX = 8
STATUS_NAMES = {0: "LL_OK", 1: "LL_EINVAL", 2: "LL_ENOMEM", 3: "LL_EHIP",
                4: "LL_ESTATE", 5: "LL_EUNSUPPORTED"}

EXPORTED = ("ll_plan_create", "ll_plan_destroy", "ll_plan_stack_bytes",
            "ll_plan_geometry", "lstm_loop_fwd", "lstm_loop_bwd",
            "ll_status_sync", "ll_last_error", "ll_version",
            "ll_plan_set_timing", "ll_plan_set_timing_stages", "ll_plan_read_timing",
            "ll_measure_mfma_peak", "ll_eval_activations", "lstm_loop_fwd_noalloc")
STAGES = ("prep", "input_proj", "fwd_loop", "bwd_loop", "bwd_operands", "dw", "dx", "loop_setup",
          "recompute")


class ll_desc(ctypes.Structure):
    _fields_ = [("T_max", ctypes.c_int32), ("B", ctypes.c_int32),
                ("I", ctypes.c_int32), ("H", ctypes.c_int32),
                ("layers", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("spill", ctypes.c_int32), ("spill_chunk_steps", ctypes.c_int32),
                ("device_stack_budget_bytes", ctypes.c_int64),
                ("recompute", ctypes.c_int32), ("cell", ctypes.c_int32),
                ("ponder_max", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class LoopError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


_lib = None
# Plans still open: closed by an exit hook that runs while the HIP runtime is
# alive (its own teardown happens later, in the C library's exit handlers).
_live_plans: "weakref.WeakSet[Plan]" = weakref.WeakSet()


def _close_live_plans() -> None:
    for plan in list(_live_plans):
        try:
            plan.close()
        except Exception:
            pass


atexit.register(_close_live_plans)


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load the HIP library (once).  Raises if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(
            f"{path} is missing: build it with `python -m paper_1805_01772_amd.build_lib` "
            "(or __graft_entry__.build()); there is no CPU fallback")
    # torch ships its own HIP runtime (SONAME libamdhip64.so.7).  Loading torch
    # first makes the library bind to that same runtime instead of a second
    # copy, so torch's streams and device pointers are valid here.
    import torch  # noqa: F401
    lib = ctypes.CDLL(path)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    lib.ll_plan_create.argtypes = [ctypes.POINTER(ll_desc), ctypes.c_int, ctypes.POINTER(vp)]
    lib.ll_plan_destroy.argtypes = [vp]
    lib.ll_plan_stack_bytes.argtypes = [vp, ctypes.POINTER(i64), ctypes.POINTER(i64)]
    lib.ll_plan_geometry.argtypes = [vp, ctypes.POINTER(i32), ctypes.POINTER(i32),
                                     ctypes.POINTER(i32), ctypes.POINTER(i32),
                                     ctypes.POINTER(i32), ctypes.POINTER(i32)]
    lib.lstm_loop_fwd.argtypes = [vp, vp, vp, vp, ctypes.POINTER(vp), ctypes.POINTER(vp),
                                  vp, vp, vp, vp, vp, vp, i32]
    lib.lstm_loop_bwd.argtypes = [vp, vp, vp, vp, ctypes.POINTER(vp), vp, vp, vp, vp,
                                  ctypes.POINTER(vp), ctypes.POINTER(vp), vp, vp]
    lib.ll_status_sync.argtypes = [vp, ctypes.POINTER(i32)]
    lib.ll_plan_set_timing.argtypes = [vp, i32]
    lib.ll_plan_set_timing_stages.argtypes = [vp, ctypes.c_uint32]
    lib.ll_plan_read_timing.argtypes = [vp, i32, ctypes.POINTER(ctypes.c_double),
                                        ctypes.POINTER(i64)]
    lib.ll_measure_mfma_peak.argtypes = [ctypes.c_int, i32, i32, ctypes.POINTER(ctypes.c_double)]
    lib.ll_eval_activations.argtypes = [ctypes.c_int32, vp, vp, i64, i32]
    lib.lstm_loop_fwd_noalloc.argtypes = [ctypes.POINTER(ll_desc), vp, vp, vp, ctypes.POINTER(vp),
                                          ctypes.POINTER(vp), vp, vp, vp, vp, vp, vp, vp]
    lib.ll_last_error.restype = ctypes.c_char_p
    lib.ll_version.restype = ctypes.c_char_p
    for name in ("ll_plan_create", "ll_plan_destroy", "ll_plan_stack_bytes", "ll_plan_geometry",
                 "lstm_loop_fwd", "lstm_loop_bwd", "ll_status_sync", "ll_plan_set_timing",
                 "ll_plan_set_timing_stages", "ll_plan_read_timing", "ll_measure_mfma_peak",
                 "ll_eval_activations", "lstm_loop_fwd_noalloc"):
        getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def ll_last_error() -> str:
    return load_library().ll_last_error().decode()


def ll_measure_mfma_peak(dtype: str, shape: int = 32, device: int = 0) -> float:
    """Sustained dense matrix-core rate of the device in TFLOP/s
    (dtype "bf16" or "f32"; shape 16: the loops' 16x16 k-step, 32: 32x32)."""
    v = ctypes.c_double()
    _check(load_library().ll_measure_mfma_peak(device, LL_BF16 if dtype == "bf16" else LL_F32, shape,
                                               ctypes.byref(v)))
    return v.value


def ll_eval_activations(x, fn: str):
    """The loop kernels' sigmoid ("sigmoid") or tanh ("tanh") of the float32
    device tensor x (ll_eval_activations); returns a new tensor."""
    import torch
    out = torch.empty_like(x)
    _check(load_library().ll_eval_activations(x.device.index or 0, _ptr(x), _ptr(out), x.numel(),
                                              {"sigmoid": 0, "tanh": 1}[fn]))
    return out


def ll_version() -> str:
    return load_library().ll_version().decode()


def _check(status: int) -> None:
    if status != LL_OK:
        raise LoopError(status, ll_last_error())


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("tensors passed to the library must live on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensors passed to the library must be contiguous")
    return t.data_ptr()


def _ptr_array(ts):
    arr = (ctypes.c_void_p * len(ts))()
    for i, t in enumerate(ts):
        arr[i] = _ptr(t)
    return arr


def _stream(stream) -> Optional[int]:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


class Plan:
    """Owner of an ll_plan (ll_plan_create / ll_plan_destroy)."""

    def __init__(self, T_max: int, B: int, I: int, H: int, layers: int = 1,
                 dtype: str = "f32", spill: int = 0, spill_chunk_steps: int = 0,
                 device_stack_budget_bytes: int = 0, device: int = 0, recompute: int = 0,
                 cell: int = 0, ponder_max: int = 0):
        lib = load_library()
        self._lib = lib
        self.desc = make_desc(T_max, B, I, H, layers, dtype, spill, spill_chunk_steps,
                              device_stack_budget_bytes, recompute, cell, ponder_max)
        self.dtype = dtype
        self.device = device
        h = ctypes.c_void_p()
        _check(lib.ll_plan_create(ctypes.byref(self.desc), device, ctypes.byref(h)))
        self._h = h
        _live_plans.add(self)

    def close(self) -> None:
        if getattr(self, "_h", None) is not None and self._h.value:
            self._lib.ll_plan_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    @property
    def handle(self) -> int:
        return self._h.value

    def stack_bytes(self):
        d, h = ctypes.c_int64(), ctypes.c_int64()
        _check(self._lib.ll_plan_stack_bytes(self._h, ctypes.byref(d), ctypes.byref(h)))
        return d.value, h.value

    def geometry(self):
        n, hj, rg, xl, wf, dwp = (ctypes.c_int32() for _ in range(6))
        _check(self._lib.ll_plan_geometry(self._h, ctypes.byref(n), ctypes.byref(hj),
                                          ctypes.byref(rg), ctypes.byref(xl), ctypes.byref(wf),
                                          ctypes.byref(dwp)))
        form = {LL_LOOPS_GRID: "grid", LL_LOOPS_XCD: "xcd", LL_LOOPS_CHIP: "chip"}[xl.value]
        return dict(workgroups=n.value, units_per_workgroup=hj.value, row_groups=rg.value,
                    loops=form, xcd_local=form == "xcd", wavefront=bool(wf.value),
                    dw_in_place=[bool(dwp.value >> l & 1) for l in range(self.desc.layers)])

    def fwd(self, x, seq_len, W: Sequence, bias: Sequence, h0, c0, y, hT, cT,
            trip_count=None, save_for_backward: bool = True, stream=None) -> None:
        """lstm_loop_fwd (asynchronous on `stream`, default: torch's current)."""
        _check(self._lib.lstm_loop_fwd(
            self._h, _stream(stream), _ptr(x), _ptr(seq_len), _ptr_array(W), _ptr_array(bias),
            _ptr(h0), _ptr(c0), _ptr(y), _ptr(hT), _ptr(cT), _ptr(trip_count),
            1 if save_for_backward else 0))

    def bwd(self, x, seq_len, W: Sequence, dy, dhT, dcT, dx, dW: Sequence, dbias: Sequence,
            dh0, dc0, stream=None) -> None:
        """lstm_loop_bwd (asynchronous on `stream`); x, seq_len and W are the
        tensors the saved forward was given."""
        _check(self._lib.lstm_loop_bwd(
            self._h, _stream(stream), _ptr(x), _ptr(seq_len), _ptr_array(W), _ptr(dy),
            _ptr(dhT), _ptr(dcT), _ptr(dx), _ptr_array(dW), _ptr_array(dbias), _ptr(dh0),
            _ptr(dc0)))

    def set_timing(self, enable) -> None:
        """ll_plan_set_timing: clear the stage accumulators, start/stop recording
        every stage; a collection of stage names records only those
        (ll_plan_set_timing_stages)."""
        if isinstance(enable, (bool, int)):
            _check(self._lib.ll_plan_set_timing(self._h, 1 if enable else 0))
            return
        mask = 0
        for name in enable:
            mask |= 1 << STAGES.index(name)
        _check(self._lib.ll_plan_set_timing_stages(self._h, mask))

    def read_timing(self) -> dict:
        """ll_plan_read_timing for every stage: {name: (total_ms, instances)}."""
        out = {}
        for i, name in enumerate(STAGES):
            ms, n = ctypes.c_double(), ctypes.c_int64()
            _check(self._lib.ll_plan_read_timing(self._h, i, ctypes.byref(ms), ctypes.byref(n)))
            out[name] = (ms.value, n.value)
        return out

    def status_sync(self) -> int:
        """ll_status_sync: wait, then return (and clear) the device error word."""
        e = ctypes.c_int32()
        _check(self._lib.ll_status_sync(self._h, ctypes.byref(e)))
        return e.value


def lstm_loop_fwd(plan: Plan, *args, **kw):
    return plan.fwd(*args, **kw)


def lstm_loop_bwd(plan: Plan, *args, **kw):
    return plan.bwd(*args, **kw)


NOALLOC_SCRATCH_BYTES = 128 << 20   # LL_NOALLOC_SCRATCH_BYTES


def make_desc(T_max: int, B: int, I: int, H: int, layers: int = 1, dtype: str = "f32",
              spill: int = 0, spill_chunk_steps: int = 0, device_stack_budget_bytes: int = 0,
              recompute: int = 0, cell: int = 0, ponder_max: int = 0) -> ll_desc:
    return ll_desc(T_max, B, I, H, layers,
                   LL_BF16 if dtype == "bf16" else LL_F32 if dtype == "f32" else int(dtype),
                   spill, spill_chunk_steps, device_stack_budget_bytes, recompute, cell, ponder_max, 0)


def lstm_loop_fwd_noalloc(desc: ll_desc, x, seq_len, W: Sequence, bias: Sequence, h0, c0, y, hT,
                          cT, trip_count=None, device_error=None, stream=None) -> None:
    """lstm_loop_fwd_noalloc: the inference forward without a plan, every
    buffer carved from the library's scratch array (asynchronous on `stream`)."""
    _check(load_library().lstm_loop_fwd_noalloc(
        ctypes.byref(desc), _stream(stream), _ptr(x), _ptr(seq_len), _ptr_array(W), _ptr_array(bias),
        _ptr(h0), _ptr(c0), _ptr(y), _ptr(hT), _ptr(cT), _ptr(trip_count), _ptr(device_error)))


def ll_plan_create(*args, **kw) -> Plan:
    return Plan(*args, **kw)


def ll_plan_destroy(plan: Plan) -> None:
    plan.close()


def ll_status_sync(plan: Plan) -> int:
    return plan.status_sync()


def ll_plan_stack_bytes(plan: Plan):
    return plan.stack_bytes()
