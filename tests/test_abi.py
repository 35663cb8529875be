"""Host-side checks of the C-ABI library (no GPU needed).

- the shared library loads and exports every function include/lstmloop.h
  declares;
- descriptor validation rejects bad problems before touching a device.
"""
import ctypes
import os
import re

import pytest

from paper_1805_01772_amd import lstmloop as ll

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lstmloop.h")


def _lib():
    if not os.path.exists(ll.LIB_PATH):
        from paper_1805_01772_amd import build_lib
        build_lib.build()
    return ll.load_library()


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[A-Za-z_][A-Za-z0-9_]*\s*\*?\s*([a-z_][a-z0-9_]*)\s*\(",
                       text, flags=re.M)
    return sorted(set(names))


def test_header_declares_the_entry_points():
    names = _declared_functions()
    for n in ("ll_plan_create", "ll_plan_destroy", "lstm_loop_fwd", "lstm_loop_bwd",
              "ll_status_sync", "ll_last_error"):
        assert n in names


def test_library_exports_every_declared_symbol():
    lib = _lib()
    for name in _declared_functions():
        assert hasattr(lib, name), name
    assert set(ll.EXPORTED) == set(_declared_functions())


def test_version_string():
    _lib()
    assert "gfx950" in ll.ll_version()


@pytest.mark.parametrize("fields,status", [
    (dict(T_max=0), ll.LL_EINVAL),
    (dict(B=0), ll.LL_EINVAL),
    (dict(layers=3), ll.LL_EINVAL),
    (dict(dtype=7), ll.LL_EINVAL),
    (dict(cell=3, spill=1), ll.LL_EUNSUPPORTED),
    (dict(cell=3, recompute=1), ll.LL_EUNSUPPORTED),
    (dict(cell=-1), ll.LL_EINVAL),
    (dict(cell=1, spill=1), ll.LL_EUNSUPPORTED),
    (dict(cell=2, spill=1), ll.LL_EUNSUPPORTED),
    (dict(cell=2, recompute=1), ll.LL_EUNSUPPORTED),
    (dict(spill=2), ll.LL_EINVAL),
    (dict(recompute=2), ll.LL_EINVAL),
    (dict(recompute=1, spill=1), ll.LL_EUNSUPPORTED),
    (dict(H=48), ll.LL_EUNSUPPORTED),
    (dict(I=6), ll.LL_EUNSUPPORTED),
    (dict(B=5000), ll.LL_EUNSUPPORTED),
    (dict(reserved=1), ll.LL_EINVAL),
    (dict(cell=4, ponder_max=0), ll.LL_EINVAL),
    (dict(cell=4, ponder_max=9), ll.LL_EINVAL),
    (dict(cell=4, ponder_max=3, layers=2), ll.LL_EUNSUPPORTED),
    (dict(cell=4, ponder_max=3, spill=1), ll.LL_EUNSUPPORTED),
    (dict(cell=0, ponder_max=2), ll.LL_EINVAL),
    (dict(cell=5), ll.LL_EINVAL),
    (dict(reserved=-7), ll.LL_EINVAL),
])
def test_descriptor_validation(fields, status):
    lib = _lib()
    base = dict(T_max=8, B=4, I=32, H=32, layers=1, dtype=ll.LL_BF16, spill=0,
                spill_chunk_steps=0, device_stack_budget_bytes=0, recompute=0, cell=0, ponder_max=0,
                reserved=0)
    base.update(fields)
    d = ll.ll_desc(**base)
    h = ctypes.c_void_p(123)
    st = lib.ll_plan_create(ctypes.byref(d), 0, ctypes.byref(h))
    assert st == status, ll.ll_last_error()
    assert h.value is None
    assert ll.ll_last_error() != ""


def test_null_arguments_rejected():
    lib = _lib()
    assert lib.ll_plan_create(None, 0, None) == ll.LL_EINVAL
    assert lib.lstm_loop_bwd(None, None, None, None, None, None, None, None, None, None, None,
                             None, None) == ll.LL_EINVAL
    assert lib.ll_plan_destroy(None) == ll.LL_OK


def test_binding_constants_match_the_header():
    """Stage names and status codes of the binding follow the header's enums."""
    text = open(HEADER).read()
    stages = dict((int(v), k.lower()) for k, v in re.findall(r"LL_STAGE_([A-Z_]+) = (\d+)", text))
    count = [k for k in stages.values() if k == "count"]
    assert count and max(stages) == len(ll.STAGES)
    assert tuple(stages[i] for i in range(len(ll.STAGES))) == ll.STAGES
    status = dict(re.findall(r"(LL_E[A-Z]+) = (\d+)", text))
    for name, val in status.items():
        if hasattr(ll, name):
            assert getattr(ll, name) == int(val), name
    forms = dict(re.findall(r"#define (LL_LOOPS_[A-Z]+) (\d+)", text))
    assert len(forms) == 3
    for name, val in forms.items():
        assert getattr(ll, name) == int(val), name


def test_descriptor_layout_matches_the_header():
    """The binding's ll_desc has the header's fields in the header's order
    (the C struct is passed by pointer, so a mismatch would shift fields)."""
    text = open(HEADER).read()
    body = text[text.index("typedef struct {", text.index("Problem description")):]
    body = body[:body.index("} ll_desc;")]
    fields = re.findall(r"^\s*(int32_t|int64_t)\s+([a-z_A-Z0-9]+);", body, flags=re.M)
    names = [f[1] for f in fields]
    assert names == [f[0] for f in ll.ll_desc._fields_]
    for (ctype, name), (bname, btype) in zip(fields, ll.ll_desc._fields_):
        assert ctypes.sizeof(btype) == (8 if ctype == "int64_t" else 4), name
    assert names[-1] == "reserved"


def test_bwd_signature_takes_the_forward_operands():
    """lstm_loop_bwd takes x, seq_len and W (checked against the saved
    forward) before the gradients."""
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    decl = text[text.index("ll_status lstm_loop_bwd("):]
    decl = decl[:decl.index(");")]
    params = [p.strip() for p in decl[decl.index("(") + 1:].split(",")]
    names = [re.findall(r"([A-Za-z_0-9]+)$", p)[0] for p in params]
    assert names[:5] == ["plan", "stream", "x", "seq_len", "W"]
    assert names[5:] == ["dy", "dhT", "dcT", "dx", "dW", "dbias", "dh0", "dc0"]
    assert len(ll.load_library().lstm_loop_bwd.argtypes) == len(names)
