"""C ABI checks that need no GPU: the library loads, exports every function that
include/*.h declares, and rejects bad arguments before touching the device."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    names = set()
    for h in sorted(os.listdir(os.path.join(ROOT, "include"))):
        if h.endswith(".h"):
            src = open(os.path.join(ROOT, "include", h)).read()
            src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
            names |= set(re.findall(r"\b(wn_[a-z_]+)\s*\(", src))
    return sorted(names)


@pytest.fixture(scope="module")
def lib():
    import paper_1702_07825_amd as wn
    if not os.path.exists(wn.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    return wn.load_library()


def test_exports_every_declared_function(lib):
    import paper_1702_07825_amd as wn
    names = _declared()
    assert set(names) == set(wn.EXPORTED)
    for n in names:
        assert hasattr(lib, n), n


def test_error_strings(lib):
    for code in (0, -1, -2, -3, -4, -5, -6):
        assert lib.wn_error_string(code).decode()
    assert lib.wn_error_string(99).decode() == "unknown error"


def _cfg(wn, **kw):
    import numpy as np
    d = np.array(kw.pop("dil", [1, 2, 4, 8]), np.int32)
    c = wn.Config(kw.get("L", 4), kw.get("r", 16), kw.get("s", 32), kw.get("a", 256),
                  d.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), kw.get("taps", 1), kw.get("init", 128),
                  kw.get("dtype", 0), kw.get("nl", 0))
    return c, d


def _weights(wn):
    import numpy as np
    import synth
    w = synth.make_weights(4, 16, 32)
    keep = {k: np.ascontiguousarray(w[k]) for k in wn.WEIGHT_FIELDS}
    return wn.Weights(*[keep[k].ctypes.data_as(ctypes.POINTER(ctypes.c_float)) for k in wn.WEIGHT_FIELDS]), keep


@pytest.mark.parametrize("kw,code", [
    (dict(L=0), -1), (dict(L=65), -1), (dict(init=256), -1), (dict(init=-1), -1), (dict(dtype=7), -1),
    (dict(dil=[1, 0, 4, 8]), -1), (dict(taps=3), -1), (dict(r=0), -1), (dict(nl=2), -1), (dict(nl=-1), -1),
    (dict(a=255), -2), (dict(r=48, s=32), -2), (dict(r=16, s=64), -2),
])
def test_create_rejects_before_any_device_call(lib, kw, code):
    import paper_1702_07825_amd as wn
    c, _d = _cfg(wn, **kw)
    w, _keep = _weights(wn)
    h = ctypes.c_void_p()
    assert lib.wn_create(ctypes.byref(c), ctypes.byref(w), ctypes.byref(h)) == code
    assert h.value is None
    assert lib.wn_last_error().decode()


def test_null_arguments(lib):
    import paper_1702_07825_amd as wn
    c, _d = _cfg(wn)
    h = ctypes.c_void_p()
    assert lib.wn_create(None, None, ctypes.byref(h)) == -1
    assert lib.wn_create(ctypes.byref(c), None, ctypes.byref(h)) == -1
    w, _keep = _weights(wn)
    w.w_out = None
    assert lib.wn_create(ctypes.byref(c), ctypes.byref(w), ctypes.byref(h)) == -1
    assert lib.wn_workspace_bytes(None, 1) == 0
    assert lib.wn_generate(None, 1, 1, None, None, None, None, 0, 1, None) == -1
    assert lib.wn_teacher_force(None, 1, 1, None, None, None, None, 0, 1, None) == -1
    assert lib.wn_status(None, None, None) == -1
    assert lib.wn_abort(None, 1) == -1
    assert lib.wn_kernel_variant(None, 1) == b""
    wg, rep = ctypes.c_int32(7), ctypes.c_int32(7)
    assert lib.wn_launch_info(None, 1, ctypes.byref(wg), ctypes.byref(rep)) == -1
    assert (wg.value, rep.value) == (7, 7)
    lib.wn_destroy(None)


def test_binding_fails_loudly_without_library(tmp_path):
    import paper_1702_07825_amd as wn
    with pytest.raises(RuntimeError):
        wn.load_library.__wrapped__(str(tmp_path / "missing.so")) if hasattr(wn.load_library, "__wrapped__") \
            else _load_missing(wn, str(tmp_path / "missing.so"))


def _load_missing(wn, path):
    saved = wn._lib
    wn._lib = None
    try:
        wn.load_library(path)
    finally:
        wn._lib = saved


def test_conditioning_network_rejects_before_any_device_call(lib):
    import paper_1702_07825_amd as wn
    vp = ctypes.c_void_p
    out = vp()
    w = wn.CondWeights(*([ctypes.cast(ctypes.create_string_buffer(4), ctypes.POINTER(ctypes.c_float))] * 4))
    for cfg in [wn.CondConfig(0, 8, 2, 4, 256, 16000), wn.CondConfig(227, 0, 2, 4, 256, 16000),
                wn.CondConfig(227, 8, 0, 4, 256, 16000), wn.CondConfig(227, 8, 2, 4, 0, 16000),
                wn.CondConfig(227, 8, 4096, 4, 256, 16000)]:
        assert lib.wn_cond_create(ctypes.byref(cfg), ctypes.byref(w), ctypes.byref(out)) == wn.WN_EINVAL
        assert lib.wn_last_error().decode()
    assert lib.wn_cond_create(None, None, None) == wn.WN_EINVAL
    assert lib.wn_cond_workspace_bytes(None, 1, 1) == 0
    assert lib.wn_condition(None, 1, 1, None, 1, None, None, 0, None) == wn.WN_EINVAL
    assert lib.wn_condition_static(None, 1, 1, None, 1, None, None) == wn.WN_EINVAL
    lib.wn_cond_destroy(None)


def test_static_scratch_size_matches_the_header():
    """The binding's COND_SCRATCH_BYTES is the header's WN_COND_SCRATCH_BYTES."""
    import paper_1702_07825_amd as wn
    src = open(os.path.join(ROOT, "include", "wn_cond.h")).read()
    m = re.search(r"#define\s+WN_COND_SCRATCH_BYTES\s+\(\(size_t\)(\d+)\s*<<\s*(\d+)\)", src)
    assert m
    assert wn.COND_SCRATCH_BYTES == int(m.group(1)) << int(m.group(2))
