"""C ABI checks that need no GPU: the library loads, exports every function
include/mosa.h declares, sizes its workspace and rejects bad arguments before
touching the device."""
import ctypes
import os
import re

import pytest

from paper_2505_00315_amd import mosa

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "mosa.h")).read()
    return sorted(set(re.findall(r"^(?:int|const char\*)\s+(mosa_\w+)\s*\(", src, re.M)))


def test_header_declares_the_binding_symbols():
    assert declared_functions() == sorted(mosa.SYMBOLS)


def test_library_exports_every_declared_symbol():
    L = mosa.lib()
    for name in declared_functions():
        assert hasattr(L, name), name
        assert ctypes.cast(getattr(L, name), ctypes.c_void_p).value


def test_status_strings():
    for st in (0, -1, -2, -3, -4, 7):
        assert isinstance(mosa.status_string(st), str) and mosa.status_string(st)


def test_workspace_size_and_layout():
    s = mosa.make_shape(8, 1024, 1024, 256, 64, 16, True, 4, "bf16")
    saved, scratch = mosa.workspace_size(s)
    off = mosa.saved_offsets(s)
    assert off["total"] == saved
    B, T, H, Hd, k, dh = 8, 1024, 256, 4, 16, 64
    assert off["QKV"] >= B * H * k * 4 * 2 + B * H * T * 2  # after I, r and the slot map
    assert saved >= 4 * B * H * k * dh * 2 + 4 * B * Hd * T * dh * 2
    assert scratch >= B * H * T * 4
    for v in off.values():
        assert v % 256 == 0


@pytest.mark.parametrize("kw,status", [
    (dict(k=0), mosa.MOSA_ERR_INVALID_ARG),
    (dict(k=1025), mosa.MOSA_ERR_INVALID_ARG),
    (dict(batch=0), mosa.MOSA_ERR_INVALID_ARG),
    (dict(heads=0, dense_heads=0), mosa.MOSA_ERR_INVALID_ARG),
    (dict(d_head=48), mosa.MOSA_ERR_UNSUPPORTED),
    (dict(d_model=96), mosa.MOSA_ERR_UNSUPPORTED),
    (dict(seq_len=20000, k=10), mosa.MOSA_ERR_UNSUPPORTED),
    # variants
    (dict(fixed_stride=64, k=17), mosa.MOSA_ERR_INVALID_ARG),    # 16 * 64 > T - 1
    (dict(fixed_stride=8, first_token=True), mosa.MOSA_ERR_INVALID_ARG),
    (dict(rope=True, rope_base=1.0), mosa.MOSA_ERR_INVALID_ARG),
    (dict(window=8, causal=False, dense_heads=1), mosa.MOSA_ERR_INVALID_ARG),
    (dict(fixed_stride=-1), mosa.MOSA_ERR_INVALID_ARG),
])
def test_invalid_shapes_rejected(kw, status):
    base = dict(batch=2, seq_len=1024, d_model=128, heads=4, d_head=32, k=16, causal=True, dense_heads=0,
                dtype="bf16")
    base.update(kw)
    s = mosa.make_shape(**base)
    if kw.get("k", 1) == 0:
        s.k = 0
    with pytest.raises(mosa.MosaError) as ei:
        mosa.workspace_size(s)
    assert ei.value.status == status


def test_bad_dtype_and_causal_rejected():
    s = mosa.make_shape(1, 64, 64, 1, 32, 8)
    s.dtype = 7
    with pytest.raises(mosa.MosaError):
        mosa.workspace_size(s)
    s = mosa.make_shape(1, 64, 64, 1, 32, 8)
    s.causal = 2
    with pytest.raises(mosa.MosaError):
        mosa.workspace_size(s)


def _call_forward(shape, X=0x1000, Y=0x2000, saved=0x10000, scratch=0x20000, saved_bytes=1 << 40,
                  scratch_bytes=1 << 40, weights=None):
    w = mosa.Weights(*([0x3000] * 5 + [None] * 4)) if weights is None else weights
    return mosa.lib().mosa_forward(ctypes.byref(shape), ctypes.c_void_p(X), ctypes.byref(w), ctypes.c_void_p(Y),
                                   0, None, None, ctypes.c_void_p(saved), saved_bytes, ctypes.c_void_p(scratch),
                                   scratch_bytes, None)


def test_forward_rejects_before_any_device_work():
    s = mosa.make_shape(1, 64, 64, 1, 32, 8)
    assert _call_forward(s, X=0) == mosa.MOSA_ERR_INVALID_ARG
    assert _call_forward(s, X=0x1001) == mosa.MOSA_ERR_INVALID_ARG       # misaligned
    assert _call_forward(s, saved=0x10010) == mosa.MOSA_ERR_INVALID_ARG  # not 256-aligned
    assert _call_forward(s, saved_bytes=16) == mosa.MOSA_ERR_WORKSPACE
    assert _call_forward(s, scratch_bytes=16) == mosa.MOSA_ERR_WORKSPACE
    nul = mosa.Weights(*([None] * 9))
    assert _call_forward(s, weights=nul) == mosa.MOSA_ERR_INVALID_ARG
    dense = mosa.make_shape(1, 64, 64, 1, 32, 8, dense_heads=1)
    assert _call_forward(dense) == mosa.MOSA_ERR_INVALID_ARG  # dense weights missing


def test_backward_rejects_before_any_device_work():
    s = mosa.make_shape(1, 64, 64, 1, 32, 8)
    w = mosa.Weights(*([0x3000] * 5 + [None] * 4))
    g = mosa.Grads(*([0x4000] * 5 + [None] * 4))
    L = mosa.lib()
    st = L.mosa_backward(ctypes.byref(s), ctypes.c_void_p(0x1000), ctypes.byref(w), None, ctypes.c_void_p(0x10000),
                         1 << 40, ctypes.c_void_p(0x2000), 0, ctypes.byref(g), ctypes.c_void_p(0x20000), 1 << 40,
                         None)
    assert st == mosa.MOSA_ERR_INVALID_ARG  # dY missing


def test_variant_fields_and_rope_table_offset():
    s = mosa.make_shape(2, 1024, 128, 4, 64, 64, True, 1, "bf16", first_token=True, rope=True, rope_base=500.0)
    assert (s.first_token, s.rope, s.rope_base) == (1, 1, 500.0)
    off = mosa.saved_offsets(s)
    assert off["rope"] % 256 == 0 and off["total"] >= off["rope"] + 1024 * (64 // 4) * 8
    s2 = mosa.make_shape(2, 1024, 128, 4, 64, 64, True, 1, "bf16")
    assert mosa.saved_offsets(s2)["total"] < off["total"]
    fixed = mosa.make_shape(2, 1024, 128, 4, 64, 16, True, 0, "bf16", fixed_stride=64)
    mosa.workspace_size(fixed)  # 15 * 64 <= 1023


def test_adaptive_k():
    # Section 3.5: k = max(floor(T / rho), 2), at most T
    assert mosa.adaptive_k(1024, 64) == 16
    assert mosa.adaptive_k(1024, 8) == 128
    assert mosa.adaptive_k(10, 8) == 2
    assert mosa.adaptive_k(1, 8) == 1
    with pytest.raises(ValueError):
        mosa.adaptive_k(0, 8)
