"""CPU oracle of the Mixture of Sparse Attention layer (fp64, plain loops in C).

TEST INFRASTRUCTURE ONLY: this package may be imported by ``tests/``, by
``__graft_entry__.smoke()`` and by the CPU-baseline leg of ``bench.py``.  The
GPU product path (``paper_2505_00315_amd``) never imports it; the two share no
code.  What the oracle computes, step by step, is documented in
``mosa_oracle.c`` with the paper passages it follows (Section 2.2, Eq. 1-3).

Inputs are numpy arrays holding the exact stored values: ``float32`` for the
fp32 storage type, ``uint16`` bit patterns for bf16.  Outputs are float64.
"""
import ctypes
import os

import numpy as np

from . import build as _build

F32, BF16, F64 = 0, 1, 2

_lib = None


def lib():
    """Load (building on first use if needed) the oracle shared library."""
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        _lib = ctypes.CDLL(_build.LIB)
        _declare(_lib)
    return _lib


_p = ctypes.c_void_p
_i = ctypes.c_int


class Options(ctypes.Structure):
    """Layer variants (``orc_options`` in mosa_oracle.c): forced first token,
    fixed sparse stride, rotary encoding at positions I, local window of the
    dense heads."""
    _fields_ = [("first_token", ctypes.c_int32), ("fixed_stride", ctypes.c_int32),
                ("rope", ctypes.c_int32), ("window", ctypes.c_int32), ("rope_base", ctypes.c_double)]


def options(first_token=False, fixed_stride=0, rope=False, rope_base=10000.0, window=0):
    return Options(int(bool(first_token)), int(fixed_stride), int(bool(rope)), int(window), float(rope_base))


def _declare(L):
    L.orc_fsum.argtypes = [_p, ctypes.c_int64, _p]
    L.orc_router_keys.argtypes = [_i, _i, _i, _i, _i, _p, _p, _p]
    L.orc_select.argtypes = [_i, _i, _i, _i, _p, _p]
    L.orc_head_attend.argtypes = [_i, _i, _i, _i, _i, _p, _p, _p, _p, _p, _p, _p, _p]
    L.orc_forward.argtypes = [_i] * 9 + [_p] * 18
    L.orc_backward.argtypes = [_i] * 9 + [_p] * 21
    L.orc_forward_ex.argtypes = [_i] * 9 + [_p] * 18 + [ctypes.POINTER(Options)]
    L.orc_backward_ex.argtypes = [_i] * 9 + [_p] * 21 + [ctypes.POINTER(Options)]
    L.orc_select_ex.argtypes = [_i, _i, _i, _i, _i, _p, _p]
    L.orc_rope.argtypes = [_i, _i, ctypes.c_double, _p, _i, _p]
    L.orc_max_threads.argtypes = []
    L.orc_set_threads.argtypes = [_i]
    L.orc_set_threads.restype = None
    for name in ("orc_fsum", "orc_router_keys", "orc_select", "orc_head_attend",
                 "orc_forward", "orc_backward", "orc_max_threads", "orc_forward_ex", "orc_backward_ex",
                 "orc_select_ex", "orc_rope"):
        getattr(L, name).restype = ctypes.c_int


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _check(status, what):
    if status != 0:
        raise RuntimeError(f"oracle {what} failed with status {status}")


def _dtype_code(arr):
    if arr.dtype == np.float32:
        return F32
    if arr.dtype == np.uint16:
        return BF16
    if arr.dtype == np.float64:
        return F64  # oracle self-checks only (finite differences)
    raise TypeError(f"oracle inputs must be float32, uint16 (bf16 bits) or float64, got {arr.dtype}")


def _c(a):
    return None if a is None else np.ascontiguousarray(a)


def set_threads(n: int) -> None:
    lib().orc_set_threads(int(n))


def max_threads() -> int:
    return int(lib().orc_max_threads())


def fsum(values) -> float:
    """Correctly rounded sum of float64 values (exact expansion sum)."""
    v = np.ascontiguousarray(values, dtype=np.float64)
    out = np.zeros(1, dtype=np.float64)
    _check(lib().orc_fsum(_ptr(v), v.size, _ptr(out)), "fsum")
    return float(out[0])


def router_keys(X, Wr):
    """keys[b,h,t] = RN64(sum_c X[b,t,c] Wr[h,c]) with the sum taken exactly."""
    X, Wr = _c(X), _c(Wr)
    B, T, d = X.shape
    H = Wr.shape[0]
    keys = np.empty((B, H, T), dtype=np.float64)
    _check(lib().orc_router_keys(_dtype_code(X), B, T, d, H, _ptr(X), _ptr(Wr), _ptr(keys)),
           "router_keys")
    return keys


def select(keys, k, first_token=False):
    """Expert-choice TopK per (b,h) row of keys [B,H,T]: I [B,H,k] ascending
    (first_token: token 0 plus the best k - 1 of t >= 1)."""
    keys = np.ascontiguousarray(keys, dtype=np.float64)
    B, H, T = keys.shape
    I = np.empty((B, H, k), dtype=np.int32)
    _check(lib().orc_select_ex(B, H, T, k, int(bool(first_token)), _ptr(keys), _ptr(I)), "select")
    return I


def rope(v, positions, base=10000.0, sign=1):
    """Rotary encoding of the rows of v [n, dh] at the given positions (sign -1:
    the inverse rotation); returns a new float64 array."""
    out = np.array(v, dtype=np.float64, copy=True, order="C")
    p = np.ascontiguousarray(positions, dtype=np.int32)
    n, dh = out.shape
    assert p.shape == (n,)
    _check(lib().orc_rope(n, dh, float(base), _ptr(p), int(sign), _ptr(out)), "rope")
    return out


def head_attend(Xb, Wq, Wk, Wv, Wo, I, r=None, causal=True, Y=None):
    """One head over the token set I with router values r (None: all ones).
    Xb [T,d], W* [d,dh], Wo [dh,d] as float64; returns Y [T,d] with
    Y[I_i] += r_i A_i W^O."""
    Xb = np.ascontiguousarray(Xb, dtype=np.float64)
    T, d = Xb.shape
    dh = Wq.shape[1]
    I = np.ascontiguousarray(I, dtype=np.int32)
    n = I.size
    ws = [np.ascontiguousarray(w, dtype=np.float64) for w in (Wq, Wk, Wv, Wo)]
    rr = None if r is None else np.ascontiguousarray(r, dtype=np.float64)
    out = np.zeros((T, d), dtype=np.float64) if Y is None else Y
    _check(lib().orc_head_attend(T, d, dh, n, int(causal), _ptr(Xb), *[_ptr(w) for w in ws],
                                 _ptr(I), _ptr(rr), _ptr(out)), "head_attend")
    return out


def _unpack(inp):
    X = _c(inp["X"])
    H = inp["Wq"].shape[0] if inp.get("Wq") is not None else 0
    Hd = inp["Wq_d"].shape[0] if inp.get("Wq_d") is not None else 0
    ws = [_c(inp.get(n)) for n in ("Wr", "Wq", "Wk", "Wv", "Wo", "Wq_d", "Wk_d", "Wv_d", "Wo_d")]
    if H > 0:
        dh = inp["Wq"].shape[2]
    else:
        dh = inp["Wq_d"].shape[2]
    return X, H, Hd, dh, ws


def forward(inp, k, causal=True, intermediates=False, opts=None):
    """Layer forward.  ``inp`` holds X [B,T,d] and the weights (see workloads.py).
    Returns dict with Y [B,T,d], I [B,H,k], r [B,H,k], keys [B,H,T] and, if
    ``intermediates``, Q, K, V (after the rotary encoding, if any), A
    [B,H,k,dh] of the MoSA heads (float64).  ``opts``: ``options(...)``."""
    X, H, Hd, dh, ws = _unpack(inp)
    B, T, d = X.shape
    kk = k if H > 0 else 0
    Y = np.empty((B, T, d), dtype=np.float64)
    I = np.empty((B, H, kk), dtype=np.int32)
    r = np.empty((B, H, kk), dtype=np.float64)
    keys = np.empty((B, H, T), dtype=np.float64)
    qkva = [np.empty((B, H, kk, dh), dtype=np.float64) if intermediates else None for _ in range(4)]
    o = options() if opts is None else opts
    st = lib().orc_forward_ex(_dtype_code(X), B, T, d, H, dh, kk, int(causal), Hd, _ptr(X),
                              *[_ptr(w) for w in ws], _ptr(Y), _ptr(I), _ptr(r), _ptr(keys),
                              *[_ptr(a) for a in qkva], ctypes.byref(o))
    _check(st, "forward")
    out = {"Y": Y, "I": I, "r": r, "keys": keys}
    if intermediates:
        out.update(Q=qkva[0], K=qkva[1], V=qkva[2], A=qkva[3])
    return out


def backward(inp, dY, k, causal=True, opts=None):
    """Layer backward (I held fixed).  Returns dict of float64 gradients:
    dX, dWr, dWq, dWk, dWv, dWo and, with dense heads, dWq_d, dWk_d, dWv_d, dWo_d."""
    X, H, Hd, dh, ws = _unpack(inp)
    B, T, d = X.shape
    dY = _c(dY)
    assert dY.dtype == X.dtype and dY.shape == X.shape
    kk = k if H > 0 else 0
    g = {"dX": np.empty((B, T, d), dtype=np.float64)}
    if H > 0:
        g.update(dWr=np.empty((H, d)), dWq=np.empty((H, d, dh)), dWk=np.empty((H, d, dh)),
                 dWv=np.empty((H, d, dh)), dWo=np.empty((H, dh, d)))
    if Hd > 0:
        g.update(dWq_d=np.empty((Hd, d, dh)), dWk_d=np.empty((Hd, d, dh)),
                 dWv_d=np.empty((Hd, d, dh)), dWo_d=np.empty((Hd, dh, d)))
    names = ("dWr", "dWq", "dWk", "dWv", "dWo", "dWq_d", "dWk_d", "dWv_d", "dWo_d")
    o = options() if opts is None else opts
    st = lib().orc_backward_ex(_dtype_code(X), B, T, d, H, dh, kk, int(causal), Hd, _ptr(X),
                               *[_ptr(w) for w in ws], _ptr(dY), _ptr(g["dX"]),
                               *[_ptr(g.get(n)) for n in names], ctypes.byref(o))
    _check(st, "backward")
    return g
