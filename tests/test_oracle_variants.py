"""Pins of the oracle's layer variants against facts that do not depend on it.

Variants (all from the paper): forced first-token inclusion (Section 3.2,
IsoFLOP setting), fixed sparse attention as MoSA with strided I and r = 1
(Section 3.1), rotary encoding at the original positions I (Section 2.2,
"Positional encodings"), local (sliding-window) dense heads (Section 3.4).

Routes used: Python's ``sorted`` for the selection, PyTorch's
scaled-dot-product attention over explicit masks, closed forms of special
cases (window 1, k = 1, rotations of one pair), invariants of rotations,
and central finite differences for the backward pass.
"""
import math
from fractions import Fraction

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import workloads as wl

pytestmark = pytest.mark.filterwarnings("ignore::UserWarning")


def to64(a):
    if a is None or a.dtype == np.float64:
        return a
    return wl.as_f32(a).astype(np.float64)


def exact_keys(X, Wr):
    """Router logits of one (b, h) row summed with exact rationals, rounded once."""
    return [float(sum((Fraction(float(x)) * Fraction(float(w)) for x, w in zip(row, Wr)), Fraction(0)))
            for row in X]


def sdpa(q, k, v, mask):
    q, k, v = (torch.from_numpy(np.ascontiguousarray(a))[None, None] for a in (q, k, v))
    return F.scaled_dot_product_attention(q, k, v, attn_mask=torch.from_numpy(mask)[None, None])[0, 0].numpy()


# --------------------------------------------------------------------------
# Forced first token (Section 3.2)
# --------------------------------------------------------------------------

def test_first_token_select_matches_sorted(orc):
    rng = np.random.default_rng(3)
    B, H, T, k = 2, 3, 50, 9
    keys = rng.integers(-6, 6, size=(B, H, T)).astype(np.float64)  # many ties
    keys[0, 0, 0] = -100.0  # token 0 is taken however low its score
    I = orc.select(keys, k, first_token=True)
    for b in range(B):
        for h in range(H):
            rest = sorted(range(1, T), key=lambda t: (-keys[b, h, t], t))[:k - 1]
            assert I[b, h].tolist() == sorted([0] + rest)


def test_first_token_k1_closed_form(orc):
    # k = 1: every head keeps only token 0, which attends to itself (A = V):
    # Y[b, 0] = sum_h sigma(s_0) X_0 W^V W^O, every other row zero.
    w = wl.small(batch=2, seq_len=20, d_model=16, heads=3, d_head=8, k=1, dtype="f32")
    inp = wl.make_inputs(w)
    out = orc.forward(inp, 1, opts=orc.options(first_token=True))
    X = to64(inp["X"])
    for b in range(w.batch):
        ref = np.zeros(w.d_model)
        for h in range(w.heads):
            s = exact_keys(X[b, :1], to64(inp["Wr"])[h])[0]
            ref += (1.0 / (1.0 + math.exp(-s))) * (X[b, 0] @ to64(inp["Wv"])[h] @ to64(inp["Wo"])[h])
        np.testing.assert_allclose(out["Y"][b, 0], ref, rtol=1e-12, atol=1e-13)
        assert (out["Y"][b, 1:] == 0).all()
    assert (out["I"] == 0).all()


@pytest.mark.parametrize("causal", [True, False])
def test_first_token_bruteforce(orc, causal):
    w = wl.small(batch=2, seq_len=40, d_model=16, heads=2, d_head=8, k=7, causal=causal)
    inp = wl.make_inputs(w)
    out = orc.forward(inp, w.k, causal=causal, opts=orc.options(first_token=True))
    X = to64(inp["X"])
    Y = np.zeros_like(X)
    for b in range(w.batch):
        for h in range(w.heads):
            key = exact_keys(X[b], to64(inp["Wr"])[h])
            sel = sorted([0] + sorted(range(1, w.seq_len), key=lambda t: (-key[t], t))[:w.k - 1])
            r = np.array([1.0 / (1.0 + math.exp(-key[t])) for t in sel])
            Xs = X[b, sel]
            mask = np.ones((w.k, w.k), dtype=bool)
            if causal:
                mask = np.array(sel)[:, None] >= np.array(sel)[None, :]
            A = sdpa(Xs @ to64(inp["Wq"])[h], Xs @ to64(inp["Wk"])[h], Xs @ to64(inp["Wv"])[h], mask)
            Y[b, sel] += (r[:, None] * A) @ to64(inp["Wo"])[h]
    np.testing.assert_allclose(out["Y"], Y, rtol=1e-11, atol=1e-12)


# --------------------------------------------------------------------------
# Fixed sparse attention (Section 3.1): I = 0, rho, 2 rho, ...; r = 1
# --------------------------------------------------------------------------

def test_fixed_stride_layer_matches_strided_sdpa(orc):
    w = wl.small(batch=2, seq_len=64, d_model=16, heads=3, d_head=8, k=8, dense_heads=1, dtype="f32")
    inp = wl.make_inputs(w)
    rho = 8
    inp_nr = dict(inp, Wr=None)  # no router
    out = orc.forward(inp_nr, w.k, opts=orc.options(fixed_stride=rho))
    X = to64(inp["X"])
    sel = list(range(0, w.seq_len, rho))
    Y = np.zeros_like(X)
    T = w.seq_len
    for b in range(w.batch):
        Xs = X[b, sel]
        mask = np.array(sel)[:, None] >= np.array(sel)[None, :]
        for h in range(w.heads):
            A = sdpa(Xs @ to64(inp["Wq"])[h], Xs @ to64(inp["Wk"])[h], Xs @ to64(inp["Wv"])[h], mask)
            Y[b, sel] += A @ to64(inp["Wo"])[h]
        full = np.tril(np.ones((T, T), dtype=bool))
        A = sdpa(X[b] @ to64(inp["Wq_d"])[0], X[b] @ to64(inp["Wk_d"])[0], X[b] @ to64(inp["Wv_d"])[0], full)
        Y[b] += A @ to64(inp["Wo_d"])[0]
    np.testing.assert_allclose(out["Y"], Y, rtol=1e-11, atol=1e-12)
    assert (out["I"] == np.array(sel)).all() and (out["r"] == 1.0).all()


def test_fixed_stride_rejects_out_of_range(orc):
    w = wl.small(batch=1, seq_len=30, d_model=16, heads=1, d_head=8, k=5, dtype="f32")
    inp = dict(wl.make_inputs(w), Wr=None)
    with pytest.raises(RuntimeError):
        orc.forward(inp, 5, opts=orc.options(fixed_stride=8))  # 4 * 8 = 32 > T - 1


# --------------------------------------------------------------------------
# Rotary encoding (Section 2.2): the primitive
# --------------------------------------------------------------------------

def test_rope_one_pair_is_a_plane_rotation(orc):
    # dh = 4: one rotated pair (dims 0, 1) with theta_0 = 1, dims 2, 3 untouched.
    v = np.array([[1.0, 0.0, 3.0, -2.0], [0.3, -0.7, 1.0, 5.0]])
    p = np.array([2, 11])
    got = orc.rope(v, p)
    for i in range(2):
        c, s = math.cos(p[i]), math.sin(p[i])
        x, y = v[i, 0], v[i, 1]
        np.testing.assert_allclose(got[i, :2], [x * c - y * s, x * s + y * c], rtol=1e-15, atol=1e-15)
        assert (got[i, 2:] == v[i, 2:]).all()


def test_rope_invariants(orc):
    rng = np.random.default_rng(8)
    n, dh = 200, 64
    q, k = rng.standard_normal((n, dh)), rng.standard_normal((n, dh))
    p1, p2 = rng.integers(0, 8192, n), rng.integers(0, 8192, n)
    rq = orc.rope(q, p1)
    # norms kept, second half untouched, the inverse undoes it
    np.testing.assert_allclose(np.linalg.norm(rq, axis=1), np.linalg.norm(q, axis=1), rtol=1e-13)
    assert (rq[:, dh // 2:] == q[:, dh // 2:]).all()
    np.testing.assert_allclose(orc.rope(rq, p1, sign=-1), q, rtol=1e-11, atol=1e-11)
    # scores depend only on the offset: <R(p1) q, R(p2) k> = <q, R(p2 - p1) k>
    lhs = np.einsum("ne,ne->n", rq, orc.rope(k, p2))
    d = p2 - p1
    kk = np.where(d[:, None] >= 0, orc.rope(k, np.abs(d)), orc.rope(k, np.abs(d), sign=-1))
    rhs = np.einsum("ne,ne->n", q, kk)
    np.testing.assert_allclose(lhs, rhs, rtol=1e-9, atol=1e-9)
    # the pair frequencies fall geometrically: pair j turns by base^(-2j/(dh/2)) per position
    e = np.zeros((1, dh))
    e[0, 2 * 3] = 1.0  # pair j = 3
    got = orc.rope(e, np.array([1]))[0]
    ang = 10000.0 ** (-2 * 3 / (dh // 2))
    np.testing.assert_allclose(got[6:8], [math.cos(ang), math.sin(ang)], rtol=1e-14)


# --------------------------------------------------------------------------
# Rotary encoding in the layer: positions are the ORIGINAL indices I
# --------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_rope_layer_matches_dense_masked_attention(orc, dtype):
    # Every head rotates q, k of ALL T tokens at positions 0..T-1 and attends over
    # a T x T mask that allows (t, u) only when both are selected and t >= u; the
    # rows of unselected tokens are dropped.  MoSA with rope must equal it.
    w = wl.small(batch=2, seq_len=40, d_model=16, heads=2, d_head=8, k=9, dense_heads=1, dtype=dtype)
    inp = wl.make_inputs(w)
    out = orc.forward(inp, w.k, opts=orc.options(rope=True, rope_base=100.0))
    X = to64(inp["X"])
    T = w.seq_len
    pos = np.arange(T)
    tril = np.tril(np.ones((T, T), dtype=bool))
    Y = np.zeros_like(X)
    for b in range(w.batch):
        for h in range(w.heads):
            key = exact_keys(X[b], to64(inp["Wr"])[h])
            sel = sorted(sorted(range(T), key=lambda t: (-key[t], t))[:w.k])
            r = np.array([1.0 / (1.0 + math.exp(-key[t])) for t in sel])
            q = orc.rope(X[b] @ to64(inp["Wq"])[h], pos, base=100.0)
            kk = orc.rope(X[b] @ to64(inp["Wk"])[h], pos, base=100.0)
            selm = np.zeros(T, dtype=bool)
            selm[sel] = True
            mask = selm[:, None] & selm[None, :] & tril
            mask[~selm, 0] = True
            A = sdpa(q, kk, X[b] @ to64(inp["Wv"])[h], mask)
            Y[b, sel] += (r[:, None] * A[sel]) @ to64(inp["Wo"])[h]
        q = orc.rope(X[b] @ to64(inp["Wq_d"])[0], pos, base=100.0)
        kk = orc.rope(X[b] @ to64(inp["Wk_d"])[0], pos, base=100.0)
        Y[b] += sdpa(q, kk, X[b] @ to64(inp["Wv_d"])[0], tril) @ to64(inp["Wo_d"])[0]
    np.testing.assert_allclose(out["Y"], Y, rtol=1e-11, atol=1e-12)


# --------------------------------------------------------------------------
# Local dense heads (Section 3.4)
# --------------------------------------------------------------------------

def _dense_only(w_kw):
    w = wl.small(**w_kw)
    return w, wl.make_inputs(w)


def test_window_one_is_value_projection(orc):
    # window 1: every query sees only itself, A = V, Y = X W^V W^O per head.
    w, inp = _dense_only(dict(batch=2, seq_len=24, d_model=16, heads=0, dense_heads=2, d_head=8, k=0,
                              dtype="f32"))
    out = orc.forward(inp, 0, opts=orc.options(window=1))
    X = to64(inp["X"])
    ref = sum(X @ to64(inp["Wv_d"])[h] @ to64(inp["Wo_d"])[h] for h in range(2))
    np.testing.assert_allclose(out["Y"], ref, rtol=1e-12, atol=1e-13)


def test_window_at_least_T_is_full_causal(orc):
    w, inp = _dense_only(dict(batch=1, seq_len=30, d_model=16, heads=2, dense_heads=2, d_head=8, k=6))
    a = orc.forward(inp, w.k)["Y"]
    b = orc.forward(inp, w.k, opts=orc.options(window=30))["Y"]
    assert (a == b).all()


@pytest.mark.parametrize("window", [3, 7])
def test_window_matches_banded_sdpa(orc, window):
    w, inp = _dense_only(dict(batch=2, seq_len=33, d_model=16, heads=0, dense_heads=2, d_head=8, k=0))
    out = orc.forward(inp, 0, opts=orc.options(window=window))
    X = to64(inp["X"])
    T = w.seq_len
    t = np.arange(T)
    band = (t[:, None] >= t[None, :]) & (t[:, None] - t[None, :] < window)
    Y = np.zeros_like(X)
    for b in range(w.batch):
        for h in range(2):
            A = sdpa(X[b] @ to64(inp["Wq_d"])[h], X[b] @ to64(inp["Wk_d"])[h], X[b] @ to64(inp["Wv_d"])[h], band)
            Y[b] += A @ to64(inp["Wo_d"])[h]
    np.testing.assert_allclose(out["Y"], Y, rtol=1e-11, atol=1e-12)


# --------------------------------------------------------------------------
# Backward of every variant: central finite differences
# --------------------------------------------------------------------------

def _f64_inputs(seed, B=2, T=14, d=8, H=2, dh=8, Hd=1):
    rng = np.random.default_rng(seed)
    s = 1 / np.sqrt(d)
    inp = {"X": rng.standard_normal((B, T, d)), "Wr": rng.standard_normal((H, d)) * s,
           "Wq": rng.standard_normal((H, d, dh)) * s, "Wk": rng.standard_normal((H, d, dh)) * s,
           "Wv": rng.standard_normal((H, d, dh)) * s, "Wo": rng.standard_normal((H, dh, d)) * s,
           "Wq_d": rng.standard_normal((Hd, d, dh)) * s, "Wk_d": rng.standard_normal((Hd, d, dh)) * s,
           "Wv_d": rng.standard_normal((Hd, d, dh)) * s, "Wo_d": rng.standard_normal((Hd, dh, d)) * s}
    return inp, rng.standard_normal((B, T, d))


@pytest.mark.parametrize("kw", [dict(first_token=True), dict(fixed_stride=3), dict(rope=True, rope_base=50.0),
                                dict(window=4), dict(first_token=True, rope=True, window=2)])
def test_variant_finite_differences(orc, kw):
    k = 5
    inp, dY = _f64_inputs(seed=21)
    if kw.get("fixed_stride"):
        inp["Wr"] = None
    opts = orc.options(**kw)
    g = orc.backward(inp, dY, k, opts=opts)
    base = orc.forward(inp, k, opts=opts)
    rng = np.random.default_rng(22)
    eps = 1e-5
    for name in [n for n in inp if inp[n] is not None]:
        gname = "d" + name
        for _ in range(2):
            U = rng.standard_normal(inp[name].shape)
            vals = []
            for sgn in (1, -1):
                p = dict(inp)
                p[name] = inp[name] + sgn * eps * U
                o = orc.forward(p, k, opts=opts)
                assert (o["I"] == base["I"]).all(), "selection moved under the perturbation"
                vals.append(float((o["Y"] * dY).sum()))
            fd = (vals[0] - vals[1]) / (2 * eps)
            an = float((g[gname] * U).sum())
            assert abs(fd - an) <= 1e-7 * max(1.0, abs(an)), (name, fd, an)
    if kw.get("fixed_stride"):
        assert (g["dWr"] == 0).all()
