"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

Each check reaches the oracle's result by a different route than the oracle:
exact rational arithmetic, a library routine (Python's ``sorted``,
``math.fsum``, PyTorch's scaled-dot-product attention and autograd), a
special case with a closed form, an invariant, or finite differences.
"""
import math
import random
from fractions import Fraction

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import workloads as wl

pytestmark = pytest.mark.filterwarnings("ignore::UserWarning")


def to64(a):
    if a is None:
        return None
    if a.dtype == np.float64:
        return a
    return wl.as_f32(a).astype(np.float64)


def exact_round(values):
    """Correctly rounded sum via exact rationals (Python's float(Fraction) rounds correctly)."""
    return float(sum((Fraction(v) for v in values), Fraction(0)))


# --------------------------------------------------------------------------
# Exact summation and router keys (Section 2.2: r = sigma(X W^r))
# --------------------------------------------------------------------------

def test_fsum_matches_exact_rationals(orc):
    rng = random.Random(5)
    cases = [
        [1.0, 1e100, 1.0, -1e100],
        [1e-16, 1.0, 1e16],                # needs the half-even fix across components
        [2.0 ** 53, 1.0, 2.0 ** -60],      # tie broken by a tiny third component
        [2.0 ** 53, 1.0, -(2.0 ** -60)],
        [2.0 ** 53, -1.0, 2.0 ** -60],
        [0.1] * 10,
        [-0.0],
        [],
    ]
    for _ in range(300):
        n = rng.randint(1, 60)
        cases.append([rng.choice([-1, 1]) * rng.random() * 2.0 ** rng.randint(-80, 80) for _ in range(n)])
    for _ in range(100):  # heavy cancellation
        base = [rng.uniform(-1, 1) * 2.0 ** rng.randint(0, 60) for _ in range(20)]
        cases.append(base + [-b for b in base[:-1]] + [rng.uniform(-1, 1) * 2.0 ** -50])
    for c in cases:
        got = orc.fsum(np.array(c, dtype=np.float64))
        assert got == exact_round(c), c
        assert got == math.fsum(c), c


def test_router_keys_exact_bf16_and_f32(orc):
    rng = np.random.default_rng(1)
    for dtype in ("bf16", "f32"):
        X = rng.standard_normal((2, 7, 33)).astype(np.float32) * np.float32(3.0)
        W = rng.standard_normal((3, 33)).astype(np.float32) / np.float32(5.0)
        if dtype == "bf16":
            X, W = wl.f32_to_bf16_bits(X), wl.f32_to_bf16_bits(W)
        keys = orc.router_keys(X, W)
        Xf, Wf = to64(X), to64(W)
        for b in range(2):
            for h in range(3):
                for t in range(7):
                    prods = [Fraction(float(x)) * Fraction(float(w)) for x, w in zip(Xf[b, t], Wf[h])]
                    assert keys[b, h, t] == float(sum(prods, Fraction(0)))


def test_router_key_cancellation_is_exact(orc):
    # 1 + 2^-60 - 1 is 0 in naive double arithmetic; the exact value is 2^-60.
    X = wl.f32_to_bf16_bits(np.array([[[1.0, 2.0 ** -60, -1.0]]], dtype=np.float32))
    W = wl.f32_to_bf16_bits(np.array([[1.0, 1.0, 1.0]], dtype=np.float32))
    assert orc.router_keys(X, W)[0, 0, 0] == 2.0 ** -60


# --------------------------------------------------------------------------
# Expert-choice TopK (Section 2.2; ties -> lower index; I ascending)
# --------------------------------------------------------------------------

def brute_topk(key, k):
    order = sorted(range(len(key)), key=lambda t: (-key[t], t))
    return sorted(order[:k])


def test_select_matches_sorted_with_ties(orc):
    rng = np.random.default_rng(2)
    for T, k in [(1, 1), (5, 5), (17, 1), (64, 7), (300, 299), (257, 128)]:
        keys = rng.integers(-4, 5, size=(2, 3, T)).astype(np.float64) * 0.25  # many ties
        I = orc.select(keys, k)
        for b in range(2):
            for h in range(3):
                assert list(I[b, h]) == brute_topk(list(keys[b, h]), k)


def test_select_signed_zero_ties(orc):
    keys = np.array([[[0.0, -0.0, 0.0, -0.0, -1.0, 1.0]]])
    assert list(orc.select(keys, 3)[0, 0]) == [0, 1, 5]


def test_select_all_ties_takes_prefix(orc):
    w = wl.small(k=9, seq_len=40)
    inp = wl.make_inputs(w)
    inp["Wr"][:] = 0
    out = orc.forward(inp, w.k)
    assert (out["I"] == np.arange(w.k)).all()
    assert (out["r"] == 0.5).all()


def test_duplicate_rows_lower_index_wins(orc):
    w = wl.small(seq_len=32, k=4, heads=2)
    inp = wl.make_inputs(w)
    keys = orc.router_keys(inp["X"], inp["Wr"])
    for b in range(w.batch):
        top = int(np.argmax(keys[b, 0]))
        inp["X"][b, 31] = inp["X"][b, top]
        inp["X"][b, 0] = inp["X"][b, top]
    keys2 = orc.router_keys(inp["X"], inp["Wr"])
    I = orc.select(keys2, 2)
    for b in range(w.batch):
        assert keys2[b, 0, 0] == keys2[b, 0, 31]
        assert list(I[b, 0]) == brute_topk(list(keys2[b, 0]), 2)
        assert 0 in I[b, 0] and (31 not in I[b, 0] or top == 31 or 31 in brute_topk(list(keys2[b, 0]), 2))


# --------------------------------------------------------------------------
# Independent re-expressions of the layer
# --------------------------------------------------------------------------

def sdpa_head(Xb, Wq, Wk, Wv, rows, cols, causal):
    """Attention of query tokens ``rows`` over key tokens ``cols`` (Eq. 1) through
    PyTorch's scaled_dot_product_attention in float64; mask by original index."""
    X = torch.from_numpy(Xb)
    q = (X[rows] @ torch.from_numpy(Wq))[None, None]
    k = (X[cols] @ torch.from_numpy(Wk))[None, None]
    v = (X[cols] @ torch.from_numpy(Wv))[None, None]
    if causal:
        mask = torch.tensor(rows)[:, None] >= torch.tensor(cols)[None, :]
    else:
        mask = torch.ones(len(rows), len(cols), dtype=torch.bool)
    return F.scaled_dot_product_attention(q, k, v, attn_mask=mask[None, None])[0, 0].numpy()


def bruteforce_layer(inp, k, causal=True):
    """P1: every head computes Q, K, V for ALL T tokens and attends over a T x T
    mask that allows (t, u) only when both are selected (and t >= u if causal);
    unselected rows are dropped.  Selection by sorted() on keys summed with
    exact rationals.  Dense heads: all tokens, r = 1."""
    X = to64(inp["X"])
    B, T, d = X.shape
    Y = np.zeros_like(X)
    H = inp["Wr"].shape[0] if inp.get("Wr") is not None else 0
    for b in range(B):
        for h in range(H):
            Wr = to64(inp["Wr"])[h]
            key = [float(sum((Fraction(float(x)) * Fraction(float(w)) for x, w in zip(X[b, t], Wr)),
                             Fraction(0))) for t in range(T)]
            sel = brute_topk(key, k)
            r = np.array([1.0 / (1.0 + math.exp(-key[t])) for t in sel])
            allt = list(range(T))
            Xb = X[b]
            q = torch.from_numpy(Xb @ to64(inp["Wq"])[h])[None, None]
            kk = torch.from_numpy(Xb @ to64(inp["Wk"])[h])[None, None]
            v = torch.from_numpy(Xb @ to64(inp["Wv"])[h])[None, None]
            selmask = torch.zeros(T, dtype=torch.bool)
            selmask[sel] = True
            mask = selmask[:, None] & selmask[None, :]
            if causal:
                mask &= torch.tensor(allt)[:, None] >= torch.tensor(allt)[None, :]
            mask[~selmask, 0] = True  # keep unselected rows finite; they are dropped below
            A = F.scaled_dot_product_attention(q, kk, v, attn_mask=mask[None, None])[0, 0].numpy()
            Y[b, sel] += (r[:, None] * A[sel]) @ to64(inp["Wo"])[h]
        if inp.get("Wq_d") is not None:
            for h in range(inp["Wq_d"].shape[0]):
                A = sdpa_head(X[b], to64(inp["Wq_d"])[h], to64(inp["Wk_d"])[h], to64(inp["Wv_d"])[h],
                              list(range(T)), list(range(T)), causal)
                Y[b] += A @ to64(inp["Wo_d"])[h]
    return Y


@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_P1_bruteforce_masked_dense_attention(orc, causal, dtype):
    w = wl.small(batch=2, seq_len=48, d_model=24, heads=3, d_head=8, k=11, dense_heads=2,
                 causal=causal, dtype=dtype)
    inp = wl.make_inputs(w)
    got = orc.forward(inp, w.k, causal=causal)["Y"]
    ref = bruteforce_layer(inp, w.k, causal=causal)
    np.testing.assert_allclose(got, ref, rtol=1e-11, atol=1e-12)


def test_P2_k_equals_T_is_half_causal_mha(orc):
    # W^r = 0 => every r = sigmoid(0) = 1/2 and k = T selects all tokens:
    # the layer is exactly half of standard causal multi-head attention (Eq. 2).
    w = wl.small(batch=2, seq_len=30, d_model=16, heads=3, d_head=8, k=30)
    inp = wl.make_inputs(w)
    inp["Wr"][:] = 0
    got = orc.forward(inp, w.k)["Y"]
    X = to64(inp["X"])
    ref = np.zeros_like(X)
    T = w.seq_len
    for b in range(w.batch):
        for h in range(w.heads):
            A = sdpa_head(X[b], to64(inp["Wq"])[h], to64(inp["Wk"])[h], to64(inp["Wv"])[h],
                          list(range(T)), list(range(T)), True)
            ref[b] += 0.5 * A @ to64(inp["Wo"])[h]
    np.testing.assert_allclose(got, ref, rtol=1e-11, atol=1e-12)


def test_P2_k_equals_T_with_router_scaling(orc):
    w = wl.small(batch=1, seq_len=20, d_model=16, heads=2, d_head=8, k=20, dtype="f32")
    inp = wl.make_inputs(w)
    got = orc.forward(inp, w.k)["Y"]
    X = to64(inp["X"])
    ref = np.zeros_like(X)
    for h in range(w.heads):
        s = X[0] @ to64(inp["Wr"])[h]
        r = 1.0 / (1.0 + np.exp(-s))
        A = sdpa_head(X[0], to64(inp["Wq"])[h], to64(inp["Wk"])[h], to64(inp["Wv"])[h],
                      list(range(20)), list(range(20)), True)
        ref[0] += (r[:, None] * A) @ to64(inp["Wo"])[h]
    np.testing.assert_allclose(got, ref, rtol=1e-11, atol=1e-12)


def test_P3_all_ties_select_prefix_and_attend_causally(orc):
    w = wl.small(batch=2, seq_len=40, d_model=16, heads=2, d_head=8, k=13)
    inp = wl.make_inputs(w)
    inp["Wr"][:] = 0
    got = orc.forward(inp, w.k)["Y"]
    X = to64(inp["X"])
    ref = np.zeros_like(X)
    pre = list(range(w.k))
    for b in range(w.batch):
        for h in range(w.heads):
            A = sdpa_head(X[b], to64(inp["Wq"])[h], to64(inp["Wk"])[h], to64(inp["Wv"])[h], pre, pre, True)
            ref[b, pre] += 0.5 * A @ to64(inp["Wo"])[h]
    np.testing.assert_allclose(got, ref, rtol=1e-11, atol=1e-12)
    assert (got[:, w.k:] == 0).all()


def test_P4_fixed_sparse_attention_special_case(orc):
    # Section 3.1: fixed sparse attention is MoSA with I = [0, rho, 2 rho, ...] and r = 1.
    rng = np.random.default_rng(4)
    T, d, dh, rho = 64, 16, 8, 8
    Xb = rng.standard_normal((T, d))
    Wq, Wk, Wv = (rng.standard_normal((d, dh)) / 4 for _ in range(3))
    Wo = rng.standard_normal((dh, d)) / 4
    I = np.arange(0, T, rho)
    got = orc.head_attend(Xb, Wq, Wk, Wv, Wo, I, None, causal=True)
    A = sdpa_head(Xb, Wq, Wk, Wv, list(I), list(I), True)
    ref = np.zeros((T, d))
    ref[I] = A @ Wo
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-13)


def test_P5_index_order_invariance(orc):
    # The mask M_ij = 0 iff I_i >= I_j depends on the indices, not on slot order.
    rng = np.random.default_rng(5)
    T, d, dh = 50, 12, 4
    Xb = rng.standard_normal((T, d))
    Wq, Wk, Wv = (rng.standard_normal((d, dh)) / 3 for _ in range(3))
    Wo = rng.standard_normal((dh, d)) / 3
    I = np.sort(rng.choice(T, 17, replace=False))
    r = rng.uniform(0.1, 0.9, 17)
    base = orc.head_attend(Xb, Wq, Wk, Wv, Wo, I, r)
    for _ in range(3):
        p = rng.permutation(17)
        np.testing.assert_allclose(orc.head_attend(Xb, Wq, Wk, Wv, Wo, I[p], r[p]), base,
                                   rtol=1e-13, atol=1e-14)


def _slice_heads(inp, hs):
    out = dict(inp)
    for n in ("Wr", "Wq", "Wk", "Wv", "Wo"):
        out[n] = np.ascontiguousarray(inp[n][hs])
    for n in ("Wq_d", "Wk_d", "Wv_d", "Wo_d"):
        out[n] = None
    return out


def test_P6_layer_is_sum_of_heads(orc):
    w = wl.small(batch=2, seq_len=40, d_model=16, heads=4, d_head=8, k=9)
    inp = wl.make_inputs(w)
    full = orc.forward(inp, w.k)["Y"]
    parts = sum(orc.forward(_slice_heads(inp, [h]), w.k)["Y"] for h in range(w.heads))
    np.testing.assert_allclose(full, parts, rtol=1e-13, atol=1e-14)


def test_P7_unselected_rows_are_exactly_zero(orc):
    w = wl.small(batch=2, seq_len=64, d_model=16, heads=3, d_head=8, k=5)
    out = orc.forward(wl.make_inputs(w), w.k)
    for b in range(w.batch):
        picked = set(out["I"][b].ravel().tolist())
        for t in range(w.seq_len):
            if t not in picked:
                assert (out["Y"][b, t] == 0).all()
            else:
                assert np.abs(out["Y"][b, t]).max() > 0


def test_P8_first_selected_token_attends_only_itself(orc):
    w = wl.small(batch=2, seq_len=40, d_model=16, heads=3, d_head=8, k=7)
    out = orc.forward(wl.make_inputs(w), w.k, intermediates=True)
    assert (out["A"][:, :, 0, :] == out["V"][:, :, 0, :]).all()


def test_thread_count_does_not_change_results(orc):
    w = wl.small(batch=3, seq_len=40, d_model=16, heads=4, d_head=8, k=9, dense_heads=1)
    inp = wl.make_inputs(w)
    n0 = orc.max_threads()
    try:
        orc.set_threads(1)
        a = orc.forward(inp, w.k)["Y"]
        ga = orc.backward(inp, inp["dY"], w.k)
        orc.set_threads(4)
        b = orc.forward(inp, w.k)["Y"]
        gb = orc.backward(inp, inp["dY"], w.k)
    finally:
        orc.set_threads(n0)
    assert (a == b).all()
    for n in ga:
        assert (ga[n] == gb[n]).all(), n


# --------------------------------------------------------------------------
# Backward (I held fixed): finite differences and autograd re-expression
# --------------------------------------------------------------------------

def _f64_inputs(seed=7, B=2, T=12, d=8, H=2, dh=4, Hd=1):
    rng = np.random.default_rng(seed)
    inp = {"X": rng.standard_normal((B, T, d)),
           "Wr": rng.standard_normal((H, d)) / np.sqrt(d),
           "Wq": rng.standard_normal((H, d, dh)) / np.sqrt(d),
           "Wk": rng.standard_normal((H, d, dh)) / np.sqrt(d),
           "Wv": rng.standard_normal((H, d, dh)) / np.sqrt(d),
           "Wo": rng.standard_normal((H, dh, d)) / np.sqrt(d)}
    if Hd:
        inp.update(Wq_d=rng.standard_normal((Hd, d, dh)) / np.sqrt(d),
                   Wk_d=rng.standard_normal((Hd, d, dh)) / np.sqrt(d),
                   Wv_d=rng.standard_normal((Hd, d, dh)) / np.sqrt(d),
                   Wo_d=rng.standard_normal((Hd, dh, d)) / np.sqrt(d))
    else:
        inp.update(Wq_d=None, Wk_d=None, Wv_d=None, Wo_d=None)
    dY = rng.standard_normal((B, T, d))
    return inp, dY


@pytest.mark.parametrize("causal", [True, False])
def test_P9_finite_differences(orc, causal):
    k = 5
    inp, dY = _f64_inputs()
    g = orc.backward(inp, dY, k, causal=causal)
    base = orc.forward(inp, k, causal=causal)
    rng = np.random.default_rng(9)
    eps = 1e-5
    grad_of = {"X": "dX", "Wr": "dWr", "Wq": "dWq", "Wk": "dWk", "Wv": "dWv", "Wo": "dWo",
               "Wq_d": "dWq_d", "Wk_d": "dWk_d", "Wv_d": "dWv_d", "Wo_d": "dWo_d"}
    for name, gname in grad_of.items():
        for _ in range(3):
            U = rng.standard_normal(inp[name].shape)
            vals = []
            for sgn in (1, -1):
                p = dict(inp)
                p[name] = inp[name] + sgn * eps * U
                out = orc.forward(p, k, causal=causal)
                assert (out["I"] == base["I"]).all(), "selection moved under the perturbation"
                vals.append(float((out["Y"] * dY).sum()))
            fd = (vals[0] - vals[1]) / (2 * eps)
            an = float((g[gname] * U).sum())
            assert abs(fd - an) <= 1e-7 * max(1.0, abs(an)), (name, fd, an)


def torch_layer(t, I, causal=True):
    """The layer written with einsum / gather / scatter (the operations the paper
    names for its own implementation, Section 2.2), differentiated by autograd."""
    X = t["X"]
    B, T, d = X.shape
    Y = torch.zeros_like(X)
    if "Wr" in t:
        H, k = I.shape[1], I.shape[2]
        s = torch.einsum("btd,hd->bht", X, t["Wr"])
        idx = torch.from_numpy(I.astype(np.int64))
        r = torch.sigmoid(torch.gather(s, 2, idx))                       # [B,H,k]
        Xs = torch.gather(X[:, None].expand(B, H, T, d), 2, idx[..., None].expand(B, H, k, d))
        Q = torch.einsum("bhkd,hde->bhke", Xs, t["Wq"])
        K = torch.einsum("bhkd,hde->bhke", Xs, t["Wk"])
        V = torch.einsum("bhkd,hde->bhke", Xs, t["Wv"])
        S = torch.einsum("bhie,bhje->bhij", Q, K) / math.sqrt(Q.shape[-1])
        if causal:
            allowed = idx[..., :, None] >= idx[..., None, :]
            S = S.masked_fill(~allowed, float("-inf"))
        A = torch.softmax(S, dim=-1) @ V
        Xo = torch.einsum("bhke,hed->bhkd", r[..., None] * A, t["Wo"])
        Y = Y.scatter_add(1, idx.reshape(B, H * k)[..., None].expand(B, H * k, d), Xo.reshape(B, H * k, d))
    if "Wq_d" in t:
        Q = torch.einsum("btd,hde->bhte", X, t["Wq_d"])
        K = torch.einsum("btd,hde->bhte", X, t["Wk_d"])
        V = torch.einsum("btd,hde->bhte", X, t["Wv_d"])
        S = torch.einsum("bhie,bhje->bhij", Q, K) / math.sqrt(Q.shape[-1])
        if causal:
            S = S.masked_fill(~torch.ones(T, T, dtype=torch.bool).tril(), float("-inf"))
        A = torch.softmax(S, dim=-1) @ V
        Y = Y + torch.einsum("bhte,hed->btd", A, t["Wo_d"])
    return Y


@pytest.mark.parametrize("causal", [True, False])
def test_P10_autograd_reexpression(orc, causal):
    k = 6
    inp, dY = _f64_inputs(seed=10, B=2, T=16, d=12, H=3, dh=4, Hd=2)
    out = orc.forward(inp, k, causal=causal)
    g = orc.backward(inp, dY, k, causal=causal)
    t = {n: torch.tensor(v, requires_grad=True) for n, v in inp.items() if v is not None}
    Y = torch_layer(t, out["I"], causal)
    np.testing.assert_allclose(Y.detach().numpy(), out["Y"], rtol=1e-12, atol=1e-13)
    Y.backward(torch.from_numpy(dY))
    for n, v in t.items():
        np.testing.assert_allclose(g["d" + n], v.grad.numpy(), rtol=1e-10, atol=1e-12, err_msg=n)


def test_P10_autograd_bf16_workload(orc):
    w = wl.small(batch=2, seq_len=64, d_model=32, heads=4, d_head=16, k=10, dense_heads=1)
    inp = wl.make_inputs(w)
    out = orc.forward(inp, w.k)
    g = orc.backward(inp, inp["dY"], w.k)
    t = {n: torch.tensor(to64(v), requires_grad=True) for n, v in inp.items()
         if v is not None and n != "dY"}
    Y = torch_layer(t, out["I"])
    np.testing.assert_allclose(Y.detach().numpy(), out["Y"], rtol=1e-11, atol=1e-12)
    Y.backward(torch.from_numpy(to64(inp["dY"])))
    for n, v in t.items():
        np.testing.assert_allclose(g["d" + n], v.grad.numpy(), rtol=1e-9, atol=1e-11, err_msg=n)
