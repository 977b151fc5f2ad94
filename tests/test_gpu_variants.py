"""GPU parity of the layer variants through the C ABI against the CPU oracle:
forced first token (Section 3.2), fixed sparse attention (Section 3.1),
rotary encoding at the original positions (Section 2.2) and local
(sliding-window) dense heads (Section 3.4), forward and backward.  Bars as
everywhere: indices bit-exact; max |gpu - oracle| / max |oracle| <= 2e-2
(bf16) or 1e-5 (fp32) per tensor."""
import numpy as np
import pytest
import torch

import workloads as wl
from gpu_util import TOL, device_inputs, rel_err, run_forward, shape_of, to_f64
from paper_2505_00315_amd import mosa

pytestmark = pytest.mark.gpu


def _opts(orc, w):
    return orc.options(**w.variants())


def check_forward(orc, w, inp=None, drop_router=False):
    print(f"\n[case] {w}", flush=True)
    inp = wl.make_inputs(w) if inp is None else inp
    gin = dict(inp, Wr=None) if drop_router else inp
    out = run_forward(w, gin)
    ref = orc.forward(inp, w.k, causal=w.causal, opts=_opts(orc, w))
    if w.heads:
        mism = np.argwhere(out["I"] != ref["I"])
        assert mism.size == 0, f"index mismatch at {mism[:5].tolist()} (of {len(mism)})"
        assert rel_err(out["r"], ref["r"]) <= 1e-6
    e = rel_err(to_f64(out["Y"]), ref["Y"])
    print(f"[case] Y rel err {e:.3e}", flush=True)
    assert e <= TOL[w.dtype], e
    return out, ref


def check_backward(orc, w, drop_router=False, zero=()):
    """``zero``: gradients that are exactly 0 in exact arithmetic (the oracle
    gives 0); they are held to the tolerance relative to the largest of the
    other gradients instead."""
    print(f"\n[case] bwd {w}", flush=True)
    inp = wl.make_inputs(w, with_grad=True)
    shape = shape_of(w)
    dev = device_inputs(dict(inp, Wr=None) if drop_router else inp)
    weights = {n: dev.get(n) for n in mosa.WEIGHT_NAMES}
    Y, saved, scratch = mosa.forward(shape, dev["X"], weights)
    grads = {"d" + n: torch.empty_like(dev[n]) for n in mosa.WEIGHT_NAMES if dev.get(n) is not None}
    dX = mosa.backward(shape, dev["X"], weights, dev["dY"], saved, grads, scratch=scratch)
    torch.cuda.synchronize()
    ref = orc.backward(inp, inp["dY"], w.k, causal=w.causal, opts=_opts(orc, w))
    errs = {"dX": rel_err(to_f64(dX), ref["dX"])}
    for n, t in grads.items():
        if n in ref and n not in zero:  # no MoSA heads: no MoSA weight gradients
            errs[n] = rel_err(to_f64(t), ref[n])
    scale = max(float(np.abs(ref[n]).max()) for n in errs if n != "dX")
    for n in zero:
        assert (ref[n] == 0).all(), n
        errs[n] = float(np.abs(to_f64(grads[n])).max()) / scale
    print("[case] rel err " + " ".join(f"{n}={e:.2e}" for n, e in errs.items()), flush=True)
    bad = {n: e for n, e in errs.items() if not e <= TOL[w.dtype]}
    assert not bad, bad
    return grads


# k = 20 (separate projection and attention), 64 (one fused launch), 50 with a
# 64-wide head; fp32; dense heads beside the MoSA heads
CASES = [
    dict(),
    dict(dtype="f32"),
    dict(seq_len=256, k=64, d_head=64, d_model=128),
    dict(seq_len=200, k=50, d_head=64, d_model=128, dense_heads=1),
    dict(dense_heads=2, dtype="f32", seq_len=130),
    dict(causal=False),
]


@pytest.mark.parametrize("kw", CASES)
def test_first_token(orc, kw):
    w = wl.small(first_token=True, **kw)
    out, _ = check_forward(orc, w)
    assert (out["I"][..., 0] == 0).all()
    check_backward(orc, w)


def test_first_token_k1_and_k_equals_T(orc):
    check_forward(orc, wl.small(first_token=True, k=1))
    check_forward(orc, wl.small(first_token=True, seq_len=70, k=70))


@pytest.mark.parametrize("kw", CASES)
def test_rope(orc, kw):
    w = wl.small(rope=True, **kw)
    check_forward(orc, w)
    check_backward(orc, w)


def test_rope_small_base_and_first_token(orc):
    # a small base turns every pair quickly: a wrong position shows at once
    w = wl.small(rope=True, rope_base=30.0, first_token=True, seq_len=256, k=64, d_head=64, d_model=128,
                 dense_heads=1)
    check_forward(orc, w)
    check_backward(orc, w)


def test_rope_stage_intermediates(orc):
    """The saved Q and K are the rotated ones (positions I), V is not rotated."""
    w = wl.small(rope=True, rope_base=50.0, batch=2, seq_len=200, heads=3, k=64, d_head=64, d_model=128)
    inp = wl.make_inputs(w)
    out = run_forward(w, inp)
    ref = orc.forward(inp, w.k, intermediates=True, opts=_opts(orc, w))
    for n in ("Q", "K", "V"):
        e = rel_err(to_f64(mosa.saved_view(out["shape"], out["saved"], n)), ref[n])
        assert e <= TOL[w.dtype], (n, e)


@pytest.mark.parametrize("kw", [
    dict(seq_len=96, k=12, fixed_stride=8),
    dict(seq_len=100, k=13, fixed_stride=8, dtype="f32"),   # ragged: last token 96
    dict(seq_len=256, k=64, fixed_stride=4, d_head=64, d_model=128, dense_heads=1),
    dict(seq_len=128, k=16, fixed_stride=8, rope=True),
])
@pytest.mark.parametrize("drop_router", [False, True])
def test_fixed_stride(orc, kw, drop_router):
    w = wl.small(**kw)
    out, _ = check_forward(orc, w, drop_router=drop_router)
    assert (out["I"] == np.arange(w.k) * w.fixed_stride).all() and (out["r"] == 1.0).all()
    grads = check_backward(orc, w, drop_router=drop_router)
    if not drop_router:
        assert (to_f64(grads["dWr"]) == 0).all()


def test_workload_rope_first_full(orc):
    w = wl.WORKLOADS["fwd_d512_rope_first"]
    check_forward(orc, w, wl.make_inputs(w, with_grad=False))


def test_workload_fixed_full(orc):
    w = wl.WORKLOADS["fixed_d512"]
    check_forward(orc, w, wl.make_inputs(w, with_grad=False))


@pytest.mark.parametrize("kw", [
    dict(seq_len=96, window=7, dense_heads=2),                        # MoSA + local heads
    dict(seq_len=24, window=5, dense_heads=1, heads=0, k=0),          # n <= 32
    dict(seq_len=100, window=1, dense_heads=1, heads=0, k=0),         # A = V
    dict(seq_len=200, window=64, dense_heads=2, d_head=64, d_model=128),
    dict(seq_len=300, window=100, dense_heads=1, heads=2, k=30),      # window not a tile multiple
    dict(seq_len=130, window=17, dense_heads=2, dtype="f32"),
    dict(seq_len=64, window=64, dense_heads=1),                       # window = T: full causal
    dict(seq_len=96, window=9, dense_heads=1, rope=True, first_token=True),
])
def test_local_window(orc, kw):
    w = wl.small(**kw)
    check_forward(orc, w)
    # window 1: P = 1 on the diagonal, dS = P (dP - D) = 0, so dW^Q = dW^K = 0
    check_backward(orc, w, zero=("dWq_d", "dWk_d") if w.window == 1 else ())


def test_workload_long_local_full(orc):
    """60 MoSA heads (k = 64) beside 4 local heads (window 512) at T = 8192,
    forward at full size."""
    w = wl.WORKLOADS["long_local_t8192"]
    check_forward(orc, w, wl.make_inputs(w, with_grad=False))
