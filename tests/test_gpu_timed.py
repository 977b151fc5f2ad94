"""The stage-timed entry points (mosa_forward_timed / mosa_backward_timed with
events) launch exactly the kernels of the untimed calls: their outputs must be
bitwise equal to the untimed ones and within the parity bar of the oracle, for
every launch shape the benchmark times (projection and attention in one launch
for k | 128; the tiled attention for k > 128; dense heads; local dense heads;
fp32 storage)."""
import numpy as np
import pytest
import torch

import workloads as wl
from gpu_util import ROW_TOL, TOL, device_inputs, rel_err, row_rel_err, shape_of, to_f64
from paper_2505_00315_amd import mosa

pytestmark = pytest.mark.gpu

CASES = {
    "fused_k64": dict(batch=2, seq_len=256, heads=3, k=64, d_head=64, d_model=128),
    "tiled_k200": dict(batch=2, seq_len=400, heads=2, k=200, d_head=64, d_model=128),
    "k16_dense2": dict(batch=2, seq_len=256, heads=4, k=16, d_head=64, d_model=128, dense_heads=2),
    "window": dict(batch=1, seq_len=300, heads=2, k=40, d_head=64, d_model=128, dense_heads=2, window=24),
    "f32": dict(batch=2, seq_len=128, heads=3, k=30, dtype="f32", dense_heads=1),
}


def _step(w, dev, timer=None):
    shape = shape_of(w)
    weights = {n: dev.get(n) for n in mosa.WEIGHT_NAMES}
    fe = timer.sets[0] if timer else None
    be = timer.sets[1] if timer else None
    Y, saved, scratch = mosa.forward(shape, dev["X"], weights, events=fe)
    grads = {"d" + n: torch.empty_like(dev[n]) for n in mosa.WEIGHT_NAMES if dev.get(n) is not None}
    dX = mosa.backward(shape, dev["X"], weights, dev["dY"], saved, grads, scratch=scratch, events=be)
    torch.cuda.synchronize()
    mosa.check_selection(shape, saved)
    return Y, dX, grads, saved


@pytest.mark.parametrize("case", sorted(CASES))
def test_timed_equals_untimed_and_oracle(orc, case):
    w = wl.small(name=case, **CASES[case])
    print(f"\n[case] {w}", flush=True)
    inp = wl.make_inputs(w, with_grad=True)
    dev = device_inputs(inp)
    Y0, dX0, g0, s0 = _step(w, dev)
    timer = mosa.StageTimer(sets=2)
    try:
        Y1, dX1, g1, s1 = _step(w, dev, timer)
        fwd = timer.stages(timer.sets[0])
        bwd = timer.stages(timer.sets[1])
    finally:
        timer.close()
    print(f"[case] stages {[n for n, _ in fwd]} | {[n for n, _ in bwd]}", flush=True)
    assert fwd and bwd and all(ms >= 0 for _, ms in fwd + bwd)
    names = [n for n, _ in fwd + bwd]
    assert "out_combine" in names and "dx_combine" in names
    if w.heads:
        assert "select" in names and ("bwd_proj" in names or "dx_proj" in names)
    if w.dense_heads:
        assert "attn_dense" in names and any(n.startswith("attn_bwd") and n.endswith("dense") for n in names)
    # the timed calls launch the same kernels: bitwise equal results
    assert torch.equal(Y0, Y1) and torch.equal(dX0, dX1)
    for n in g0:
        assert torch.equal(g0[n], g1[n]), n
    shape = shape_of(w)
    for n in ("I", "r"):
        assert torch.equal(mosa.saved_view(shape, s0, n), mosa.saved_view(shape, s1, n)), n
    # and they agree with the oracle
    ref_f = orc.forward(inp, w.k, causal=w.causal, opts=orc.options(**w.variants()))
    ref_b = orc.backward(inp, inp["dY"], w.k, causal=w.causal, opts=orc.options(**w.variants()))
    I1 = mosa.saved_view(shape, s1, "I").cpu().numpy()
    assert np.array_equal(I1, ref_f["I"])
    got = {"Y": to_f64(Y1), "dX": to_f64(dX1)}
    got.update({n: to_f64(t) for n, t in g1.items() if n in ref_b})
    want = {"Y": ref_f["Y"], **ref_b}
    for n, v in got.items():
        e, er = rel_err(v, want[n]), row_rel_err(v, want[n])
        assert e <= TOL[w.dtype] and er <= ROW_TOL[w.dtype], (n, e, er)
