"""The algorithmic work behind the benchmark's roofline, checked against byte
and FLOP counts written out by hand, and the labelling of rocprofv3 dispatches
by their position in a step."""
import pytest

import perfmodel as pm
import workloads as wl


def test_output_side_of_the_forward_workload():
    w = wl.WORKLOADS["fwd_d512"]  # B=8, T=1024, d=512, 32 heads, dh=64, k=128, bf16
    st = pm.stage_work(w, with_backward=False)
    rows = 8 * 32 * 128
    X = 8 * 1024 * 512 * 2
    # r A rows and W^O read; the k x d rows it writes are an intermediate
    assert st["out_proj"].bytes == rows * 64 * 2 + 32 * 64 * 512 * 2
    assert st["out_proj"].flops == 2 * rows * 64 * 512
    # the head-ordered sum: slot map read, Y written
    assert st["out_combine"].bytes == X + 8 * 32 * 1024 * 2
    assert st["out_scatter"].bytes == st["out_proj"].bytes + st["out_combine"].bytes + rows * 8
    assert "bwd_proj" not in st


def test_grouped_backward_of_the_hybrid_workload():
    w = wl.WORKLOADS["hybrid_d1024"]  # B=8, T=1024, d=1024, 256 MoSA heads (k=16) + 4 dense, dh=64
    st = pm.stage_work(w, with_backward=True)
    rows, X, H, d, dh = 8 * 256 * 16, 8 * 1024 * 1024 * 2, 256, 1024, 64
    wgrad = 2 * X + 4 * rows * dh * 2 + rows * 4 + 4 * H * d * dh * 2 + H * d * 2
    assert st["wgrad"].bytes == wgrad
    # weight gradients + the dX rows' weight reads (W^Q, W^K, W^V and W^r)
    assert st["bwd_proj"].bytes == wgrad + 3 * H * d * dh * 2 + H * d * 2
    assert round(st["bwd_proj"].bytes / 1e6, 1) == 286.4
    assert st["bwd_proj"].flops == 2 * rows * d * (3 * dh + 1) * 2 + 2 * rows * dh * d
    # dense heads' attention backward: 2.5 times the forward's causal pairs work
    assert st["attn_bwd_dense"].flops == 2.5 * st["attn_dense"].flops


def test_causal_pairs_and_window():
    assert pm._pairs(4, causal=False) == 16
    assert pm._pairs(4, causal=True) == 10
    # window 2 at n = 4: query t sees t-1, t -> 1 + 2 + 2 + 2
    assert pm._pairs(4, causal=True, window=2) == 7
    assert pm._pairs(4, causal=True, window=4) == 10


def test_roofline_fraction():
    st = pm.StageWork("x", 8e9, 0.0)
    r = pm.roofline(st, 1e-3, "bf16")
    assert r["bound"] == "hbm" and abs(r["frac"] - 1.0) < 1e-9
    st = pm.StageWork("y", 1e6, 2.5e12)
    r = pm.roofline(st, 1e-3, "bf16")
    assert r["bound"] == "mfma" and abs(r["frac"] - 1.0) < 1e-9


def _disp(name, t0=0, dur=1000, **ctr):
    return (name, dict(ctr), t0, t0 + dur)


def test_dispatches_labelled_by_position():
    info = {"order": ["router", "select", "bwd_proj"], "warmup": 1, "steps": 2}
    k = ["void mosa::gemm2_kernel<R>(A)", "void mosa::select_rows_kernel<S>(B)", "void mosa::group3_kernel<G>(C)"]
    disp = []
    for step in range(3):
        disp += [_disp(k[0], dur=1000 + step), _disp(k[1], dur=2000), _disp(k[2], dur=3000, FETCH_SIZE=10.0)]
        if step == 0:
            disp.append(_disp("void at::native::reduce_kernel<X>(Y)"))  # torch's own kernel in between
    disp.append(_disp("__amd_rocclr_copyBuffer", FETCH_SIZE=5.0))
    lab, other = pm.label_dispatches(disp, info)
    # the warm-up step (untimed, its own launch order) is left out
    assert [s for s, _ in lab] == info["order"] * 2
    assert other[-1][0] == "__amd_rocclr_copyBuffer"
    ps = pm.per_stage(lab)
    assert ps["router"]["calls"] == 2 and abs(ps["router"]["us"] - 1.0015) < 1e-9
    assert ps["bwd_proj"]["FETCH_SIZE"] == 10.0 and ps["select"]["kernel"] == "select_rows_kernel<S>"
    assert pm.copy_scale(other, 1024 * 5 * 2, "FETCH_SIZE") == 2.0
    warm = list(disp)
    warm[0], warm[1] = warm[1], warm[0]  # a warm-up step in another order is fine
    assert [s for s, _ in pm.label_dispatches(warm, info)[0]] == info["order"] * 2
    with pytest.raises(ValueError):  # a position that changes kernel is refused
        bad = list(disp)
        bad[4] = _disp(k[1])
        pm.label_dispatches(bad, info)
    with pytest.raises(ValueError):  # a missing dispatch is refused
        pm.label_dispatches(disp[1:], info)
