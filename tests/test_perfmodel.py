"""The algorithmic work behind the benchmark's roofline, checked against the
byte and FLOP counts written out for the default workload (B=8, T=1024,
d=512, 32 heads, dh=64, k=128, bf16: 2-byte elements)."""
import perfmodel as pm
import workloads as wl


def test_scatter_stages_of_the_default_workload():
    w = wl.WORKLOADS["fwd_d512"]
    st = pm.stage_work(w, with_backward=True)
    rows = 8 * 32 * 128          # selected rows over all heads
    X = 8 * 1024 * 512 * 2       # one [B, T, d] bf16 tensor
    # dX side: dQ|dK|dV rows, I and dz per row, W^{Q,K,V} and W^r read once, dX written
    assert st["dx_scatter"].bytes == 3 * rows * 64 * 2 + rows * 8 + 3 * 32 * 512 * 64 * 2 + 32 * 512 * 2 + X
    assert st["dx_scatter"].bytes == 27557888
    assert st["dx_scatter"].flops == 2 * rows * 192 * 512 + 2 * rows * 512
    # output side: A rows, I and r, W^O once, Y written
    assert st["out_scatter"].bytes == rows * 64 * 2 + rows * 8 + 32 * 64 * 512 * 2 + X
    assert st["out_scatter"].flops == 2 * rows * 64 * 512


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
