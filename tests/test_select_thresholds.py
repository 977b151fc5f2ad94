"""The one-wave selection classifies most tokens by comparing their fp32
logit with two row-wide thresholds instead of evaluating their own interval
[lo_t, hi_t].  This checks, on the CPU with the same float operations, that
the shortcut never decides differently: z <= Lo implies hi_t < A (certainly
out) and z >= Hi implies lo_t > B (certainly in) for every beta_t <= bmax,
including logits at and next to the thresholds."""
import numpy as np

F32 = np.float32


def order_key(f):
    u = np.asarray(f, dtype=F32).view(np.uint32).copy()
    u[u == 0x80000000] = 0
    return np.where(u & 0x80000000, ~u, u | 0x80000000).astype(np.uint32)


def key_float(k):
    k = np.asarray(k, dtype=np.uint32)
    return np.where(k & 0x80000000, k & 0x7FFFFFFF, ~k).astype(np.uint32).view(F32)


def f32_down(x):
    f = x.astype(F32)
    return np.where(f.astype(np.float64) > x, np.nextafter(f, F32(-np.inf)), f)


def f32_up(x):
    f = x.astype(F32)
    return np.where(f.astype(np.float64) < x, np.nextafter(f, F32(np.inf)), f)


def next_up(f):
    return np.nextafter(np.asarray(f, dtype=F32), F32(np.inf))


def next_down(f):
    return -next_up(-np.asarray(f, dtype=F32))


def thresholds(pref, bmax):
    tlo, thi = key_float(pref), key_float(pref | 0x3FF)
    A = order_key(f32_down(tlo.astype(np.float64) - bmax))
    B = order_key(f32_up(thi.astype(np.float64) + bmax))
    lf = next_down(f32_down(next_down(key_float(A)).astype(np.float64) - bmax))
    hf = next_up(f32_up(next_up(key_float(B)).astype(np.float64) + bmax))
    return A, B, lf, hf


def test_threshold_shortcut_is_sound():
    rng = np.random.default_rng(7)
    checked = 0
    for _ in range(400):
        scale = F32(10.0 ** rng.uniform(-3, 3))
        z = (rng.standard_normal(512) * scale).astype(F32)
        tau = F32(np.sort(z)[-rng.integers(1, 64)])
        pref = int(order_key(tau)) & ~0x3FF
        bmax = float(abs(tau) + scale) * 10.0 ** rng.uniform(-9, -2)
        A, B, lf, hf = thresholds(np.uint32(pref), bmax)
        lo_key, hi_key = order_key(lf), order_key(hf)
        # logits at, just beside and around both thresholds, and random ones
        edges = np.array([lf, hf, next_up(lf), next_down(lf), next_up(hf), next_down(hf)], dtype=F32)
        probe = np.concatenate([z, edges, np.linspace(lf, hf, 64).astype(F32)])
        for beta in (bmax, bmax * rng.uniform(0, 1), 0.0):
            lo = order_key(f32_down(probe.astype(np.float64) - beta))
            hi = order_key(f32_up(probe.astype(np.float64) + beta))
            k = order_key(probe)
            fin, fout = k >= hi_key, k <= lo_key
            assert (lo[fin] > B).all()
            assert (hi[fout] < A).all()
            checked += int(fin.sum() + fout.sum())
    assert checked > 100000


def test_thresholds_leave_a_narrow_band():
    """The shortcut decides all but the tokens near tau."""
    rng = np.random.default_rng(8)
    z = rng.standard_normal(1024).astype(F32)
    tau = F32(np.sort(z)[-17])
    A, B, lf, hf = thresholds(order_key(tau) & np.uint32(0xFFFFFC00), 1e-5)
    k = order_key(z)
    band = (k > order_key(lf)) & (k < order_key(hf))
    assert 1 <= band.sum() <= 4
