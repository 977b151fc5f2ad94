"""GPU parity at the edges of the supported range: the longest sequence,
the widest model, many heads, ragged group and tile sizes, k = T, fp32
beyond one tile, local heads over many tiles.  Same bars as the other
parity tests (indices bit-exact, relative errors per tensor)."""
import pytest

import workloads as wl
from test_gpu_variants import check_backward, check_forward

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("kw", [
    dict(batch=1, seq_len=16384, d_model=64, heads=2, d_head=32, k=64),       # longest T
    dict(batch=1, seq_len=16384, d_model=64, heads=1, d_head=64, k=2048),     # longest T, k > 128
    dict(batch=1, seq_len=64, d_model=2048, heads=2, d_head=64, k=16),        # widest d
    dict(batch=2, seq_len=128, d_model=64, heads=300, d_head=32, k=8),        # heads past 4 x 64
    dict(batch=2, seq_len=77, d_model=64, heads=2, d_head=32, k=77),          # k = T, ragged T
    dict(batch=5, seq_len=100, d_model=128, heads=3, d_head=64, k=48),        # group not dividing 128
    dict(batch=1, seq_len=300, d_model=64, heads=2, d_head=32, k=200, dtype="f32"),
    dict(batch=1, seq_len=400, d_model=64, heads=2, d_head=64, k=300, causal=False),
    dict(batch=1, seq_len=2048, d_model=64, heads=1, d_head=32, k=32, dense_heads=1, window=200),
])
def test_limits(orc, kw):
    w = wl.small(**kw)
    check_forward(orc, w)
    check_backward(orc, w)
