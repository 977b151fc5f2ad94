"""The allocation-free forward (mosa_forward_noalloc, scratch in the library's
static per-GPU buffer) through the C ABI against mosa_forward with a caller
scratch buffer: bitwise equal outputs and saved state, on two calls in a row,
the second with a smaller input; a shape whose forward needs more than the
static buffer is refused before any work."""
import numpy as np
import pytest
import torch

import workloads as wl
from gpu_util import device_inputs, shape_of
from paper_2505_00315_amd import mosa

pytestmark = pytest.mark.gpu


def _compare(w):
    print(f"\n[case] {w}", flush=True)
    inp = wl.make_inputs(w, with_grad=False)
    dev = device_inputs(inp)
    shape = shape_of(w)
    weights = {n: dev.get(n) for n in mosa.WEIGHT_NAMES}
    Y0, s0, _ = mosa.forward(shape, dev["X"], weights)
    sel = w.batch * w.heads * w.k
    I_out = torch.full((sel,), -7, dtype=torch.int32, device="cuda")
    r_out = torch.full((sel,), -7.0, dtype=torch.float32, device="cuda")
    Y1 = torch.full_like(dev["X"], 3.0)
    s1 = torch.full_like(s0, 0x5A)
    Y1, s1 = mosa.forward_noalloc(shape, dev["X"], weights, Y=Y1, saved=s1, I_out=I_out, r_out=r_out)
    torch.cuda.synchronize()
    mosa.check_selection(shape, s1)
    assert torch.equal(Y0, Y1)
    for n in ("I", "r", "slot", "QKV", "A", "lse", "status") + (("QKVd", "Ad", "lsed") if w.dense_heads else ()):
        assert torch.equal(mosa.saved_view(shape, s0, n), mosa.saved_view(shape, s1, n)), n
    assert torch.equal(I_out.view(w.batch, w.heads, w.k), mosa.saved_view(shape, s0, "I"))
    assert torch.equal(r_out.view(w.batch, w.heads, w.k), mosa.saved_view(shape, s0, "r"))


def test_noalloc_equals_forward_twice_second_smaller():
    big = wl.WORKLOADS["fwd_d512"]  # B=8, T=1024, d=512, 32 heads, k=128 (about 40 MB of scratch)
    small = wl.small(batch=2, seq_len=200, heads=3, k=40, d_model=128, dense_heads=1)
    _compare(big)
    _compare(small)


def test_noalloc_refuses_a_shape_beyond_the_static_buffer():
    w = wl.WORKLOADS["hybrid_d1024"]  # its forward needs well over 64 MiB of scratch
    shape = shape_of(w)
    X = torch.zeros(w.batch, w.seq_len, w.d_model, dtype=torch.bfloat16, device="cuda")
    weights = {}
    for n, numel in mosa._weight_numel(shape).items():
        weights[n] = torch.zeros(numel, dtype=torch.bfloat16, device="cuda") if numel else None
    with pytest.raises(mosa.MosaError) as e:
        mosa.forward_noalloc(shape, X, weights)
    assert e.value.status == mosa.MOSA_ERR_WORKSPACE
