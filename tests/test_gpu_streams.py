"""The layer on caller streams other than the default one, and from several
host threads at once.  The untimed calls of a layer with both kinds of heads
run the dense heads' kernels on the library's auxiliary stream, forked from
and joined back into the caller's stream inside each call: results must be
bitwise the same whatever stream the caller uses, for back-to-back calls
without a host synchronisation between them, and for calls that two host
threads enqueue at the same time on two streams."""
import threading

import numpy as np
import pytest
import torch

import workloads as wl
from gpu_util import device_inputs, shape_of
from paper_2505_00315_amd import mosa

pytestmark = pytest.mark.gpu

W = wl.small(name="streams_hybrid", batch=2, seq_len=256, heads=4, k=16, d_head=64, d_model=128, dense_heads=2)


def _alloc(dev):
    grads = {"d" + n: torch.empty_like(dev[n]) for n in mosa.WEIGHT_NAMES if dev.get(n) is not None}
    return grads


def _step(dev, stream=None):
    """Forward and backward on `stream` (None: the current stream), no host sync."""
    shape = shape_of(W)
    weights = {n: dev.get(n) for n in mosa.WEIGHT_NAMES}
    Y, saved, scratch = mosa.forward(shape, dev["X"], weights, stream=stream)
    grads = _alloc(dev)
    dX = mosa.backward(shape, dev["X"], weights, dev["dY"], saved, grads, scratch=scratch, stream=stream)
    return {"Y": Y, "dX": dX, **grads, "saved": saved}


def _host(out):
    return {k: v.detach().cpu().view(torch.int16).numpy() if v.dtype == torch.bfloat16 else v.detach().cpu().numpy()
            for k, v in out.items() if k != "saved"}


def _same(a, b, what):
    for k in a:
        assert np.array_equal(a[k], b[k]), f"{what}: {k} differs"


@pytest.fixture(scope="module")
def reference():
    inp = wl.make_inputs(W, with_grad=True)
    dev = device_inputs(inp)
    out = _step(dev)
    torch.cuda.synchronize()
    mosa.check_selection(shape_of(W), out["saved"])
    return dev, _host(out)


def test_side_stream_matches_default(reference):
    dev, ref = reference
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        out = _step(dev, stream=s)
    s.synchronize()
    _same(_host(out), ref, "side stream")


def test_back_to_back_calls(reference):
    dev, ref = reference
    # two different inputs enqueued back to back, then the reference input
    # again, with no host synchronisation in between
    other = device_inputs(wl.make_inputs(wl.small(name="streams_other", batch=2, seq_len=256, heads=4, k=16,
                                                  d_head=64, d_model=128, dense_heads=2, seed=9), with_grad=True))
    out_a = _step(dev)
    out_b = _step(other)
    out_c = _step(dev)
    torch.cuda.synchronize()
    _same(_host(out_a), ref, "first call")
    _same(_host(out_c), ref, "third call")
    assert not np.array_equal(_host(out_b)["Y"], ref["Y"])


def test_two_host_threads(reference):
    dev, ref = reference
    results, errors = {}, []

    def worker(tid):
        try:
            torch.cuda.set_device(0)
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                outs = [_step(dev, stream=s) for _ in range(3)]
            s.synchronize()
            results[tid] = [_host(o) for o in outs]
        except Exception as exc:  # reported by the main thread
            errors.append(repr(exc))

    torch.cuda.synchronize()
    threads = [threading.Thread(target=worker, args=(t,)) for t in range(2)]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not errors, errors
    assert sorted(results) == [0, 1]
    for tid, outs in results.items():
        for i, o in enumerate(outs):
            _same(o, ref, f"thread {tid} call {i}")
