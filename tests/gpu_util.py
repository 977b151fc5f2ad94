"""Helpers for the GPU parity tests: move seeded inputs to the device and back."""
import numpy as np
import torch

import workloads as wl
from paper_2505_00315_amd import mosa

TOL = {"bf16": 2e-2, "f32": 1e-5}


def to_dev(a):
    if a is None:
        return None
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def to_f64(t):
    if t.dtype == torch.bfloat16:
        return t.detach().float().cpu().numpy().astype(np.float64)
    return t.detach().cpu().numpy().astype(np.float64)


def rel_err(got, ref):
    den = np.abs(ref).max()
    return float(np.abs(got - ref).max() / (den if den > 0 else 1.0))


def shape_of(w: wl.Workload):
    return mosa.make_shape(w.batch, w.seq_len, w.d_model, w.heads, w.d_head, w.k, w.causal, w.dense_heads,
                           w.dtype, **w.variants())


def device_inputs(inp):
    return {n: to_dev(v) for n, v in inp.items() if v is not None}


def run_forward(w: wl.Workload, inp, accumulate=False, Y0=None):
    shape = shape_of(w)
    dev = device_inputs(inp)
    weights = {n: dev.get(n) for n in mosa.WEIGHT_NAMES}
    Y = Y0.clone() if Y0 is not None else None
    Y, saved, scratch = mosa.forward(shape, dev["X"], weights, Y=Y, accumulate=accumulate)
    torch.cuda.synchronize()
    out = {"Y": Y, "saved": saved, "scratch": scratch, "shape": shape, "dev": dev}
    if w.heads > 0:
        out["I"] = mosa.saved_view(shape, saved, "I").cpu().numpy()
        out["r"] = mosa.saved_view(shape, saved, "r").cpu().numpy().astype(np.float64)
    return out
