"""Helpers for the GPU parity tests: move seeded inputs to the device and back."""
import numpy as np
import torch

import workloads as wl
from paper_2505_00315_amd import mosa

TOL = {"bf16": 2e-2, "f32": 1e-5}
# Per-row bar (row_rel_err): 2.5 times the normwise one.  A row of a gradient
# sums as few as B k terms computed from bf16-rounded operands, and where they
# cancel its rounding error reaches about 2e-2 of its own magnitude (measured:
# up to 2.0e-2 on rows at 15% of the tensor maximum); a missing, extra or
# wrongly scaled head contribution moves the rows it touches by far more.
ROW_TOL = {"bf16": 5e-2, "f32": 2.5e-5}


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
    """Normwise error of a whole tensor: max |got - ref| / max |ref|."""
    den = np.abs(ref).max()
    return float(np.abs(got - ref).max() / (den if den > 0 else 1.0))


def row_rel_err(got, ref, floor=1e-2):
    """Worst per-row error: for every row (last axis) max |got - ref| over the
    row divided by max |ref| over the row, the divisor held at least at
    ``floor`` times the tensor's max |ref| (rows far below the tensor's scale
    are covered by rel_err alone).  A wrong contribution to a few rows of a
    low-magnitude head shows here even when it hides under the tensor max."""
    g = np.asarray(got, dtype=np.float64).reshape(-1, got.shape[-1])
    r = np.asarray(ref, dtype=np.float64).reshape(-1, ref.shape[-1])
    top = np.abs(r).max()
    if top == 0:
        return float(np.abs(g).max())
    den = np.maximum(np.abs(r).max(axis=1), floor * top)
    return float((np.abs(g - r).max(axis=1) / den).max())


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
    mosa.check_selection(shape, saved)
    out = {"Y": Y, "saved": saved, "scratch": scratch, "shape": shape, "dev": dev}
    if w.heads > 0:
        out["I"] = mosa.saved_view(shape, saved, "I").cpu().numpy()
        out["r"] = mosa.saved_view(shape, saved, "r").cpu().numpy().astype(np.float64)
    return out
