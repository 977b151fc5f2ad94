"""Why the per-row bar is not applied to the MoSA heads' weight gradients when
a head has very few selected rows (test_gpu_random_shapes.py): a CPU emulation
of the path's bf16 roundings alone (A and dA stored in bf16, D = <dA~, A> from
the stored A, dS rounded to bf16 as an MFMA operand; Section 2.2 backward with
I fixed, the R13 precision reading) against the exact oracle.  Under causal
masking the first selected row of each (b, h) attends only to itself, so its dS
is zero exactly; the residue dP - D of the rounded values is then a large
share of some rows of dW^Q when there are only B k = 4 rows per head, while
the whole tensor stays far inside its bar."""
import numpy as np

import oracle as orc
import workloads as wl
from gpu_util import ROW_TOL, TOL, rel_err, row_rel_err


def _bf16(x):
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def _f64(a):
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def _dwq(w, inp, rounded):
    opts = orc.options(**w.variants())
    f = orc.forward(inp, w.k, causal=w.causal, intermediates=True, opts=opts)
    X, dY, Wo = _f64(inp["X"]), _f64(inp["dY"]), _f64(inp["Wo"])
    I, r, Q, K, V = f["I"], f["r"], f["Q"], f["K"], f["V"]
    B, H, k, dh = Q.shape
    out = np.zeros((H, X.shape[2], dh))
    allowed = np.tril(np.ones((k, k))) > 0 if w.causal else np.ones((k, k), dtype=bool)
    for h in range(H):
        for b in range(B):
            S = np.where(allowed, Q[b, h] @ K[b, h].T / np.sqrt(dh), -np.inf)
            P = np.exp(S - S.max(1, keepdims=True))
            P /= P.sum(1, keepdims=True)
            rb = r[b, h][:, None]
            dAt = dY[b, I[b, h]] @ Wo[h].T
            if rounded:
                A, dA = _bf16(rb * (P @ V[b, h])), _bf16(rb * dAt)
                dP = dA @ V[b, h].T
                dS = _bf16(P * (dP - (dAt * A).sum(1)[:, None]))
            else:
                dP = (rb * dAt) @ V[b, h].T
                dS = P * (dP - (P * dP).sum(1)[:, None])
            out[h] += X[b, I[b, h]].T @ (dS @ K[b, h] / np.sqrt(dh))
    return out


def test_emulation_exact_path_is_the_oracle():
    w = wl.small(batch=2, seq_len=134, d_model=192, heads=2, d_head=64, k=2, dense_heads=1, first_token=True, seed=1015)
    inp = wl.make_inputs(w, with_grad=True)
    ref = orc.backward(inp, inp["dY"], w.k, causal=w.causal, opts=orc.options(**w.variants()))["dWq"]
    assert rel_err(_dwq(w, inp, rounded=False), ref) < 1e-12


def test_bf16_roundings_alone_exceed_the_row_bar_for_two_rows_per_head():
    w = wl.small(batch=2, seq_len=134, d_model=192, heads=2, d_head=64, k=2, dense_heads=1, first_token=True, seed=1015)
    inp = wl.make_inputs(w, with_grad=True)
    ref = orc.backward(inp, inp["dY"], w.k, causal=w.causal, opts=orc.options(**w.variants()))["dWq"]
    emu = _dwq(w, inp, rounded=True)
    assert rel_err(emu, ref) <= TOL["bf16"]
    assert row_rel_err(emu, ref) > ROW_TOL["bf16"]
