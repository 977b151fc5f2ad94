"""Work accounting for the MoSA layer: algorithmic bytes and FLOPs per kernel
launch (the roofline of every stage), and the paper's FLOP model.

Algorithmic bytes count each input once and each output once (activations,
weights, compact k-sized per-head tensors); they exclude re-reads a kernel
does for its tiling and the T x T / k x d intermediates the method avoids.
FLOPs: 2 per multiply-add; attention counts only the causally allowed
(query, key) pairs.  The paper's own FLOP model (Section 3.2 and Appendix A)
is `paper_flops_*` below.
"""
from dataclasses import dataclass

HBM_PEAK = 8.0e12  # bytes/s, MI355X HBM3E
MFMA_PEAK = {"bf16": 2.5e15, "f32": 157.3e12}  # dense FLOP/s by operand type


@dataclass
class StageWork:
    name: str
    bytes: float
    flops: float


def _pairs(n, causal, window=0):
    """(query, key) pairs attention computes: all, the causal triangle, or the
    causal band of a local window (query t sees keys t - window + 1 .. t)."""
    if not causal:
        return n * n
    if window and window < n:
        return window * (window + 1) / 2 + (n - window) * window
    return n * (n + 1) / 2


def stage_work(w, with_backward=True):
    """Algorithmic work of every kernel the library times, keyed by stage name.
    The output side (out_proj + out_combine) and the dX side (dx_proj +
    dx_combine) are accounted as one stage each (GROUPS): their algorithmic
    bytes are those of the paper's operation (A, W^O and Y once; the per-head
    k x d rows that the two-kernel design writes and reads back are not
    algorithmic traffic)."""
    es = 2 if w.dtype == "bf16" else 4
    B, T, d, H, dh, k, Hd = w.batch, w.seq_len, w.d_model, w.heads, w.d_head, w.k, w.dense_heads
    X = B * T * d * es
    rows = B * H * k  # selected rows over all heads
    out = {}

    def add(name, nbytes, flops):
        out[name] = StageWork(name, float(nbytes), float(flops))

    if w.rope:
        add("rope_table", T * (dh // 4) * 8, 0.0)
    if H and w.fixed_stride:
        add("select", rows * 8 + B * H * T * 2, 0.0)  # I, r and the slot map written
    elif H:
        add("router", X + H * d * es + B * H * T * 4 + B * T * 4, 2.0 * B * T * H * d)
        add("select", B * H * T * 4 + B * T * 4 + H * d * es + rows * 8 + B * H * T * 2, 0.0)
    if H:
        add("qkv", X + 3 * H * d * dh * es + 3 * rows * dh * es + rows * 4, 2.0 * rows * d * 3 * dh)
        add("attn", 4 * rows * dh * es + rows * 4, 4.0 * dh * _pairs(k, w.causal) * B * H)
        # the two in one launch (groups of k | 128 rows): Q|K|V written once
        # and not read back, A and lse written, r read
        add("qkv_attn", out["qkv"].bytes + rows * dh * es + rows * 8, out["qkv"].flops + out["attn"].flops)
    if Hd:
        add("qkv_dense", X + 3 * Hd * d * dh * es + 3 * B * Hd * T * dh * es, 2.0 * B * Hd * T * d * 3 * dh)
        add("attn_dense", 4 * B * Hd * T * dh * es + B * Hd * T * 4,
            4.0 * dh * _pairs(T, w.causal, w.window) * B * Hd)
    add("out_scatter",
        rows * dh * es + rows * 8 + H * dh * d * es + B * Hd * T * dh * es + Hd * dh * d * es + X,
        2.0 * rows * dh * d + 2.0 * B * Hd * T * dh * d)
    if not with_backward:
        return out
    if H:
        add("bwd_out", X + H * dh * d * es + 2 * rows * dh * es + rows * 16, 2.0 * rows * d * dh)
        add("attn_bwd_kv", 6 * rows * dh * es + rows * 8, 8.0 * dh * _pairs(k, w.causal) * B * H)
        add("attn_bwd_q", 5 * rows * dh * es + rows * 8, 6.0 * dh * _pairs(k, w.causal) * B * H)
        # both passes: Q, K, V, dA read, dQ | dK | dV written, lse and D read
        add("attn_bwd", 7 * rows * dh * es + rows * 8, 14.0 * dh * _pairs(k, w.causal) * B * H)
        # dW^{Q,K,V,r} and dW^O (one grouped launch): X and dY read, the
        # selected rows' dQ|dK|dV and r A, I, the gradients written once
        add("wgrad", 2 * X + 4 * rows * dh * es + rows * 4 + 4 * H * d * dh * es + H * d * es,
            2.0 * rows * d * (3 * dh + 1) + 2.0 * rows * dh * d)
    if Hd:
        R = B * Hd * T
        add("bwd_out_dense", X + Hd * dh * d * es + 2 * R * dh * es + R * 4, 2.0 * R * d * dh)
        add("attn_bwd_kv_dense", 6 * R * dh * es + R * 8, 8.0 * dh * _pairs(T, w.causal, w.window) * B * Hd)
        add("attn_bwd_q_dense", 5 * R * dh * es + R * 8, 6.0 * dh * _pairs(T, w.causal, w.window) * B * Hd)
        add("attn_bwd_dense", 7 * R * dh * es + R * 8, 14.0 * dh * _pairs(T, w.causal, w.window) * B * Hd)
        add("wgrad_qkv_dense", X + 3 * R * dh * es + 3 * Hd * d * dh * es, 2.0 * R * d * 3 * dh)
        add("wgrad_o_dense", X + R * dh * es + Hd * dh * d * es, 2.0 * R * dh * d)
    add("dx_scatter",
        3 * rows * dh * es + rows * 8 + 3 * H * d * dh * es + H * d * es
        + 3 * B * Hd * T * dh * es + 3 * Hd * d * dh * es + X,
        2.0 * rows * 3 * dh * d + 2.0 * rows * d + 2.0 * B * Hd * T * 3 * dh * d)
    return out


# Stages made of two kernels (the library records one event per kernel); the
# attention backward's two passes are one stage (one launch does both when
# the group fits one workgroup).
GROUPS = {"out_scatter": ("out_proj", "out_combine"), "dx_scatter": ("dx_proj", "dx_combine"),
          "attn_bwd": ("attn_bwd_kv", "attn_bwd_q"), "attn_bwd_dense": ("attn_bwd_kv_dense", "attn_bwd_q_dense")}


def group_stage_times(kernel_ms):
    """Per-stage times from per-kernel times: a group is the sum of its kernels."""
    out = {}
    for name, ms in kernel_ms.items():
        for g, members in GROUPS.items():
            if name in members:
                out[g] = out.get(g, 0.0) + ms
                break
        else:
            out[name] = ms
    return out


def roofline(stage: StageWork, seconds: float, dtype: str):
    """Binding roofline of one stage at a measured time."""
    peak_f = MFMA_PEAK[dtype]
    ridge = peak_f / HBM_PEAK
    ai = stage.flops / stage.bytes if stage.bytes else float("inf")
    if stage.flops > 0 and ai >= ridge:
        achieved = stage.flops / seconds
        return {"bound": "mfma", "achieved": achieved / 1e12, "peak": peak_f / 1e12, "unit": "TFLOP/s",
                "frac": achieved / peak_f, "ai": ai}
    achieved = stage.bytes / seconds
    return {"bound": "hbm", "achieved": achieved / 1e9, "peak": HBM_PEAK / 1e9, "unit": "GB/s",
            "frac": achieved / HBM_PEAK, "ai": ai}


# ---------------------------------------------------------------------------
# The paper's FLOP model (Section 3.2 "FLOPs Calculation", Appendix A)
# ---------------------------------------------------------------------------

def paper_flops_dense_head(h, hp, T):
    """Q, K, V, O mappings 8 h h' T plus attention 4 h' T^2."""
    return 8 * h * hp * T + 4 * hp * T * T


def paper_flops_mosa_head(h, hp, T, k):
    """Mappings 8 h h' k, attention 4 h' k^2, routing overhead 2 h T + h' k."""
    return 8 * h * hp * k + 4 * hp * k * k + 2 * h * T + hp * k


def paper_flops_model(layers, h, hp, T, dense_heads, mosa_heads=0, k=0):
    """Forward FLOPs of a whole model: attention heads per layer plus the
    4h feed-forward block 16 h^2 T (Appendix A)."""
    return (layers * dense_heads * paper_flops_dense_head(h, hp, T)
            + layers * mosa_heads * (paper_flops_mosa_head(h, hp, T, k) if mosa_heads else 0)
            + 16 * layers * h * h * T)


def paper_mosa_heads_for_budget(layers, h, hp, T, baseline_heads, dense_heads, sparsity):
    """Largest number of MoSA heads whose model does not exceed the FLOPs of the
    dense baseline with `baseline_heads` heads (Section 3.2, Appendix A)."""
    budget = paper_flops_model(layers, h, hp, T, baseline_heads)
    k = T // sparsity
    fixed = paper_flops_model(layers, h, hp, T, dense_heads)
    return int((budget - fixed) // (layers * paper_flops_mosa_head(h, hp, T, k)))


# ---------------------------------------------------------------------------
# Measured HBM traffic per stage from rocprofv3 counter runs
# ---------------------------------------------------------------------------

# Kernel-name patterns of each stage (MoSA heads only: dense heads reuse the
# same kernels, so workloads with dense heads are not attributed here).
STAGE_KERNELS = {
    "router": (r"router_kernel", r"RouterPolicy2"),
    "select": (r"select_\w*kernel",),
    "rope_table": (r"rope_table_kernel",),
    "qkv": (r"(?<!Wgrad)QkvPolicy",),
    "qkv_attn": (r"QkvAttnPolicy",),
    "attn": (r"attn_fwd",),
    "out_scatter": (r"OutProj\w*Policy", r"OutCombinePolicy", r"OutDensePolicy", r"combine_rows_kernel<[^>]*, 0>"),
    "bwd_out": (r"BwdOutPolicy",),
    "attn_bwd": (r"attn_bwd_kv", r"attn_bwd_q", r"attn_bwd_lds", r"attn_bwd_tiled_both"),
    "wgrad": (r"WgradQkvPolicy<[^>]*, true, true>", r"WgradQkvPolicy2", r"WgradOPolicy<[^>]*, true>",
              r"WgradOPolicy2", r"wgrad_qkv_reduce", r"wgrad_o_reduce"),
    "dx_scatter": (r"DxProj\w*Policy", r"DxCombinePolicy", r"DxDensePolicy", r"combine_rows_kernel<[^>]*, 1>"),
}


GROUPED_KERNEL = r"group3_kernel"


def _read_counter_csv(run_dir):
    import csv
    import glob
    import os
    rows = []
    for f in sorted(glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True)):
        rows += list(csv.DictReader(open(f)))
    rows.sort(key=lambda r: int(r["Dispatch_Id"]))
    return rows


def traffic_summary(fetch_dir, write_dir, copy_bytes):
    """Per-stage HBM bytes per launch from a FETCH_SIZE run and a WRITE_SIZE
    run (KiB per dispatch) of `bench.py --calibrate-copy`: the last dispatch of
    each run is the plain copy of `copy_bytes` bytes, whose readings give the
    scale of each counter.  Returns (per-stage dict, fetch scale, write scale)."""
    import re
    fetch, write = _read_counter_csv(fetch_dir), _read_counter_csv(write_dir)
    if not fetch or not write:
        raise ValueError("no counter rows")
    f_scale = copy_bytes / (float(fetch[-1]["Counter_Value"]) * 1024.0)
    w_scale = copy_bytes / (float(write[-1]["Counter_Value"]) * 1024.0)
    out = {}
    for rows, key, scale in ((fetch, "fetch", f_scale), (write, "write", w_scale)):
        for stage, pats in STAGE_KERNELS.items():
            # grouped launches (several stages' work in one kernel) are left out;
            # a stage's traffic per launch = the sum over its kernels of each
            # kernel's average per dispatch (kernels may run in different steps)
            hit = [r for r in rows[:-1] if not re.search(GROUPED_KERNEL, r["Kernel_Name"])
                   and any(re.search(p, r["Kernel_Name"]) for p in pats)]
            if not hit:
                continue
            per = {}
            for r in hit:
                per.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
            kib = sum(sum(v) / len(v) for v in per.values())
            if kib:
                d = out.setdefault(stage, {})
                d[key + "_kib"] = kib
                d[key + "_bytes"] = kib * 1024.0 * scale
    for d in out.values():
        d["hbm_bytes_per_launch"] = d.get("fetch_bytes", 0.0) + d.get("write_bytes", 0.0)
    return out, f_scale, w_scale


if __name__ == "__main__":
    import argparse

    ap = argparse.ArgumentParser(description="write the per-stage HBM traffic summary from two rocprofv3 "
                                             "counter runs of bench.py --calibrate-copy")
    ap.add_argument("--fetch", required=True, help="output directory of the FETCH_SIZE run")
    ap.add_argument("--write", required=True, help="output directory of the WRITE_SIZE run")
    ap.add_argument("--copy-bytes", type=int, required=True)
    ap.add_argument("--workload", required=True)
    ap.add_argument("--source", default="paper_2505_00315_amd/csrc")
    ap.add_argument("--source-sha", required=True)
    ap.add_argument("--command", default="")
    a = ap.parse_args()
    stages, fs, ws = traffic_summary(a.fetch, a.write, a.copy_bytes)
    print(f"# HBM traffic per launch of each stage, workload {a.workload}: rocprofv3 FETCH_SIZE and WRITE_SIZE "
          f"(KiB per dispatch, one run each), scaled by the readings of a plain {a.copy_bytes}-byte device copy "
          f"in the same run (fetch x{fs:.4f}, write x{ws:.4f}).")
    if a.command:
        print(f"# command: {a.command}")
    for name, d in stages.items():
        print(f"stage={name} workload={a.workload} source={a.source} source_sha={a.source_sha} "
              f"fetch_kib={d.get('fetch_kib', 0):.1f} write_kib={d.get('write_kib', 0):.1f} "
              f"hbm_bytes_per_launch={d['hbm_bytes_per_launch']:.0f}")
