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
SIMDS = 1024  # 256 CUs x 4
SHADER_ENGINES = 32  # 8 XCDs x 4; SQ_BUSY_CYCLES is summed over them
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
    """Algorithmic work per launch of every kernel the library launches, keyed
    by the stage name the timed entry points give that launch, plus the
    paper's two-kernel operations (GROUPS) as composite entries.  Per-head
    k x d rows that the two-kernel output and dX sides write and read back,
    fp32 partial sums and the dense heads' fp32 part of Y or dX are
    intermediates of this implementation, not algorithmic traffic: the
    kernels that produce or consume them are charged only for the layer's own
    tensors they read or write."""
    es = 2 if w.dtype == "bf16" else 4
    B, T, d, H, dh, k, Hd = w.batch, w.seq_len, w.d_model, w.heads, w.d_head, w.k, w.dense_heads
    X = B * T * d * es
    rows = B * H * k  # selected rows over all heads
    R = B * Hd * T    # dense-head rows
    out = {}

    def add(name, nbytes, flops):
        out[name] = StageWork(name, float(nbytes), float(flops))

    if w.rope:
        add("rope_table", T * (dh // 4) * 8, 0.0)
    if H and w.fixed_stride:
        add("select", rows * 8 + B * H * T * 2 + B * H * 4, 0.0)  # I, r, the slot map and status written
    elif H:
        add("router", X + H * d * es + B * H * T * 4 + B * T * 4, 2.0 * B * T * H * d)
        add("select", B * H * T * 4 + B * T * 4 + H * d * es + rows * 8 + B * H * T * 2 + B * H * 4, 0.0)
    if H:
        add("qkv", X + 3 * H * d * dh * es + 3 * rows * dh * es + rows * 4, 2.0 * rows * d * 3 * dh)
        add("attn", 4 * rows * dh * es + rows * 4, 4.0 * dh * _pairs(k, w.causal) * B * H)
        # the two in one launch (groups of k | 128 rows): Q|K|V written once
        # and not read back, A and lse written, r read
        add("qkv_attn", out["qkv"].bytes + rows * dh * es + rows * 8, out["qkv"].flops + out["attn"].flops)
        # X^o = (r A) W^O: the scaled rows and W^O read (the k x d rows it
        # writes are an intermediate)
        add("out_proj", rows * dh * es + H * dh * d * es, 2.0 * rows * dh * d)
    if Hd:
        add("qkv_dense", X + 3 * Hd * d * dh * es + 3 * R * dh * es, 2.0 * R * d * 3 * dh)
        add("attn_dense", 4 * R * dh * es + R * 4, 4.0 * dh * _pairs(T, w.causal, w.window) * B * Hd)
        add("out_dense", R * dh * es + Hd * dh * d * es, 2.0 * R * dh * d)
    # head-ordered sum: the slot map read, Y written
    add("out_combine", X + B * H * T * 2, 0.0)
    add("out_scatter", out["out_combine"].bytes + (out["out_proj"].bytes if H else 0.0)
        + (out["out_dense"].bytes if Hd else 0.0) + rows * 8,
        (out["out_proj"].flops if H else 0.0) + (out["out_dense"].flops if Hd else 0.0))
    if not with_backward:
        return out
    if H:
        add("bwd_out", X + H * dh * d * es + 2 * rows * dh * es + rows * 16, 2.0 * rows * d * dh)
        add("attn_bwd_kv", 6 * rows * dh * es + rows * 8, 8.0 * dh * _pairs(k, w.causal) * B * H)
        add("attn_bwd_q", 5 * rows * dh * es + rows * 8, 6.0 * dh * _pairs(k, w.causal) * B * H)
        # both passes: Q, K, V, dA read, dQ | dK | dV written, lse and D read;
        # five products over the allowed pairs (S recomputed, dP, dV, dK, dQ),
        # 2.5 times the forward's two
        add("attn_bwd", 7 * rows * dh * es + rows * 8, 10.0 * dh * _pairs(k, w.causal) * B * H)
        # dW^{Q,K,V,r} and dW^O: X and dY read, the selected rows' dQ|dK|dV
        # and r A, I, the gradients written once
        add("wgrad", 2 * X + 4 * rows * dh * es + rows * 4 + 4 * H * d * dh * es + H * d * es,
            2.0 * rows * d * (3 * dh + 1) + 2.0 * rows * dh * d)
        # the per-head dX rows: dQ|dK|dV, dz, W^{Q,K,V} and W^r read (the rows
        # written are an intermediate)
        add("dx_proj", 3 * rows * dh * es + rows * 4 + 3 * H * d * dh * es + H * d * es,
            2.0 * rows * 3 * dh * d + 2.0 * rows * d)
        # the grouped launch of both (dQ|dK|dV counted once)
        add("bwd_proj", out["wgrad"].bytes + 3 * H * d * dh * es + H * d * es,
            out["wgrad"].flops + out["dx_proj"].flops)
    if Hd:
        add("bwd_out_dense", X + Hd * dh * d * es + 2 * R * dh * es + R * 4, 2.0 * R * d * dh)
        add("attn_bwd_kv_dense", 6 * R * dh * es + R * 8, 8.0 * dh * _pairs(T, w.causal, w.window) * B * Hd)
        add("attn_bwd_q_dense", 5 * R * dh * es + R * 8, 6.0 * dh * _pairs(T, w.causal, w.window) * B * Hd)
        add("attn_bwd_dense", 7 * R * dh * es + R * 8, 10.0 * dh * _pairs(T, w.causal, w.window) * B * Hd)
        add("wgrad_qkv_dense", X + 3 * R * dh * es + 3 * Hd * d * dh * es, 2.0 * R * d * 3 * dh)
        add("wgrad_o_dense", X + R * dh * es + Hd * dh * d * es, 2.0 * R * dh * d)
        add("dx_dense", 3 * R * dh * es + 3 * Hd * d * dh * es, 2.0 * R * 3 * dh * d)
    add("dx_combine", X + B * H * T * 2, 0.0)
    return out


# The paper's operations that run as two kernels here (composite entries of
# stage_work): the router-scaled output projection with the head-ordered sum.
GROUPS = {"out_scatter": ("out_proj", "out_dense", "out_combine")}


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
# rocprofv3 summaries per kernel launch (stage names from the kernel order)
# ---------------------------------------------------------------------------
#
# `bench.py --profile --order-file F` runs W warm-up and K stage-timed steps
# of one workload and writes the stage names of one step's launches, in
# order, to F.  Every step launches the same kernels in the same order, so the
# library's dispatches of a rocprofv3 run map to stage names by position.
# Kernels outside the library's namespace (torch's own, the calibration copy)
# are set aside.


def _read_csvs(run_dir, suffix):
    import csv
    import glob
    import os
    rows = []
    for f in sorted(glob.glob(os.path.join(run_dir, "**", "*" + suffix), recursive=True)):
        rows += list(csv.DictReader(open(f)))
    return rows


def _by_dispatch(rows):
    """{dispatch id: (kernel name, {counter: value}, start ns, end ns)} in dispatch order."""
    out = {}
    for r in rows:
        d = int(r["Dispatch_Id"])
        e = out.setdefault(d, [r["Kernel_Name"], {}, int(r["Start_Timestamp"]), int(r["End_Timestamp"])])
        if "Counter_Name" in r:
            e[1][r["Counter_Name"]] = e[1].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    return [tuple(out[d]) for d in sorted(out)]


def label_dispatches(dispatches, order_info):
    """Stage name of every library dispatch of the stage-timed steps (by
    position in the step; the warm-up steps before them are untimed steps,
    whose launch order differs where two streams are used, and are left out)
    and the dispatches outside the library (in order).  Checks that each
    position always runs the same kernel."""
    lib = [x for x in dispatches if "mosa::" in x[0]]
    other = [x for x in dispatches if "mosa::" not in x[0]]
    order = order_info["order"]
    n = (order_info["warmup"] + order_info["steps"]) * len(order)
    if len(lib) != n:
        raise ValueError(f"{len(lib)} library dispatches, expected {n} ({order_info['warmup']} + "
                         f"{order_info['steps']} steps of {len(order)} launches)")
    lib = lib[order_info["warmup"] * len(order):]
    kern = {}
    labelled = []
    for i, x in enumerate(lib):
        st = order[i % len(order)]
        if kern.setdefault(st, x[0]) != x[0]:
            raise ValueError(f"stage {st} ran {x[0]} and {kern[st]}")
        labelled.append((st, x))
    return labelled, other


def short_kernel(name):
    """Kernel name without namespaces and argument lists."""
    import re
    n = re.sub(r"mosa::|\(anonymous namespace\)::", "", name)
    n = n[5:] if n.startswith("void ") else n
    return n.split("(")[0].replace("unsigned short", "bf16")


def per_stage(labelled):
    """{stage: {"kernel", "calls", "us" (mean), "us_min", "us_max", counters averaged}}."""
    acc = {}
    for st, (name, ctr, t0, t1) in labelled:
        e = acc.setdefault(st, {"kernel": short_kernel(name), "dur": [], "ctr": {}})
        e["dur"].append((t1 - t0) / 1e3)
        for c, v in ctr.items():
            e["ctr"].setdefault(c, []).append(v)
    out = {}
    for st, e in acc.items():
        d = e["dur"]
        out[st] = {"kernel": e["kernel"], "calls": len(d), "us": sum(d) / len(d), "us_min": min(d), "us_max": max(d),
                   **{c: sum(v) / len(v) for c, v in e["ctr"].items()}}
    return out


def copy_scale(other, copy_bytes, counter):
    """Bytes per counter unit (KiB readings) from the calibration copy, the
    last dispatch outside the library."""
    if not other or counter not in other[-1][1]:
        raise ValueError("no calibration copy in the counter run")
    return copy_bytes / (other[-1][1][counter] * 1024.0)


def profile_tables(w, order_info, trace_dir=None, fetch_dir=None, write_dir=None, pmc_dirs=(), copy_bytes=256 << 20):
    """Per-stage rows for the profile summary of workload `w` (copy_bytes: the
    size of the calibration copy at the end of the FETCH_SIZE / WRITE_SIZE runs)."""
    with_bwd = order_info["pass"] != "forward"
    work = stage_work(w, with_backward=with_bwd)
    rows = {st: {"stage": st} for st in order_info["order"]}
    for st, us in order_info.get("kernel_us", {}).items():
        rows[st]["event_us"] = us
    if trace_dir:
        lab, _ = label_dispatches(_by_dispatch(_read_csvs(trace_dir, "kernel_trace.csv")), order_info)
        for st, e in per_stage(lab).items():
            rows[st].update(kernel=e["kernel"], calls=e["calls"], us=e["us"], us_min=e["us_min"], us_max=e["us_max"])
    scales = {}
    for key, d, ctr in (("fetch", fetch_dir, "FETCH_SIZE"), ("write", write_dir, "WRITE_SIZE")):
        if not d:
            continue
        lab, other = label_dispatches(_by_dispatch(_read_csvs(d, "counter_collection.csv")), order_info)
        scales[key] = sc = copy_scale(other, copy_bytes, ctr)
        for st, e in per_stage(lab).items():
            rows[st][key + "_kib"] = e[ctr]
            rows[st][key + "_bytes"] = e[ctr] * 1024.0 * sc
            rows[st].setdefault("kernel", e["kernel"])
    for d in pmc_dirs:
        lab, _ = label_dispatches(_by_dispatch(_read_csvs(d, "counter_collection.csv")), order_info)
        for st, e in per_stage(lab).items():
            for c, v in e.items():
                if c.startswith(("SQ_", "GRBM_", "TCC_", "TCP_", "TA_", "TD_")):
                    rows[st][c] = v
            rows[st].setdefault("kernel", e["kernel"])
    for st, r in rows.items():
        wk = work.get(st)
        if wk is not None:
            r["alg_bytes"], r["alg_flops"] = wk.bytes, wk.flops
            t = r.get("us")
            if t and (wk.bytes or wk.flops):
                rl = roofline(wk, t / 1e6, w.dtype)
                r["bound"], r["frac"] = rl["bound"], rl["frac"]
        if "fetch_bytes" in r and "write_bytes" in r:
            r["hbm_bytes"] = r["fetch_bytes"] + r["write_bytes"]
        mops = r.get("SQ_INSTS_VALU_MFMA_MOPS_BF16")
        if mops is not None and r.get("us"):
            # one MOPS unit = 512 FLOPs of a bf16 MFMA
            r["mfma_flops"] = 512.0 * mops
            r["mfma_util"] = 512.0 * mops / (r["us"] * 1e-6) / MFMA_PEAK["bf16"]
    return [rows[st] for st in order_info["order"]], scales


def _fmt(v, spec):
    return "" if v is None else format(v, spec)


def profile_markdown(w, order_info, rows, scales, commands):
    """The committed profile summary of one workload (markdown)."""
    out = [f"# Kernel profile: {w.name}, {order_info['pass']}", "",
           f"Workload: B={w.batch}, T={w.seq_len}, d_model={w.d_model}, {w.heads} MoSA heads (k={w.k}) + "
           f"{w.dense_heads} dense heads, d_head={w.d_head}, {w.dtype} storage, fp32 accumulation.  One step = "
           f"{len(order_info['order'])} kernel launches; {order_info['warmup']} warm-up + {order_info['steps']} "
           f"stage-timed steps per run (bench.py --profile).  Kernel sources: paper_2505_00315_amd/csrc, digest "
           f"{order_info.get('source_sha')}.", "", "Commands (repository root, one MI355X):", ""]
    out += ["    " + c for c in commands]
    out += ["", "Columns: `us` = mean kernel duration from the kernel trace (all calls); `event us` = the same "
            "launch timed by bench.py's HIP events (includes the gap to the previous launch); `alg MB` / "
            "`alg GF` = algorithmic bytes / FLOPs per launch (perfmodel.stage_work); `frac` = achieved fraction "
            "of the binding roofline (HBM 8 TB/s or bf16 MFMA 2.5 PFLOP/s) at `us`; `HBM MB` = FETCH_SIZE + "
            "WRITE_SIZE per dispatch scaled by a plain copy of known size"
            + (f" (fetch x{scales['fetch']:.3f}, write x{scales['write']:.3f})" if len(scales) == 2 else "")
            + "; `HBM/alg` their ratio; `MFMA %` = 512 x SQ_INSTS_VALU_MFMA_MOPS_BF16 / `us` / 2.5 PFLOP/s; "
            "`clk GHz` = SQ_BUSY_CYCLES / 32 shader engines / `us`, the clock the kernel ran at; `MFMA busy %` = "
            "SQ_VALU_MFMA_BUSY_CYCLES (summed over the 1024 SIMDs) / (1024 x SQ_BUSY_CYCLES / 32), the share of "
            "the SIMDs' cycles at that clock with the matrix core busy; "
            "`wait %` = SQ_WAIT_ANY / SQ_WAVE_CYCLES; `LDS conf %` = SQ_LDS_BANK_CONFLICT / SQ_LDS_IDX_ACTIVE.",
            "", "| stage | kernel | calls | us | event us | alg MB | alg GF | bound | frac | HBM MB | HBM/alg | "
            "MFMA % | clk GHz | MFMA busy % | wait % | LDS conf % |",
            "|---|---|---:|---:|---:|---:|---:|---|---:|---:|---:|---:|---:|---:|---:|---:|"]
    total = 0.0
    for r in rows:
        total += r.get("us", 0.0)
        ratio = r["hbm_bytes"] / r["alg_bytes"] if r.get("hbm_bytes") and r.get("alg_bytes") else None
        wait = (100.0 * r["SQ_WAIT_ANY"] / r["SQ_WAVE_CYCLES"]) if r.get("SQ_WAVE_CYCLES") else None
        conf = (100.0 * r["SQ_LDS_BANK_CONFLICT"] / r["SQ_LDS_IDX_ACTIVE"]) if r.get("SQ_LDS_IDX_ACTIVE") else None
        clk = r["SQ_BUSY_CYCLES"] / SHADER_ENGINES / (r["us"] * 1e3) if r.get("SQ_BUSY_CYCLES") and r.get("us") else None
        busy = (100.0 * r["SQ_VALU_MFMA_BUSY_CYCLES"] * SHADER_ENGINES / (SIMDS * r["SQ_BUSY_CYCLES"])
                if r.get("SQ_BUSY_CYCLES") and r.get("SQ_VALU_MFMA_BUSY_CYCLES") is not None else None)
        kern = r.get("kernel", "")
        if len(kern) > 60:
            kern = kern[:57] + "..."
        out.append("| " + " | ".join([
            r["stage"], f"`{kern}`", str(r.get("calls", "")), _fmt(r.get("us"), ".2f"), _fmt(r.get("event_us"), ".2f"),
            _fmt(r.get("alg_bytes", 0) / 1e6 if r.get("alg_bytes") is not None else None, ".2f"),
            _fmt(r.get("alg_flops", 0) / 1e9 if r.get("alg_flops") is not None else None, ".2f"),
            r.get("bound", ""), _fmt(r.get("frac"), ".3f"),
            _fmt(r["hbm_bytes"] / 1e6 if r.get("hbm_bytes") is not None else None, ".2f"), _fmt(ratio, ".2f"),
            _fmt(100.0 * r["mfma_util"] if r.get("mfma_util") is not None else None, ".1f"), _fmt(clk, ".2f"),
            _fmt(busy, ".1f"), _fmt(wait, ".0f"),
            _fmt(conf, ".1f")]) + " |")
    out += ["", f"Sum of the mean kernel durations of one step: {total:.1f} us."]
    return "\n".join(out) + "\n"


def traffic_lines(w, rows, source, source_sha):
    """Machine-readable HBM traffic per launch (read by bench.py's roofline)."""
    lines = []
    for r in rows:
        if r.get("hbm_bytes") is None:
            continue
        lines.append(f"stage={r['stage']} workload={w.name} source={source} source_sha={source_sha} "
                     f"fetch_kib={r['fetch_kib']:.1f} write_kib={r['write_kib']:.1f} "
                     f"hbm_bytes_per_launch={r['hbm_bytes']:.0f}")
    return lines


def main(argv=None):
    import argparse
    import json
    import os

    import workloads as wl

    ap = argparse.ArgumentParser(description="write the per-kernel profile summary of one workload from "
                                             "rocprofv3 runs of bench.py --profile")
    ap.add_argument("--order", required=True, help="the --order-file of the runs")
    ap.add_argument("--trace", help="output directory of the --kernel-trace run")
    ap.add_argument("--fetch", help="output directory of the FETCH_SIZE run")
    ap.add_argument("--write", help="output directory of the WRITE_SIZE run")
    ap.add_argument("--pmc", action="append", default=[], help="output directories of other counter runs")
    ap.add_argument("--copy-bytes", type=int, default=256 << 20, help="calibration copy of the counter runs")
    ap.add_argument("--command", action="append", default=[], help="commands that produced the runs")
    ap.add_argument("--markdown", required=True, help="summary file to write")
    ap.add_argument("--traffic", help="counter file to update (lines of this workload replaced)")
    a = ap.parse_args(argv)
    info = json.load(open(a.order))
    w = wl.WORKLOADS[info["workload"]]
    rows, scales = profile_tables(w, info, a.trace, a.fetch, a.write, a.pmc, a.copy_bytes)
    with open(a.markdown, "w") as f:
        f.write(profile_markdown(w, info, rows, scales, a.command))
    if a.traffic and a.fetch and a.write:
        keep = []
        if os.path.exists(a.traffic):
            keep = [ln.rstrip("\n") for ln in open(a.traffic)
                    if not ln.startswith("#") and f"workload={w.name} " not in ln and ln.strip()]
        head = ["# HBM bytes per launch: rocprofv3 FETCH_SIZE + WRITE_SIZE (KiB per dispatch, one run each) of "
                "bench.py --profile --calibrate-copy 256, scaled by the readings of the plain copy of known size "
                "at the end of the same run; written by perfmodel.py from the runs listed in the profile summaries."]
        lines = traffic_lines(w, rows, "paper_2505_00315_amd/csrc", info.get("source_sha"))
        with open(a.traffic, "w") as f:
            f.write("\n".join(head + keep + lines) + "\n")


if __name__ == "__main__":
    main()
