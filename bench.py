"""Benchmark of the MoSA layer hot path on one MI355X.

One step = one forward and one backward of the layer (router, certified
top-k, gather + QKV projection, attention among the selected tokens,
router-scaled output projection with the deterministic scatter-add, and the
whole backward including the router gradient) over one batch of seeded
synthetic inputs that are resident in HBM before timing starts.

Prints ONE JSON line: whole-step tokens/s (K uninstrumented steps), per-stage
times measured live with HIP events recorded by the library on the stream the
kernels run on (K further steps in the same process), the roofline of the
dominant stage, and the CPU oracle timed on a bounded sample of the same
workload.
"""
import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import perfmodel as pm  # noqa: E402
import workloads as wl  # noqa: E402

METRIC = "MoSA layer tokens/sec fwd & fwd+bwd at T=1024; % HBM GB/s and % MFMA peak"
COUNTERS_FILE = os.path.join(ROOT, "profiles", "hbm_traffic_counters.txt")


def parse_args():
    p = argparse.ArgumentParser(description=__doc__)
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--workload", default="fwd_d512", choices=sorted(wl.WORKLOADS))
    p.add_argument("--fwd-only", action="store_true", help="time the forward pass only")
    p.add_argument("--cpu-seconds", type=float, default=15.0, help="target length of the oracle sample")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-stage-events", action="store_true",
                   help="time whole steps only (no per-stage events inside the timed region)")
    p.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                   help="after the timed steps, copy MIB MiB device to device once (a plain copy kernel of known "
                        "size whose counter readings calibrate the HBM traffic counters)")
    return p.parse_args()


def source_digest(rel):
    """sha256[:16] of a source file, or of every file of a directory in name
    order (any change to the kernels' sources invalidates their counters)."""
    path = os.path.join(ROOT, rel)
    h = hashlib.sha256()
    if os.path.isdir(path):
        for name in sorted(os.listdir(path)):
            f = os.path.join(path, name)
            if os.path.isfile(f):
                h.update(name.encode())
                h.update(open(f, "rb").read())
    elif os.path.exists(path):
        h.update(open(path, "rb").read())
    else:
        return None
    return h.hexdigest()[:16]


class HipEvents:
    """hipEvent_t handles created through the HIP runtime (for the library's
    timed entry points)."""

    def __init__(self, n):
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.handles = []
        for _ in range(n):
            h = ctypes.c_void_p()
            if self.hip.hipEventCreate(ctypes.byref(h)) != 0:
                raise RuntimeError("hipEventCreate failed")
            self.handles.append(h.value)

    def elapsed_ms(self, a, b):
        out = ctypes.c_float()
        if self.hip.hipEventElapsedTime(ctypes.byref(out), ctypes.c_void_p(a), ctypes.c_void_p(b)) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return out.value

    def close(self):
        for h in self.handles:
            self.hip.hipEventDestroy(ctypes.c_void_p(h))


def traffic_for(kernel, w):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter
    summary, or None when there is none for this workload or the kernel's
    source changed since the counters were taken."""
    if not os.path.exists(COUNTERS_FILE):
        return None
    for line in open(COUNTERS_FILE):
        if line.startswith("#") or not line.strip():
            continue
        f = dict(kv.split("=", 1) for kv in line.split())
        if f.get("stage") != kernel or f.get("workload") != w.name:
            continue
        if source_digest(f["source"]) != f["source_sha"]:
            return None
        return float(f["hbm_bytes_per_launch"])
    return None


def cpu_baseline(w, inp, with_backward, target_s):
    """The oracle as it stands, on the host cores, over the first batch
    elements of the same workload (whole layer for those elements)."""
    import numpy as np

    import oracle

    def run(nb):
        sub = dict(inp)
        sub["X"] = np.ascontiguousarray(inp["X"][:nb])
        t0 = time.perf_counter()
        oracle.forward(sub, w.k, causal=w.causal, opts=oracle.options(**w.variants()))
        if with_backward:
            oracle.backward(sub, np.ascontiguousarray(inp["dY"][:nb]), w.k, causal=w.causal,
                            opts=oracle.options(**w.variants()))
        return time.perf_counter() - t0

    t1 = run(1)
    nb = max(1, min(w.batch, int(target_s / max(t1, 1e-3))))
    reps, t = 0, 0.0
    while True:  # whole passes over the sample until about target_s of CPU work
        t += run(nb)
        reps += 1
        if t >= 0.5 * target_s or reps * nb * t1 >= 4 * target_s:
            break
    return {"value": reps * nb * w.seq_len / t, "unit": "tokens/s", "cores": oracle.max_threads(), "kind": "oracle",
            "sample": f"{reps} x {nb} of {w.batch} batch elements of {w.name} (all {w.heads} MoSA + "
                      f"{w.dense_heads} dense heads), {'forward+backward' if with_backward else 'forward'}, "
                      f"fp64 CPU oracle, {t:.1f} s"}


def time_comparator(w, steps, warmup, with_bwd):
    """Whole steps of the comparator workload on the same GPU and stream
    (inputs resident, no instrumentation inside the timed region)."""
    import numpy as np
    import torch

    from paper_2505_00315_amd import mosa

    inp = wl.make_inputs(w, with_grad=with_bwd)

    def dev(a):
        if a is None:
            return None
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16).cuda()
        return torch.from_numpy(a).cuda()

    d = {n: dev(v) for n, v in inp.items()}
    shape = mosa.make_shape(w.batch, w.seq_len, w.d_model, w.heads, w.d_head, w.k, w.causal, w.dense_heads, w.dtype,
                            **w.variants())
    weights = {n: d.get(n) for n in mosa.WEIGHT_NAMES}
    saved, scratch = mosa.alloc_workspace(shape)
    Y, dX = torch.empty_like(d["X"]), torch.empty_like(d["X"])
    grads = {"d" + n: torch.empty_like(d[n]) for n in mosa.WEIGHT_NAMES if d.get(n) is not None and d[n].numel()}
    stream = torch.cuda.current_stream()

    def step():
        mosa.forward(shape, d["X"], weights, Y=Y, saved=saved, scratch=scratch, stream=stream)
        if with_bwd:
            mosa.backward(shape, d["X"], weights, d["dY"], saved, grads, dX=dX, scratch=scratch, stream=stream)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for _ in range(steps):
        step()
    stop.record(stream)
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / steps
    return {"workload": w.name, "dense_heads": w.dense_heads, "mosa_heads": w.heads, "seq_len": w.seq_len,
            "pass": "forward+backward" if with_bwd else "forward", "ms_per_step": ms,
            "tokens_per_s": w.batch * w.seq_len / (ms / 1e3)}


def main():
    args = parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the layer's hot path runs on a single MI355X and no multi-GPU path "
              f"is built (asked for --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    from paper_2505_00315_amd import mosa

    w = wl.WORKLOADS[args.workload]
    with_bwd = not args.fwd_only
    inp = wl.make_inputs(w, with_grad=with_bwd)
    torch.cuda.set_device(0)

    def dev(a):
        if a is None:
            return None
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16).cuda()
        return torch.from_numpy(a).cuda()

    d = {n: dev(v) for n, v in inp.items()}
    shape = mosa.make_shape(w.batch, w.seq_len, w.d_model, w.heads, w.d_head, w.k, w.causal, w.dense_heads, w.dtype,
                            **w.variants())
    weights = {n: d.get(n) for n in mosa.WEIGHT_NAMES}
    saved, scratch = mosa.alloc_workspace(shape)
    Y = torch.empty_like(d["X"])
    dX = torch.empty_like(d["X"])
    grads = {"d" + n: torch.empty_like(d[n]) for n in mosa.WEIGHT_NAMES if d.get(n) is not None and d[n].numel()}
    stream = torch.cuda.current_stream()

    # one set of stage events per timed step, so that the host never waits
    # inside the timed region
    nsets = args.steps
    ev = HipEvents(2 * mosa.MAX_STAGES * nsets)
    sets = []
    for sidx in range(nsets):
        fe, be = mosa.StageEvents(), mosa.StageEvents()
        base = 2 * mosa.MAX_STAGES * sidx
        for i in range(mosa.MAX_STAGES):
            fe.events[i] = ev.handles[base + i]
            be.events[i] = ev.handles[base + mosa.MAX_STAGES + i]
        sets.append((fe, be))

    def step(evs):
        mosa.forward(shape, d["X"], weights, Y=Y, saved=saved, scratch=scratch, stream=stream,
                     events=evs[0] if evs else None)
        if with_bwd:
            mosa.backward(shape, d["X"], weights, d["dY"], saved, grads, dX=dX, scratch=scratch, stream=stream,
                          events=evs[1] if evs else None)

    for _ in range(args.warmup):
        step(None)
    torch.cuda.synchronize()

    # Headline: K whole steps with no instrumentation inside the timed region
    # (a HIP event per stage costs a few microseconds of dispatch each).
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for _ in range(args.steps):
        step(None)
    stop.record(stream)
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(stop)
    ms_per_step = total_ms / args.steps

    # Stage breakdown: K more steps with the library's per-stage HIP events,
    # recorded on the stream the kernels run on.
    if not args.no_stage_events:
        for sidx in range(args.steps):
            step(sets[sidx])
        torch.cuda.synchronize()

    stage_ms, fwd_ms_total = {}, 0.0
    for fe, be in ([] if args.no_stage_events else sets):
        for evs in ((fe, be) if with_bwd else (fe,)):
            for j in range(1, evs.count):
                name = evs.names[j].decode()
                stage_ms[name] = stage_ms.get(name, 0.0) + ev.elapsed_ms(evs.events[j - 1], evs.events[j])
        fwd_ms_total += ev.elapsed_ms(fe.events[0], fe.events[fe.count - 1])
    stage_ms = {n: v / args.steps for n, v in stage_ms.items()}
    fwd_ms = fwd_ms_total / args.steps
    ev.close()

    tokens = w.batch * w.seq_len
    work = pm.stage_work(w, with_backward=with_bwd)
    stage_times = pm.group_stage_times(stage_ms)
    stages = {}
    for n, ms in stage_times.items():
        rl = pm.roofline(work[n], ms / 1e3, w.dtype)
        stages[n] = {"us": round(ms * 1e3, 2), "bound": rl["bound"], "frac": round(rl["frac"], 4)}
        members = pm.GROUPS.get(n)
        if members:
            stages[n]["kernels_us"] = {m: round(stage_ms[m] * 1e3, 2) for m in members if m in stage_ms}
    roof = None
    if stage_times:
        dom = max(stage_times, key=stage_times.get)
        rl = pm.roofline(work[dom], stage_times[dom] / 1e3, w.dtype)
        traffic = traffic_for(dom, w)
        roof = {"bound": rl["bound"], "achieved": round(rl["achieved"], 2), "peak": rl["peak"], "unit": rl["unit"],
                "frac": round(rl["frac"], 4), "traffic": traffic, "kernel": dom,
                "kernels": list(pm.GROUPS.get(dom, (dom,))),
                "algorithmic_bytes": work[dom].bytes, "algorithmic_flops": work[dom].flops,
                "kernel_us": round(stage_times[dom] * 1e3, 2)}

    line = {
        "metric": METRIC,
        "value": tokens / (ms_per_step / 1e3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded N(0,1) activations, N(0,1/d) weights)",
        "config": {"workload": w.name, "pass": "forward+backward" if with_bwd else "forward",
                   "batch": w.batch, "seq_len": w.seq_len, "d_model": w.d_model, "mosa_heads": w.heads,
                   "dense_heads": w.dense_heads, "d_head": w.d_head, "k": w.k, "causal": w.causal},
        "fwd_tokens_per_s": tokens / (fwd_ms / 1e3) if fwd_ms > 0 else None,
        "fwd_ms": fwd_ms,
        "stages": stages,
        "roofline": roof,
    }
    comp = wl.COMPARATORS.get(w.name)
    if comp:
        cw = wl.WORKLOADS[comp]
        line["comparator"] = time_comparator(cw, args.steps, args.warmup, with_bwd)
        # the paper's FLOP formula (Appendix A) for the two layers, one sequence
        line["comparator"]["paper_gflops"] = {
            w.name: round(w.heads * pm.paper_flops_mosa_head(w.d_model, w.d_head, w.seq_len, w.k) / 1e9, 2),
            cw.name: round(cw.dense_heads * pm.paper_flops_dense_head(cw.d_model, cw.d_head, cw.seq_len) / 1e9, 2)}
    if args.calibrate_copy > 0:
        nel = args.calibrate_copy * (1 << 20) // 4
        src_t = torch.ones(nel, dtype=torch.float32, device="cuda")
        dst_t = torch.empty_like(src_t)
        torch.cuda.synchronize()
        dst_t.copy_(src_t)
        torch.cuda.synchronize()
        line["copy_calibration_bytes"] = nel * 4
        del src_t, dst_t
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(w, inp, with_bwd, args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
