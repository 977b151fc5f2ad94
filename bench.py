"""Benchmark of the MoSA layer hot path on one MI355X.

One step = one forward and one backward of the layer (router, certified
top-k, gather + QKV projection, attention among the selected tokens,
router-scaled output projection with the deterministic head-ordered sum, and
the whole backward including the router gradient; the hybrid workload adds its
dense causal heads) over one batch of seeded synthetic inputs that are
resident in HBM before timing starts.

Default workload: hybrid_d1024 (B=8, T=1024, d_model=1024, 4 dense + 256 MoSA
heads, d_head=64, k=16), forward+backward, the largest T=1024 configuration
the metric is quoted on that is timed with its backward.

Timing (all on the stream the kernels run on, nothing else inside the timed
regions):
  cold  K steps cycling over R copies of every buffer of a step (inputs,
        weights, outputs, gradients, saved state, scratch) spanning at least
        --cold-mib MiB between two uses of the same copy, so the L2 caches and
        the 256 MB Infinity Cache hold none of a step's data when it starts;
        this is the headline `value`;
  warm  K steps on one copy (the working set may stay in the caches);
  stages K further cold steps through the library's timed entry points, which
        launch exactly the same kernels and record a HIP event after every
        launch: per-kernel durations and the roofline of the longest launch.
Extra lines in the same JSON object: the forward-only workload fwd_d512
(B=8, T=1024, d=512, 32 heads, k=128) and the fwdbwd_d1024 forward+backward
workload (B=4, d=1024, 128 heads, k=64), cold and warm, and the CPU oracle
timed on a bounded sample of the default workload (all host cores and one).
"""
import argparse
import hashlib
import json
import os
import platform
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import perfmodel as pm  # noqa: E402
import workloads as wl  # noqa: E402

METRIC = "MoSA layer tokens/sec fwd & fwd+bwd at T=1024; % HBM GB/s and % MFMA peak"
COUNTERS_FILE = os.path.join(ROOT, "profiles", "hbm_traffic_counters.txt")
DEFAULT_WORKLOAD = "hybrid_d1024"
EXTRA = (("fwd_d512", False), ("fwdbwd_d1024", True))


def parse_args(argv=None):
    p = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--workload", default=DEFAULT_WORKLOAD, choices=sorted(wl.WORKLOADS))
    p.add_argument("--fwd-only", action="store_true", help="time the forward pass only")
    p.add_argument("--cold-mib", type=int, default=512,
                   help="bytes touched between two uses of the same buffer copy in the cold runs")
    p.add_argument("--cpu-seconds", type=float, default=15.0, help="target length of the all-core oracle sample")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-extra", action="store_true", help="skip the fwd_d512 and fwdbwd_d1024 lines")
    p.add_argument("--no-stage-events", action="store_true", help="skip the per-kernel (timed entry point) steps")
    p.add_argument("--profile", action="store_true",
                   help="for rocprofv3: only W warm-up and K stage-timed steps of one copy of the workload, "
                        "then the optional calibration copy; the kernel order of one step goes to --order-file")
    p.add_argument("--order-file", default=None, help="with --profile: write the kernel order of a step here")
    p.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                   help="at the end, copy MIB MiB device to device once (a plain copy of known size whose "
                        "counter readings calibrate the HBM traffic counters)")
    return p.parse_args(argv)


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


def traffic_for(kernel, w):
    """HBM bytes per launch of the kernel with stage name `kernel` from the
    committed rocprofv3 counter summary, or None when there is none for this
    workload or the kernels' sources changed since the counters were taken."""
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


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def cpu_baseline(w, inp, with_backward, target_s):
    """The oracle as it stands, on the host cores, over the first batch
    elements of the same workload (the whole layer for those elements): all
    cores on a sample of about target_s seconds, and one thread on one batch
    element."""
    import numpy as np

    import oracle

    opts = oracle.options(**w.variants())

    def run(nb):
        sub = dict(inp)
        sub["X"] = np.ascontiguousarray(inp["X"][:nb])
        t0 = time.perf_counter()
        oracle.forward(sub, w.k, causal=w.causal, opts=opts)
        if with_backward:
            oracle.backward(sub, np.ascontiguousarray(inp["dY"][:nb]), w.k, causal=w.causal, opts=opts)
        return time.perf_counter() - t0

    cores = oracle.max_threads()
    t1 = run(1)
    nb = max(1, min(w.batch, int(target_s / max(t1, 1e-3))))
    reps, t = 0, 0.0
    while True:  # whole passes over the sample until about target_s of CPU work
        t += run(nb)
        reps += 1
        if t >= 0.5 * target_s or reps * nb * t1 >= 4 * target_s:
            break
    oracle.set_threads(1)
    try:
        t_one = run(1)
    finally:
        oracle.set_threads(cores)
    what = (f"all {w.heads} MoSA + {w.dense_heads} dense heads, "
            f"{'forward+backward' if with_backward else 'forward'}, fp64 CPU oracle")
    return {"value": reps * nb * w.seq_len / t, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "sample": f"{reps} x {nb} of {w.batch} batch elements of {w.name} ({what}), {t:.1f} s",
            "single_thread": {"value": w.seq_len / t_one, "unit": "tokens/s", "cores": 1,
                              "sample": f"1 batch element of {w.name} ({what}), {t_one:.1f} s"},
            "cpu_model": cpu_model()}


class Runner:
    """R copies of every buffer one step of workload `w` touches, and the
    step itself on one copy (optionally through the timed entry points)."""

    def __init__(self, w, with_bwd, copies=1):
        import numpy as np
        import torch

        from paper_2505_00315_amd import mosa

        self.torch, self.mosa, self.w, self.with_bwd = torch, mosa, w, with_bwd
        self.inp = wl.make_inputs(w, with_grad=with_bwd)

        def dev(a):
            if a is None:
                return None
            if a.dtype == np.uint16:
                return torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16).cuda()
            return torch.from_numpy(a).cuda()

        base = {n: dev(v) for n, v in self.inp.items()}
        self.shape = mosa.make_shape(w.batch, w.seq_len, w.d_model, w.heads, w.d_head, w.k, w.causal,
                                     w.dense_heads, w.dtype, **w.variants())
        self.stream = torch.cuda.current_stream()
        self.sets = []
        for c in range(copies):
            d = base if c == 0 else {n: (t.clone() if t is not None else None) for n, t in base.items()}
            saved, scratch = mosa.alloc_workspace(self.shape)
            s = {"d": d, "w": {n: d.get(n) for n in mosa.WEIGHT_NAMES}, "saved": saved, "scratch": scratch,
                 "Y": torch.empty_like(d["X"])}
            if with_bwd:
                s["dX"] = torch.empty_like(d["X"])
                s["g"] = {"d" + n: torch.empty_like(d[n]) for n in mosa.WEIGHT_NAMES
                          if d.get(n) is not None and d[n].numel()}
            self.sets.append(s)
        torch.cuda.synchronize()

    def set_bytes(self):
        s = self.sets[0]
        ts = [t for t in s["d"].values() if t is not None] + [s["saved"], s["scratch"], s["Y"]]
        if self.with_bwd:
            ts += [s["dX"]] + list(s["g"].values())
        return sum(t.numel() * t.element_size() for t in ts)

    def step(self, c=0, events=None):
        s, m = self.sets[c], self.mosa
        m.forward(self.shape, s["d"]["X"], s["w"], Y=s["Y"], saved=s["saved"], scratch=s["scratch"],
                  stream=self.stream, events=events[0] if events else None)
        if self.with_bwd:
            m.backward(self.shape, s["d"]["X"], s["w"], s["d"]["dY"], s["saved"], s["g"], dX=s["dX"],
                       scratch=s["scratch"], stream=self.stream, events=events[1] if events else None)

    def check(self):
        """Every copy's selection certified (the forward's status array)."""
        for s in self.sets:
            self.mosa.check_selection(self.shape, s["saved"])

    def timed(self, steps, cycle):
        """K steps over the copies in `cycle` order, one event pair around the
        whole run and one event between steps (recorded on the stream, read
        after the final synchronisation).  Returns (ms per step, median ms)."""
        torch = self.torch
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
        torch.cuda.synchronize()
        ev[0].record(self.stream)
        for i in range(steps):
            self.step(cycle[i % len(cycle)])
            ev[i + 1].record(self.stream)
        torch.cuda.synchronize()
        per = [ev[i].elapsed_time(ev[i + 1]) for i in range(steps)]
        return ev[0].elapsed_time(ev[steps]) / steps, statistics.median(per)


def copies_for(runner_bytes, cold_bytes):
    """Copies such that the other copies span at least cold_bytes."""
    return max(2, 1 + -(-cold_bytes // max(runner_bytes, 1)))


def measure(w, with_bwd, steps, warmup, cold_mib):
    """Cold and warm whole-step times of workload `w`."""
    probe = Runner(w, with_bwd, copies=1)
    n = copies_for(probe.set_bytes(), cold_mib << 20)
    del probe
    r = Runner(w, with_bwd, copies=n)
    for i in range(max(warmup, n)):
        r.step(i % n)
    r.torch.cuda.synchronize()
    r.check()
    cold, cold_med = r.timed(steps, list(range(n)))
    warm, warm_med = r.timed(steps, [0])
    return r, n, {"ms_per_step": cold, "median_ms": cold_med, "warm_ms_per_step": warm, "warm_median_ms": warm_med}


def stage_times(r, steps, cycle):
    """K steps through the timed entry points (an event after every launch);
    mean ms per kernel stage (stage names are unique within a step)."""
    mosa = r.mosa
    timer = mosa.StageTimer(sets=2 * steps)
    try:
        for i in range(steps):
            r.step(cycle[i % len(cycle)], events=(timer.sets[2 * i], timer.sets[2 * i + 1]))
        r.torch.cuda.synchronize()
        acc, order = {}, []
        for i in range(steps):
            for evs in (timer.sets[2 * i], timer.sets[2 * i + 1]) if r.with_bwd else (timer.sets[2 * i],):
                for name, ms in timer.stages(evs):
                    acc.setdefault(name, []).append(ms)
                    if i == 0:
                        order.append(name)
    finally:
        timer.close()
    return {n: sum(v) / len(v) for n, v in acc.items()}, order


def roofline_line(w, with_bwd, kernel_ms):
    """Roofline of the longest single-kernel stage from its event time."""
    work = pm.stage_work(w, with_backward=with_bwd)
    timed = {n: ms for n, ms in kernel_ms.items() if n in work}
    dom = max(timed, key=timed.get)
    rl = pm.roofline(work[dom], timed[dom] / 1e3, w.dtype)
    return {"bound": rl["bound"], "achieved": round(rl["achieved"], 2), "peak": rl["peak"], "unit": rl["unit"],
            "frac": round(rl["frac"], 4), "traffic": traffic_for(dom, w), "kernel": dom,
            "kernel_us": round(timed[dom] * 1e3, 2), "algorithmic_bytes": work[dom].bytes,
            "algorithmic_flops": work[dom].flops, "ai": round(rl["ai"], 1)}


def stage_table(w, with_bwd, kernel_ms):
    work = pm.stage_work(w, with_backward=with_bwd)
    out = {}
    for n, ms in kernel_ms.items():
        e = {"us": round(ms * 1e3, 2)}
        if n in work and (work[n].bytes or work[n].flops):
            rl = pm.roofline(work[n], ms / 1e3, w.dtype)
            e.update(bound=rl["bound"], frac=round(rl["frac"], 4))
        out[n] = e
    for g, members in pm.GROUPS.items():  # two-kernel operations of the paper
        if g in work and any(m in kernel_ms for m in members):
            t = sum(kernel_ms.get(m, 0.0) for m in members)
            rl = pm.roofline(work[g], t / 1e3, w.dtype)
            out[g] = {"us": round(t * 1e3, 2), "bound": rl["bound"], "frac": round(rl["frac"], 4),
                      "kernels": [m for m in members if m in kernel_ms]}
    return out


def profile_mode(args, w, with_bwd):
    """Warm-up and stage-timed steps of one copy only (for rocprofv3): one
    step's kernel order goes to --order-file."""
    import torch

    r = Runner(w, with_bwd, copies=1)
    for _ in range(args.warmup):
        r.step(0)
    torch.cuda.synchronize()
    r.check()
    kernel_ms, order = stage_times(r, args.steps, [0])
    if args.order_file:
        os.makedirs(os.path.dirname(os.path.abspath(args.order_file)), exist_ok=True)
        with open(args.order_file, "w") as f:
            json.dump({"workload": w.name, "pass": "forward+backward" if with_bwd else "forward",
                       "warmup": args.warmup, "steps": args.steps, "order": order,
                       "calibrate_copy_bytes": (args.calibrate_copy << 20) if args.calibrate_copy else 0,
                       "kernel_us": {n: round(ms * 1e3, 3) for n, ms in kernel_ms.items()},
                       "source_sha": source_digest("paper_2505_00315_amd/csrc")}, f, indent=1)
    return kernel_ms


def calibrate_copy(mib):
    import torch

    nel = mib * (1 << 20) // 4
    src = torch.ones(nel, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    return nel * 4


def main(argv=None):
    args = parse_args(argv)
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the layer's hot path runs on a single MI355X and no multi-GPU path "
              f"is built (asked for --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)
    import torch

    torch.cuda.set_device(0)
    w = wl.WORKLOADS[args.workload]
    with_bwd = not args.fwd_only
    if args.profile:
        kernel_ms = profile_mode(args, w, with_bwd)
        line = {"profile": w.name, "steps": args.steps, "warmup": args.warmup,
                "kernel_us": {n: round(ms * 1e3, 2) for n, ms in kernel_ms.items()}}
        if args.calibrate_copy > 0:
            line["copy_calibration_bytes"] = calibrate_copy(args.calibrate_copy)
        print(json.dumps(line), flush=True)
        return

    tokens = w.batch * w.seq_len
    r, ncopies, t = measure(w, with_bwd, args.steps, args.warmup, args.cold_mib)
    print(f"[bench] {w.name}: cold {t['ms_per_step']:.4f} ms/step over {ncopies} copies, "
          f"warm {t['warm_ms_per_step']:.4f}", file=sys.stderr, flush=True)
    line = {
        "metric": METRIC,
        "value": tokens / (t["ms_per_step"] / 1e3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": t["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded N(0,1) activations, N(0,1/d) weights and upstream gradient)",
        "config": {"workload": w.name, "pass": "forward+backward" if with_bwd else "forward",
                   "batch": w.batch, "seq_len": w.seq_len, "d_model": w.d_model, "mosa_heads": w.heads,
                   "dense_heads": w.dense_heads, "d_head": w.d_head, "k": w.k, "causal": w.causal,
                   "timing": f"cold: {ncopies} copies of every buffer of a step (>= {args.cold_mib} MiB between "
                             f"uses of a copy); warm: one copy"},
        "median_ms": t["median_ms"],
        "warm": {"ms_per_step": t["warm_ms_per_step"], "median_ms": t["warm_median_ms"],
                 "tokens_per_s": tokens / (t["warm_ms_per_step"] / 1e3)},
    }
    if not args.no_stage_events:
        kernel_ms, order = stage_times(r, args.steps, list(range(ncopies)))
        line["kernels_us"] = stage_table(w, with_bwd, kernel_ms)
        line["kernel_order"] = order
        line["roofline"] = roofline_line(w, with_bwd, kernel_ms)
    del r
    torch.cuda.empty_cache()
    if not args.no_extra:
        for name, bwd in EXTRA:
            if name == w.name and bwd == with_bwd:
                continue
            ew = wl.WORKLOADS[name]
            er, en, et = measure(ew, bwd, args.steps, args.warmup, args.cold_mib)
            del er
            torch.cuda.empty_cache()
            toks = ew.batch * ew.seq_len
            line[name + ("_fwdbwd" if bwd else "_fwd")] = {
                "pass": "forward+backward" if bwd else "forward", "copies": en,
                "ms_per_step": et["ms_per_step"], "tokens_per_s": toks / (et["ms_per_step"] / 1e3),
                "median_ms": et["median_ms"], "warm_ms_per_step": et["warm_ms_per_step"],
                "warm_tokens_per_s": toks / (et["warm_ms_per_step"] / 1e3)}
            print(f"[bench] {name}: cold {et['ms_per_step']:.4f} ms/step", file=sys.stderr, flush=True)
    comp = wl.COMPARATORS.get(w.name)
    if comp:
        cw = wl.WORKLOADS[comp]
        cr, cn, ct = measure(cw, with_bwd, args.steps, args.warmup, args.cold_mib)
        del cr
        line["comparator"] = {"workload": cw.name, "pass": "forward+backward" if with_bwd else "forward",
                              "ms_per_step": ct["ms_per_step"], "warm_ms_per_step": ct["warm_ms_per_step"],
                              "tokens_per_s": cw.batch * cw.seq_len / (ct["ms_per_step"] / 1e3),
                              "paper_gflops": {
                                  w.name: round(w.heads * pm.paper_flops_mosa_head(w.d_model, w.d_head, w.seq_len,
                                                                                   w.k) / 1e9, 2),
                                  cw.name: round(cw.dense_heads * pm.paper_flops_dense_head(cw.d_model, cw.d_head,
                                                                                            cw.seq_len) / 1e9, 2)}}
    if args.calibrate_copy > 0:
        line["copy_calibration_bytes"] = calibrate_copy(args.calibrate_copy)
    if not args.no_cpu_baseline:
        inp = wl.make_inputs(w, with_grad=with_bwd)
        line["cpu_baseline"] = cpu_baseline(w, inp, with_bwd, args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
