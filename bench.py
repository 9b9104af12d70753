"""Benchmark: grid-point-steps/s of one forward+VJP call at a fixed memory
budget on one MI355X, with the dominant kernels' achieved HBM bandwidth
against the chip's peak and the CPU oracle timed on the host beside it.

One "step" of the benchmark is one adst_vjp call: the forward sweep, the
loss and seed, every recomputation the schedule needs and the reverse sweep,
over one synthetic input already resident in HBM. Throughput is
npoints * T / (time of one call). Per the paper's method (Sec. V-A: warm-up,
then repeated runs with confidence bounds) every call is timed with its own
HIP event pair; the line reports the median call and a distribution-free 95%
confidence interval of the median, and `value` is taken at the median.

The default workload is the largest one that fits one GPU: Allen-Cahn f64 on
1024^3 points, 200 steps, a 64 GB checkpoint budget (7 slots, binomial
schedule, 581 forward steps). The other workloads run after it for a few
calls each and are reported under "workloads".

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--sched S]
                    [--force-tape] [--no-fuse] [--dparams] [--limit LO HI]
                    [--no-extras] [--no-cpu-baseline]
    python bench.py --sweep [--workload NAME] [--steps K] ...
    python bench.py --rocprof-summary KT_DIR [--fetch DIR --write DIR] ...

The second form times the Allen-Cahn workloads across schedules and
budgets (SWEEP below). The third form turns rocprofv3 output (kernel stats, FETCH_SIZE and
WRITE_SIZE counter runs) into the markdown tables kept under profiles/,
with the kernels named as this file and the library name them.
"""
import argparse
import csv
import glob
import hashlib
import json
import math
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "grid-point-steps/s for fwd+VJP at fixed memory budget; achieved HBM GB/s"
HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E
SCHED_NAMES = {0: "auto", 1: "store_all", 2: "uniform", 3: "binomial"}
LOSS_NAMES = {0: "half_sq", 1: "dot_w", 2: "half_sq_diff", 3: "seed"}

# The workloads run after the headline (name, overrides): the small case,
# the 4096^2 Jacobi grid with its tape elided and forced through the
# 10-snapshot budget, the 512^3 Allen-Cahn and the 8192^2 variable-coefficient
# workloads, the in-place kind at the paper's case-study size and at 4096^2.
EXTRAS = [
    ("jacobi2d5_f64_64x64_T10", {}),
    ("jacobi2d5_f64_4096x4096_T100", {}),
    ("jacobi2d5_f64_4096x4096_T100", {"force_tape": True, "sched": 3}),
    ("allencahn3d7_f64_512cube_T50", {}),
    ("vardiff2d9_f32_8192x8192_T200", {}),
    ("gaussseidel2d5_f64_400x400_T100", {}),
    ("gaussseidel2d5_f64_4096x4096_T100", {}),
]
# The budget/schedule sweep (--sweep) of the two Allen-Cahn workloads:
# store-all where the tape fits, two or three binomial budgets and the
# uniform schedule at the workloads' own budget (state: 1 GiB at 512^3,
# 8.6 GB at 1024^3).
SWEEP = [
    ("allencahn3d7_f64_512cube_T50", "store_all", 64 << 30),
    ("allencahn3d7_f64_512cube_T50", "binomial", 3 << 30),
    ("allencahn3d7_f64_512cube_T50", "binomial", 8 << 30),
    ("allencahn3d7_f64_512cube_T50", "uniform", 8 << 30),
    ("allencahn3d7_f64_1024cube_T200", "binomial", 26_000_000_000),
    ("allencahn3d7_f64_1024cube_T200", "binomial", 64_000_000_000),
    ("allencahn3d7_f64_1024cube_T200", "binomial", 130_000_000_000),
    ("allencahn3d7_f64_1024cube_T200", "uniform", 64_000_000_000),
]
# The oracle's sample for the headline: the same kind, precision, step count,
# loss and per-point work on a 128^3 grid (a store-all tape of the full grid,
# 1.7 TB, cannot be held).
CPU_SAMPLE_SHAPE = {"allencahn3d7_f64_1024cube_T200": (128, 128, 128)}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10, help="timed calls")
    ap.add_argument("--warmup", type=int, default=2, help="untimed calls first")
    ap.add_argument("--workload", default=None)
    ap.add_argument("--sched", default=None, choices=list(SCHED_NAMES.values()))
    ap.add_argument("--budget-bytes", type=int, default=None)
    ap.add_argument("--force-tape", action="store_true")
    ap.add_argument("--no-fuse", action="store_true",
                    help="one launch per step (no temporal blocking)")
    ap.add_argument("--dparams", action="store_true",
                    help="also compute the gradients of the scalar step constants")
    ap.add_argument("--limit", type=float, nargs=2, default=None, metavar=("LO", "HI"),
                    help="clamp every step's new values to [LO, HI] (a per-point branch)")
    ap.add_argument("--traced-calls", type=int, default=2,
                    help="calls with per-launch HIP events, for the kernels' average durations")
    ap.add_argument("--no-extras", action="store_true", help="only the chosen workload")
    ap.add_argument("--sweep", action="store_true",
                    help="only the budget/schedule sweep of the Allen-Cahn workloads (one JSON "
                         "line, each entry with its phases' kernels)")
    ap.add_argument("--extra-steps", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target CPU time of the oracle sample")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="after the benchmark, copy a buffer of this size three times with the "
                         "driver's copy and three times with adst_copy (plain copies of known "
                         "size, to scale hardware byte counters)")
    ap.add_argument("--rocprof-summary", default=None, metavar="KT_DIR",
                    help="summarise a rocprofv3 --kernel-trace --stats directory and exit")
    ap.add_argument("--fetch", default=None, help="with --rocprof-summary: FETCH_SIZE run dir")
    ap.add_argument("--write", default=None, help="with --rocprof-summary: WRITE_SIZE run dir")
    ap.add_argument("--title", default="")
    ap.add_argument("--bench-json", default=None,
                    help="with --rocprof-summary: a bench output of the profiled run")
    ap.add_argument("--command", default="", help="with --rocprof-summary: the profiled command")
    ap.add_argument("--out", default=None, help="with --rocprof-summary: markdown file to write")
    return ap.parse_args()


# ------------------------------------------------------------ statistics
def median_ci95(xs):
    """Median and a distribution-free 95% confidence interval of the median
    (order statistics x_(j), x_(n-j+1) with j the largest rank such that
    P(Binomial(n, 1/2) < j) <= 0.025; the whole range when n < 6)."""
    s = sorted(xs)
    n = len(s)
    med = float(np.median(s))
    j, cum = 0, 0.0
    for k in range(n + 1):
        p = math.comb(n, k) / 2.0 ** n
        if cum + p > 0.025:
            break
        cum += p
        j = k + 1
    if j < 1:
        return med, (s[0], s[-1])
    return med, (s[j - 1], s[n - j])


# ------------------------------------------------------------ source hashes
def kernel_source(kernel):
    """The source file holding a kernel (by its library label)."""
    if kernel.startswith("jacobi_march") or kernel.startswith("jacobi_lim_adjoint"):
        return "jacobi_march.hip"
    if kernel.startswith("gs_wave"):
        return "gauss_seidel.hip"
    if ("allencahn" in kernel or kernel.startswith("ac_march")) and os.path.exists(
            os.path.join(ROOT, "paper_2509_02197_amd", "csrc", "allencahn.hip")):
        return "allencahn.hip"
    return "kernels.hip"


def source_sha(kernel):
    """Hash of the code in the source file holding the kernel: // comments
    and whitespace are dropped, so editing a comment keeps the counters."""
    with open(os.path.join(ROOT, "paper_2509_02197_amd", "csrc", kernel_source(kernel))) as fh:
        text = fh.read()
    code = "".join(line.split("//", 1)[0].strip() for line in text.splitlines())
    return hashlib.sha256(code.encode()).hexdigest()[:16]


def traffic_for(workload, kernel):
    """HBM bytes per launch from the committed rocprofv3 counter summary,
    or None when none exists for this kernel's current source."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        table = json.load(f)
    e = table.get(f"{workload}:{kernel}")
    if not e or e.get("src_sha") != source_sha(kernel):
        return None
    return e["bytes_per_launch"]


# ------------------------------------------------------------ GPU legs
def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _roof(workload, k, npts):
    """Roofline entry of one kernel from the library's per-launch events."""
    avg_ms = k["ms_sum"] / k["launches"]
    alg = k["alg_bytes_sum"] / k["launches"]
    achieved = alg / (avg_ms * 1e-3) / 1e9
    return {
        "bound": "hbm", "kernel": k["name"], "phase": k["phase"], "achieved": round(achieved, 1),
        "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
        "traffic": traffic_for(workload, k["name"]), "alg_bytes_per_launch": alg,
        "alg_bytes_per_point": round(alg / npts, 3), "avg_launch_ms": round(avg_ms, 5),
        "min_launch_ms": round(k["ms_min"], 5), "max_launch_ms": round(k["ms_max"], 5),
        "launches_per_call": None,
    }


def run_workload(adst, torch, w, opts, steps, warmup, traced_calls, say, inp=None):
    """Time `steps` adst_vjp calls of workload w (inputs resident in HBM),
    then `traced_calls` more with per-launch events. Returns the result dict
    and the host inputs (for the oracle; pass them back in to skip drawing
    them again)."""
    from paper_2509_02197_amd.workloads import dims_of, make_inputs
    sched = opts.get("sched", w.sched)
    budget = opts.get("budget", w.budget_bytes)
    flags = (adst.ADST_FORCE_TAPE if opts.get("force_tape") else 0) | \
        (adst.ADST_NO_FUSE if opts.get("no_fuse") else 0)
    lim = opts.get("limit")
    want_dp = bool(opts.get("dparams"))
    say(f"# workload {w.name} sched={SCHED_NAMES[sched]} budget={budget} flags={flags}")
    if inp is None:
        inp = make_inputs(w)
    dev = torch.device("cuda:0")
    x0 = torch.from_numpy(inp["x0"]).to(dev)
    K = torch.from_numpy(inp["K"]).to(dev) if inp["K"] is not None else None
    aux = torch.from_numpy(inp["aux"]).to(dev) if inp["aux"] is not None else None
    prob = adst.make_problem(w.kind, w.dtype, dims_of(w.shape), w.params, flags, lim)
    grads = (adst.ADST_GRAD_COEFF if w.want_dK else 0) | (adst.ADST_GRAD_PARAMS if want_dp else 0)
    info = adst.adst_plan(prob, w.steps, budget, sched, grads)
    ws = torch.empty(info.workspace_bytes, dtype=torch.uint8, device=dev)
    dx0 = torch.empty_like(x0)
    dK = torch.empty_like(x0) if w.want_dK else None
    L = torch.empty((), dtype=torch.float64, device=dev)
    dP = torch.empty(2, dtype=torch.float64, device=dev) if want_dp else None
    stream = torch.cuda.current_stream()

    def call(p):
        return adst.adst_vjp(p, x0, K, w.steps, w.loss, aux, budget, sched, dx0, dK, None, L, dP,
                             ws, ws.numel(), stream)

    for _ in range(warmup):
        call(prob)
    torch.cuda.synchronize()

    # ---- timed region: `steps` calls, each between its own pair of events
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for e0, e1 in evs:
        e0.record(stream)
        call(prob)
        e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = [e0.elapsed_time(e1) for e0, e1 in evs]
    med, (lo, hi) = median_ci95(ms)
    pts = w.npoints * w.steps

    # ---- kernel leg: the same call with an event pair around every launch
    tprob = adst.make_problem(w.kind, w.dtype, dims_of(w.shape), w.params,
                              flags | adst.ADST_TRACE, lim)
    acc, kstats = {}, {}
    for _ in range(traced_calls):
        ti = call(tprob)
        for f in ("ms_fwd_sweep", "ms_fwd_recompute", "ms_adj", "ms_seed", "ms_dparams",
                  "ms_total"):
            acc[f] = acc.get(f, 0.0) + getattr(ti, f) / traced_calls
        for k in adst.adst_trace_kernels():
            e = kstats.setdefault(k["name"], dict(k, launches=0, ms_sum=0.0, alg_bytes_sum=0.0,
                                                  ms_min=1e30, ms_max=0.0))
            e["launches"] += k["launches"]
            e["ms_sum"] += k["ms_sum"]
            e["alg_bytes_sum"] += k["alg_bytes_sum"]
            e["ms_min"] = min(e["ms_min"], k["ms_min"])
            e["ms_max"] = max(e["ms_max"], k["ms_max"])
    kl = sorted(kstats.values(), key=lambda k: -k["ms_sum"])
    roof = _roof(w.name, kl[0], w.npoints) if kl else None
    fwd = [k for k in kl if k["phase"] in ("forward sweep", "recomputation")]
    adj = [k for k in kl if k["phase"] == "adjoint"]
    roof_fwd = _roof(w.name, fwd[0], w.npoints) if fwd else None
    roof_adj = _roof(w.name, adj[0], w.npoints) if adj else None
    for r in (roof, roof_fwd, roof_adj):
        if r:
            r["launches_per_call"] = kstats[r["kernel"]]["launches"] / max(traced_calls, 1)
    fwd_ms = sum(k["ms_sum"] for k in fwd) / max(traced_calls, 1)
    adj_ms = sum(k["ms_sum"] for k in adj) / max(traced_calls, 1)
    fwd_b = sum(k["alg_bytes_sum"] for k in fwd) / max(traced_calls, 1)
    adj_b = sum(k["alg_bytes_sum"] for k in adj) / max(traced_calls, 1)
    res = {
        "workload": w.name, "grid": list(w.shape), "T": w.steps,
        "kind": adst.workloads.KIND_NAMES[w.kind],
        "dtype": "f64" if w.dtype == adst.ADST_F64 else "f32",
        "loss": LOSS_NAMES[w.loss], "budget_bytes": budget,
        "schedule": SCHED_NAMES[info.sched] + ("" if info.needs_state else " (tape elided)"),
        "slots": info.slots, "fwd_steps": info.fwd_steps_total,
        "recompute_steps": info.recompute_steps, "fwd_kernels": info.fwd_kernels,
        "adj_kernels": info.adj_kernels,
        "grads": ("dx0,dK" if w.want_dK else "dx0") + (",dparams" if want_dp else ""),
        "force_tape": bool(opts.get("force_tape")), "temporal_blocking": not opts.get("no_fuse"),
        "limiter": lim,
        "calls": steps, "ms_median": round(med, 4), "ms_ci95": [round(lo, 4), round(hi, 4)],
        "ms_mean": round(float(np.mean(ms)), 4), "ms_min": round(min(ms), 4),
        "ms_max": round(max(ms), 4), "wall_ms_per_call": round(1e3 * wall / steps, 4),
        "pt_steps_per_s": pts / (med * 1e-3),
        "hbm_gbps_effective": round(info.alg_bytes / (med * 1e-3) / 1e9, 1),
        "phase_ms": {k: round(v, 4) for k, v in acc.items()},
        "fwd_gbps": round(fwd_b / max(fwd_ms, 1e-9) / 1e6, 1),
        "adj_gbps": round(adj_b / max(adj_ms, 1e-9) / 1e6, 1),
        "roofline": roof, "roofline_fwd": roof_fwd, "roofline_adj": roof_adj,
        "kernels": [{"name": k["name"], "phase": k["phase"],
                     "launches_per_call": k["launches"] / max(traced_calls, 1),
                     "avg_ms": round(k["ms_sum"] / k["launches"], 5),
                     "alg_bytes_per_launch": k["alg_bytes_sum"] / k["launches"],
                     "gbps": round(k["alg_bytes_sum"] / (k["ms_sum"] * 1e-3) / 1e9, 1),
                     "share": round(k["ms_sum"] / max(sum(q["ms_sum"] for q in kl), 1e-9), 4)}
                    for k in kl],
    }
    del x0, K, aux, ws, dx0, dK, L, dP
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return res, inp


def copy_ceiling(adst, torch, state_bytes):
    """Bandwidth of plain device-to-device copies, read + write bytes over the
    event-timed copy: the library's one-shot copy (one 16-byte vector per
    work-item) and the driver's hipMemcpyAsync, at one state's size (at
    128 MiB a pair of buffers fits the 256 MB Infinity Cache) and at 2 GiB."""
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    out = {}
    for key, nbytes in (("state_size", min(state_bytes, 2 << 30)), ("2GiB", 2 << 30)):
        a = torch.empty(nbytes // 8, dtype=torch.float64, device=dev).fill_(1.0)
        b = torch.empty_like(a)
        for name, fn in (("adst_copy", lambda: adst.adst_copy(b, a, nbytes, stream)),
                         ("hipMemcpyAsync", lambda: b.copy_(a))):
            for _ in range(3):
                fn()
            reps = 10
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(reps):
                fn()
            e1.record(stream)
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / reps
            out.setdefault(name, {})[key] = {"bytes": 2 * nbytes, "ms": round(ms, 5),
                                             "GB/s": round(2 * nbytes / (ms * 1e-3) / 1e9, 1)}
        del a, b
    torch.cuda.empty_cache()
    return out


def cpu_baseline(w, target_s, lim=None, want_dp=False):
    """The oracle (single-threaded store-all tape, as it stands) on the
    workload's grid, or on a smaller grid with the same per-point work where
    the full grid's tape cannot be held; for as many leading steps as fit
    about target_s seconds, whole calls repeated when all T steps take less."""
    import oracle
    from paper_2509_02197_amd.workloads import make_inputs
    shape = CPU_SAMPLE_SHAPE.get(w.name, w.shape)
    inp = make_inputs(w, shape)
    x0, K, aux = inp["x0"], inp["K"], inp["aux"]
    n = x0.size
    kw = dict(K=K, loss=w.loss, aux=aux, want_dK=w.want_dK, want_dp=want_dp, lim=lim)
    oracle.vjp(w.kind, x0, steps=1, **kw)  # warm the pages once, then size the sample
    t0 = time.perf_counter()
    oracle.vjp(w.kind, x0, steps=2, **kw)
    one = (time.perf_counter() - t0) / 2
    Ts = int(max(1, min(w.steps, target_s / max(one, 1e-6))))
    reps, dt = 0, 0.0
    while reps == 0 or dt < 0.67 * target_s:
        t0 = time.perf_counter()
        oracle.vjp(w.kind, x0, steps=Ts, **kw)
        dt += time.perf_counter() - t0
        reps += 1
    grid = "x".join(map(str, shape))
    full = "x".join(map(str, w.shape))
    where = (f"full {grid} grid" if shape == tuple(w.shape) else
             f"reduced {grid} grid (same kind, precision, T, loss and per-point work as the "
             f"{full} workload, whose store-all tape cannot be held)")
    return {"value": n * Ts * reps / dt, "unit": "grid-point-steps/s", "cores": 1, "kind": "oracle",
            "sample": f"{where}, first {Ts} of {w.steps} steps, {reps} call(s), store-all tape, "
                      f"single thread, {dt:.1f} s",
            "host_cpu": _cpu_model(), "host_nproc": os.cpu_count()}


def sweep(args):
    """The budget/schedule sweep: one JSON line, one entry per (workload,
    schedule, budget) with the median call and every kernel's average launch
    duration and achieved bandwidth from the library's per-launch events."""
    import torch
    import paper_2509_02197_amd as adst
    from paper_2509_02197_amd.workloads import WORKLOADS

    def say(m):
        print(m, file=sys.stderr, flush=True)

    ids = {v: k for k, v in SCHED_NAMES.items()}
    entries, inputs = [], {}
    for name, sched, budget in SWEEP:
        if args.workload and name != args.workload:
            continue
        w = WORKLOADS[name]
        r, inputs[name] = run_workload(adst, torch, w, {"sched": ids[sched], "budget": budget},
                                       args.steps, args.warmup, args.traced_calls, say,
                                       inputs.get(name))
        say(f"# {name} {r['schedule']} slots={r['slots']}: median {r['ms_median']} ms")
        entries.append({k: r[k] for k in ("workload", "schedule", "budget_bytes", "slots",
                                          "fwd_steps", "recompute_steps", "fwd_kernels",
                                          "adj_kernels", "ms_median", "ms_ci95",
                                          "pt_steps_per_s", "phase_ms", "fwd_gbps",
                                          "adj_gbps", "kernels")})
        for k in entries[-1]["kernels"]:
            k["frac"] = round(k["gbps"] / HBM_PEAK_GBPS, 4)
        for name_ in [n for n in inputs if n != name]:
            del inputs[name_]
    print(json.dumps({"sweep": entries, "steps": args.steps, "warmup": args.warmup,
                      "traced_calls": args.traced_calls}), flush=True)


def main_bench(args):
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); this build has no "
              f"multi-GPU path", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2509_02197_amd as adst
    from paper_2509_02197_amd.workloads import HEADLINE, WORKLOADS

    def say(m):
        print(m, file=sys.stderr, flush=True)

    name = args.workload or HEADLINE
    w = WORKLOADS[name]
    opts = {"force_tape": args.force_tape, "no_fuse": args.no_fuse, "limit": args.limit,
            "dparams": args.dparams}
    if args.sched:
        opts["sched"] = {v: k for k, v in SCHED_NAMES.items()}[args.sched]
    if args.budget_bytes is not None:
        opts["budget"] = args.budget_bytes
    t_start = time.perf_counter()
    r, _ = run_workload(adst, torch, w, opts, args.steps, args.warmup, args.traced_calls, say)
    say(f"# headline done: median {r['ms_median']} ms per call")
    res = {
        "metric": METRIC, "value": r["pt_steps_per_s"], "unit": "grid-point-steps/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": r["wall_ms_per_call"], "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": r["dtype"], "data": "synthetic",
        "config": {k: r[k] for k in ("workload", "grid", "T", "kind", "loss", "budget_bytes",
                                     "schedule", "slots", "fwd_steps", "recompute_steps",
                                     "fwd_kernels", "adj_kernels", "grads", "force_tape",
                                     "temporal_blocking", "limiter")},
        "timing": {k: r[k] for k in ("calls", "ms_median", "ms_ci95", "ms_mean", "ms_min",
                                     "ms_max", "wall_ms_per_call")},
        "hbm_gbps_effective": r["hbm_gbps_effective"],
        "phase_ms": r["phase_ms"],
        "roofline": r["roofline"], "roofline_fwd": r["roofline_fwd"],
        "roofline_adj": r["roofline_adj"], "kernels": r["kernels"],
    }
    res["timing"]["method"] = ("per-call HIP event pairs on the call's stream; value = "
                               "npoints*T / median call; 95% CI of the median from order "
                               "statistics")
    res["copy_ceiling"] = copy_ceiling(adst, torch, w.state_bytes)
    if not args.no_extras and args.workload is None:
        extras = []
        for ename, eo in EXTRAS:
            ew = WORKLOADS[ename]
            er, _ = run_workload(adst, torch, ew, dict(eo), args.extra_steps, 1, 1, say)
            ent = {k: er[k] for k in ("workload", "schedule", "slots", "fwd_steps", "grads",
                                      "force_tape", "ms_median", "ms_ci95", "pt_steps_per_s",
                                      "fwd_gbps", "adj_gbps")}
            for key in ("roofline", "roofline_fwd", "roofline_adj"):
                rr = er[key]
                if rr:
                    ent[key] = {k: rr[k] for k in ("kernel", "achieved", "frac", "avg_launch_ms",
                                                   "alg_bytes_per_launch", "traffic")}
            extras.append(ent)
        res["workloads"] = extras
    if args.copy_probe_mib:
        dev = torch.device("cuda:0")
        a = torch.empty(args.copy_probe_mib << 17, dtype=torch.float64, device=dev).fill_(1.0)
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        for _ in range(3):
            adst.adst_copy(b, a, a.numel() * 8)
        torch.cuda.synchronize()
        res["copy_probe_bytes"] = a.numel() * 8
        del a, b
    if not args.no_cpu_baseline:
        say("# cpu baseline (oracle) ...")
        res["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds, args.limit, args.dparams)
    res["bench_wall_s"] = round(time.perf_counter() - t_start, 1)
    print(json.dumps(res), flush=True)


# ------------------------------------------------------------ rocprof summaries
def rocprof_label(name):
    """The library's label of a kernel from its rocprofv3 name."""
    n = name.replace("void ", "").replace("adst::(anonymous namespace)::", "")
    n = re.sub(r"\(.*$", "", n).strip()
    if n.startswith("__amd_rocclr_copyBuffer"):
        return "hipMemcpyAsync copy"
    if n.startswith("at::native::"):
        return "torch elementwise"
    m = re.match(r"(\w+)<(.*)>$", n)
    base, targs = (m.group(1), [a.strip() for a in m.group(2).split(",")]) if m else (n, [])
    t = lambda i: targs[i] == "true"  # noqa: E731
    if base == "fwd_allencahn3d7_n":   # <R, K, RPT, NZ, NT, ST>
        return f"fwd_allencahn3d7_n<{targs[1]}" + (",store>" if t(5) else ">")
    if base == "fwd_vardiff2d9_x2":    # <R, TR, NT, ST>
        return "fwd_vardiff2d9_x2" + ("<store>" if t(3) else "")
    if base == "jacobi_march":         # <R, K, ADJ, VEC>
        return f"jacobi_march<{'adj' if t(2) else 'fwd'},{targs[1]}>"
    if base == "jacobi_lim_adjoint":   # <R, VEC, DP>
        return "jacobi_lim_adjoint<dp>" if t(2) else "jacobi_lim_adjoint"
    if base == "gs_wave":              # <R, ADJ, VEC>
        return "gs_wave<adj>" if t(1) else "gs_wave<fwd>"
    if base == "ac_march":             # <R, NF, ADJ, RR, ZC, DA, ST, NT>
        if t(2):
            return "ac_march<adj>" if targs[1] == "0" else f"ac_march<fwd{targs[1]}+adj>"
        return f"ac_march<fwd,{targs[1]}" + (",store>" if t(6) else ">")
    if base == "adj_allencahn3d7":     # <R, DP, NT>
        return "adj_allencahn3d7<dp>" if t(1) else "adj_allencahn3d7"
    if base == "adj_vardiff2d9":       # <R, WANT_DK, TR, DP, NT>
        v = [s for s, on in (("dK", t(1)), ("dp", t(3))) if on]
        return "adj_vardiff2d9" + (f"<{','.join(v)}>" if v else "")
    if base in ("fwd_jacobi2d5", "fwd_vardiff2d9", "fwd_allencahn3d7"):  # <R, LIM, NT>
        return base + ("<lim>" if len(targs) > 1 and t(1) else "")
    return base


def _csv(d, suffix):
    hits = glob.glob(os.path.join(d, "**", f"*{suffix}"), recursive=True)
    if not hits:
        raise SystemExit(f"no *{suffix} under {d}")
    return list(csv.DictReader(open(sorted(hits)[0])))


def _kernel_rows(d):
    """Per-kernel rows (Name, Calls, TotalDurationNs, MinNs, MaxNs,
    Percentage) from a rocprofv3 --stats CSV, or from the kernel dispatches
    of its SQLite output (*_results.db) when it was not written as CSV."""
    if glob.glob(os.path.join(d, "**", "*kernel_stats.csv"), recursive=True):
        return _csv(d, "kernel_stats.csv")
    import sqlite3
    hits = glob.glob(os.path.join(d, "**", "*_results.db"), recursive=True)
    if not hits:
        raise SystemExit(f"no *kernel_stats.csv or *_results.db under {d}")
    con = sqlite3.connect(sorted(hits)[0])
    agg = con.execute("SELECT name, COUNT(*), SUM(duration), MIN(duration), MAX(duration) "
                      "FROM kernels GROUP BY name").fetchall()
    total = sum(r[2] for r in agg) or 1
    return [{"Name": n, "Calls": c, "TotalDurationNs": t, "MinNs": lo, "MaxNs": hi,
             "Percentage": 100.0 * t / total} for n, c, t, lo, hi in agg]


def rocprof_summary(args):
    """Markdown of kernel times (and HBM bytes with --fetch/--write) from
    rocprofv3 CSV output, kernels named by the library's labels; HBM bytes
    are FETCH_SIZE and WRITE_SIZE scaled so that the last plain copy of the
    run (a 1 GiB hipMemcpyAsync from --copy-probe-mib 1024) counts its bytes
    exactly; the per-launch figures also go to profiles/traffic.json."""
    rows = _kernel_rows(args.rocprof_summary)
    out = [f"# Kernel time: {args.title}", "",
           "Command (from the repository root on the GPU box, after "
           "`cd /tmp && export TMPDIR=/tmp`):", "", "```", args.command, "```", "",
           "| kernel | calls | avg us | min us | max us | % time |", "|---|---|---|---|---|---|"]
    agg = {}
    for r in rows:
        lab = rocprof_label(r["Name"])
        a = agg.setdefault(lab, [0, 0.0, 1e30, 0.0, 0.0])
        c = int(r["Calls"])
        a[0] += c
        a[1] += float(r["TotalDurationNs"])
        a[2] = min(a[2], float(r["MinNs"]))
        a[3] = max(a[3], float(r["MaxNs"]))
        a[4] += float(r["Percentage"])
    for lab, a in sorted(agg.items(), key=lambda kv: -kv[1][1]):
        out.append(f"| {lab} | {a[0]} | {a[1] / a[0] / 1e3:.2f} | {a[2] / 1e3:.2f} | "
                   f"{a[3] / 1e3:.2f} | {a[4]:.2f} |")
    if args.fetch and args.write:
        def load(d):
            acc = {}
            for r in _csv(d, "counter_collection.csv"):
                acc.setdefault(rocprof_label(r["Kernel_Name"]), []).append(
                    float(r["Counter_Value"]))
            return acc
        f, wr = load(args.fetch), load(args.write)
        cp = "hipMemcpyAsync copy"
        fs, ws = (1 << 20) / f[cp][-1], (1 << 20) / wr[cp][-1]
        out += ["", f"HBM bytes: FETCH_SIZE and WRITE_SIZE (KiB per dispatch, one counter per "
                    f"run), scaled by the 1 GiB plain copy of the same run (FETCH_SIZE reads "
                    f"{f[cp][-1]:.0f} KiB for it: factor {fs:.4f}; WRITE_SIZE {wr[cp][-1]:.0f} "
                    f"KiB: factor {ws:.4f}).", "",
                "| kernel | dispatches | FETCH_SIZE KiB | WRITE_SIZE KiB | HBM bytes/launch | "
                "algorithmic bytes/launch | ratio |",
                "|---|---|---|---|---|---|---|"]
        tpath = os.path.join(ROOT, "profiles", "traffic.json")
        table = json.load(open(tpath)) if os.path.exists(tpath) else {}
        wl = args.workload or "workload"
        alg = {}
        if args.bench_json:  # algorithmic bytes per launch from a bench line of the same run
            line = [ln for ln in open(args.bench_json) if ln.startswith("{")][-1]
            alg = {k["name"]: k["alg_bytes_per_launch"] for k in json.loads(line)["kernels"]}
        for lab in sorted(f, key=lambda k: -len(f[k])):
            if lab not in wr or lab.startswith("hipMemcpy") or lab.startswith("torch") \
                    or lab == "copy_once":
                continue
            fk = sum(f[lab]) / len(f[lab])
            wk = sum(wr[lab]) / len(wr[lab])
            b = (fk * fs + wk * ws) * 1024
            a = alg.get(lab)
            ratio = f"{b / a:.3f}" if a else "-"
            out.append(f"| {lab} | {len(f[lab])} | {fk:.1f} | {wk:.1f} | {b:.4g} | "
                       f"{a if a is None else f'{a:.4g}'} | {ratio} |")
            table[f"{wl}:{lab}"] = {"bytes_per_launch": int(round(b)), "fetch_kib": fk,
                                    "write_kib": wk, "fetch_scale": fs, "write_scale": ws,
                                    "src_sha": source_sha(lab)}
        with open(tpath, "w") as fh:
            json.dump(table, fh, indent=1, sort_keys=True)
    text = "\n".join(out) + "\n"
    if args.out:
        with open(args.out, "w") as fh:
            fh.write(text)
    print(text)


def main():
    args = parse()
    if args.gpus != 1 and not args.rocprof_summary:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); this build has no "
              f"multi-GPU path", file=sys.stderr)
        sys.exit(2)
    if args.rocprof_summary:
        rocprof_summary(args)
        return
    if args.sweep:
        sweep(args)
        return
    main_bench(args)


if __name__ == "__main__":
    main()
