"""Benchmark: grid-point-steps/s of one forward+VJP call at a fixed memory
budget on one MI355X, with the dominant kernel's achieved HBM bandwidth
against the chip's peak and the CPU oracle timed on the host beside it.

One "step" of the benchmark is one adst_vjp call: the forward sweep, the
loss and seed, every recomputation the schedule needs and the reverse sweep,
over one synthetic input already resident in HBM. Throughput is
npoints * T / (wall time of one call).

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--sched S]
                    [--force-tape] [--no-cpu-baseline]
"""
import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "grid-point-steps/s for fwd+VJP at fixed memory budget; achieved HBM GB/s"
HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E
SCHED_NAMES = {0: "auto", 1: "store_all", 2: "uniform", 3: "binomial"}
LOSS_NAMES = {0: "half_sq", 1: "dot_w", 2: "half_sq_diff", 3: "seed"}
KERNELS = {  # (forward, adjoint) kernel names as rocprofv3 reports them
    0: ("fwd_jacobi2d5", "adj_jacobi2d5"),
    1: ("fwd_allencahn3d7", "adj_allencahn3d7"),
    2: ("fwd_vardiff2d9", "adj_vardiff2d9"),
    3: ("gs_wave<fwd>", "gs_wave<adj>"),
}


def kernel_name(kind, adj, n, xpass=False):
    """Short name of the kernel an action of n steps launches (xpass: the
    Jacobi adjoint that also reads x_{t-1}, for the limiter or the
    constants' gradients)."""
    base = KERNELS[kind][1 if adj else 0]
    if adj and xpass and kind == 0 and n == 1:
        return "jacobi_lim_adjoint"
    if kind == 3 or n == 1:
        return base
    if kind == 1:
        return f"{base}_n<{n}>"
    if n == 2:
        return base + "_x2"
    return f"jacobi_march<{'adj' if adj else 'fwd'},{n}>"


STORE_DEPTH = {1: 3, 2: 2}  # single steps per store-through launch (Allen-Cahn, VarDiff)


def stored_run(acts, i, depth):
    """Length of the run of chained single forward steps from acts[i] that
    adst_vjp takes in one launch writing every state (1: none)."""
    if depth < 2 or acts[i][0] != 0:
        return 1
    n = 1
    while n < depth and i + n < len(acts):
        a, p = acts[i + n], acts[i + n - 1]
        if a[0] != 0 or a[2] != p[3] or a[1] != p[1] + 1:
            break
        if a[3] == acts[i][2] or any(acts[i + k][3] == a[3] for k in range(n)):
            break
        n += 1
    return n


def kernel_mix(kind, acts, adj, xpass=False, store_depth=1):
    """Launch count per kernel name over a plan's forward or adjoint actions
    (a pipelined run of the in-place kind counts once, and so does a run of
    single forward steps that one store-through launch takes)."""
    ops = (2, 4, 6) if adj else (0, 3, 5)  # ADJ, ADJ2, ADJW / FWD, FWD2, FWDW
    mix = {}
    i = 0
    while i < len(acts):
        op, n = acts[i][0], acts[i][4]
        r = 1 if adj else stored_run(acts, i, store_depth)
        if op in ops:
            if r >= 2:
                k = (f"{KERNELS[kind][0]}_n<{r},store>" if kind == 1
                     else f"{KERNELS[kind][0]}_x2<store>")
            else:
                k = kernel_name(kind, adj, n, xpass)
            mix[k] = mix.get(k, 0) + 1
        i += r
    return mix


def kernel_source(kernel):
    """The source file holding a kernel (by its short name)."""
    if kernel.startswith("jacobi_march"):
        return "jacobi_march.hip"
    if kernel.startswith("gs_wave"):
        return "gauss_seidel.hip"
    return "kernels.hip"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
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
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target CPU time of the oracle sample")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="after the benchmark, copy a buffer of this size three times (a plain "
                         "copy kernel of known size, to scale hardware byte counters)")
    return ap.parse_args()


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


def cpu_baseline(w, inp, target_s, lim=None, want_dp=False):
    """The oracle (single-threaded store-all tape, as it stands) on the same
    grid, with the same limiter and gradients, for as many leading steps as
    fit about target_s seconds (whole calls repeated when all T steps take
    less)."""
    import oracle
    from paper_2509_02197_amd.workloads import dims_of  # noqa: F401
    x0, K, aux = inp["x0"], inp["K"], inp["aux"]
    n = x0.size
    # warm the pages once, then probe two steps to size the sample
    kw = dict(K=K, loss=w.loss, aux=aux, want_dK=w.want_dK, want_dp=want_dp, lim=lim)
    oracle.vjp(w.kind, x0, steps=1, **kw)
    t0 = time.perf_counter()
    oracle.vjp(w.kind, x0, steps=2, **kw)
    one = (time.perf_counter() - t0) / 2
    Ts = int(max(1, min(w.steps, target_s / max(one, 1e-6))))
    # whole calls are repeated while the sample is shorter than two thirds of
    # target_s (the grid's T steps may take less than that)
    reps, dt = 0, 0.0
    while reps == 0 or dt < 0.67 * target_s:
        t0 = time.perf_counter()
        oracle.vjp(w.kind, x0, steps=Ts, **kw)
        dt += time.perf_counter() - t0
        reps += 1
    return {"value": n * Ts * reps / dt, "unit": "grid-point-steps/s", "cores": 1, "kind": "oracle",
            "sample": f"full {'x'.join(map(str, x0.shape))} grid, first {Ts} of {w.steps} steps, "
                      f"{reps} call(s), store-all tape, single thread, {dt:.1f} s",
            "host_cpu": _cpu_model(), "host_nproc": os.cpu_count()}


def copy_ceiling(torch, dev, stream, state_bytes):
    """Bandwidth of a plain device-to-device copy (hipMemcpyAsync), bytes read
    plus bytes written over the event-timed copy: at one state's size (the
    buffers a launch streams; at 128 MiB a pair of them fits the 256 MB
    Infinity Cache) and at 2 GiB, far beyond it."""
    out = {"kernel": "hipMemcpyAsync device-to-device"}
    for key, nbytes in (("state_size", min(state_bytes, 2 << 30)), ("2GiB", 2 << 30)):
        a = torch.empty(nbytes // 8, dtype=torch.float64, device=dev).fill_(1.0)
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        reps = 10
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            b.copy_(a)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        out[key] = {"bytes": 2 * a.numel() * 8, "ms": round(ms, 5),
                    "GB/s": round(2 * a.numel() * 8 / (ms * 1e-3) / 1e9, 1)}
        del a, b
    return out


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); this build has no "
              f"multi-GPU path", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2509_02197_amd as adst
    from paper_2509_02197_amd.workloads import HEADLINE, WORKLOADS, dims_of, make_inputs

    name = args.workload or HEADLINE
    w = WORKLOADS[name]
    sched = w.sched
    if args.sched:
        sched = {v: k for k, v in SCHED_NAMES.items()}[args.sched]
    budget = w.budget_bytes if args.budget_bytes is None else args.budget_bytes
    flags = (adst.ADST_FORCE_TAPE if args.force_tape else 0) | \
        (adst.ADST_NO_FUSE if args.no_fuse else 0)

    print(f"# bench workload={name} sched={SCHED_NAMES[sched]} budget={budget} "
          f"force_tape={args.force_tape}", file=sys.stderr, flush=True)
    inp = make_inputs(w)
    dev = torch.device("cuda:0")
    x0 = torch.from_numpy(inp["x0"]).to(dev)
    K = torch.from_numpy(inp["K"]).to(dev) if inp["K"] is not None else None
    aux = torch.from_numpy(inp["aux"]).to(dev) if inp["aux"] is not None else None
    prob = adst.make_problem(w.kind, w.dtype, dims_of(w.shape), w.params, flags, args.limit)
    grads = (adst.ADST_GRAD_COEFF if w.want_dK else 0) | \
        (adst.ADST_GRAD_PARAMS if args.dparams else 0)
    info = adst.adst_plan(prob, w.steps, budget, sched, grads)
    acts = adst.adst_plan_actions(prob, w.steps, budget, sched, grads)
    ws = torch.empty(info.workspace_bytes, dtype=torch.uint8, device=dev)
    dx0 = torch.empty_like(x0)
    dK = torch.empty_like(x0) if w.want_dK else None
    L = torch.empty((), dtype=torch.float64, device=dev)
    dP = torch.empty(2, dtype=torch.float64, device=dev) if args.dparams else None
    stream = torch.cuda.current_stream()

    def call(p):
        return adst.adst_vjp(p, x0, K, w.steps, w.loss, aux, budget, sched, dx0, dK, None, L, dP,
                             ws, ws.numel(), stream)

    for _ in range(args.warmup):
        call(prob)
    torch.cuda.synchronize()

    # ---- timed region: K calls, no tracing
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(args.steps):
        call(prob)
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ev_ms = e0.elapsed_time(e1)
    ms_per_step = 1e3 * wall / args.steps
    pts = w.npoints * w.steps
    value = pts / (wall / args.steps)

    # ---- roofline leg: the same K calls with per-launch HIP events
    tprob = adst.make_problem(w.kind, w.dtype, dims_of(w.shape), w.params,
                              flags | adst.ADST_TRACE, args.limit)
    acc = {"ms_fwd_sweep": 0.0, "ms_fwd_recompute": 0.0, "ms_adj": 0.0, "ms_seed": 0.0,
           "ms_dparams": 0.0, "ms_total": 0.0}
    for _ in range(args.steps):
        ti = call(tprob)
        for k in acc:
            acc[k] += getattr(ti, k) / args.steps
    # Roofline of the dominant phase's kernel: its algorithmic bytes (inputs
    # read once and outputs written once per launch; a launch of n fused
    # steps moves the same bytes as a single step; the in-place kind's
    # pipelined runs move 2 * itemsize per point per step) over its launch
    # time. avg_launch_ms is the phase's time over its kernel dispatches; the
    # kernel named is the phase's most frequent one, kernel_mix the rest.
    isz = 8 if w.dtype == adst.ADST_F64 else 4
    adj_B = {0: 2, 1: 3, 2: 6 if w.want_dK else 3, 3: 2}[w.kind] * isz
    if args.dparams and (w.kind == adst.ADST_JACOBI2D5 or
                         (w.kind == adst.ADST_VARDIFF2D9 and not w.want_dK)):
        adj_B += isz  # the fused constants' gradients also read x_{t-1}
    elif args.limit and w.kind == adst.ADST_JACOBI2D5:
        adj_B += isz  # the adjoint applies the branch mask, reading x_{t-1}
    in_place = w.kind == adst.ADST_GAUSSSEIDEL2D5
    # units of adj_B * npoints moved per call: one per launch, or one per step;
    # the forward launches' bytes come from the plan (a store-through launch
    # of n steps moves its input once and each of its n states once)
    adj_units = info.adj_steps if in_place else info.adj_launches
    fwd_total = info.fwd_alg_bytes
    store_depth = 1 if (args.no_fuse or args.limit) else STORE_DEPTH.get(w.kind, 1)
    n_fwd, n_adj = info.fwd_kernels, info.adj_kernels
    ms_fwd = acc["ms_fwd_sweep"] + acc["ms_fwd_recompute"]
    fwd_avg = ms_fwd / max(n_fwd, 1)
    adj_avg = acc["ms_adj"] / max(n_adj, 1)
    if ms_fwd >= acc["ms_adj"]:
        mix = kernel_mix(w.kind, acts, False, store_depth=store_depth)
        ms_k, alg_total, nl, ns = ms_fwd, fwd_total, n_fwd, info.fwd_steps_total
    else:
        mix = kernel_mix(w.kind, acts, True, bool(args.dparams or args.limit))
        ms_k, nl, ns = acc["ms_adj"], n_adj, info.adj_steps
        alg_total = adj_B * w.npoints * adj_units
    kernel = max(mix, key=lambda k: mix[k]) if mix else "none"
    avg_ms = ms_k / max(nl, 1)
    alg_bytes = alg_total / max(nl, 1)
    achieved = alg_total / (ms_k * 1e-3) / 1e9
    traffic = traffic_for(name, kernel)
    roofline = {
        "bound": "hbm", "kernel": kernel, "kernel_mix": mix, "achieved": round(achieved, 1),
        "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
        "traffic": traffic, "alg_bytes_per_launch": alg_bytes,
        "avg_launch_ms": round(avg_ms, 5), "launches_per_step": nl,
        "steps_per_launch": round(ns / max(nl, 1), 3),
        "fwd_avg_ms": round(fwd_avg, 5),
        "fwd_gbps": round(fwd_total / max(ms_fwd, 1e-9) / 1e6, 1),
        "adj_avg_ms": round(adj_avg, 5),
        "adj_gbps": round(adj_B * w.npoints * adj_units / max(acc["ms_adj"], 1e-9) / 1e6, 1),
    }
    if args.dparams:  # the final sum of the constants' per-workgroup slots
        roofline["dparam_finalize_ms"] = round(acc["ms_dparams"], 4)

    res = {
        "metric": METRIC, "value": value, "unit": "grid-point-steps/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f64" if w.dtype == adst.ADST_F64 else "f32", "data": "synthetic",
        "config": {
            "workload": name, "grid": list(w.shape), "T": w.steps, "kind": adst.workloads.KIND_NAMES[w.kind],
            "loss": LOSS_NAMES[w.loss], "budget_bytes": budget,
            "schedule": SCHED_NAMES[info.sched] + ("" if info.needs_state else " (tape elided)"),
            "slots": info.slots, "fwd_steps": info.fwd_steps_total,
            "recompute_steps": info.recompute_steps, "fwd_launches": info.fwd_launches,
            "adj_launches": info.adj_launches, "fwd_kernels": info.fwd_kernels,
            "adj_kernels": info.adj_kernels,
            "grads": ("dx0,dK" if w.want_dK else "dx0") + (",dparams" if args.dparams else ""),
            "force_tape": bool(args.force_tape), "temporal_blocking": not args.no_fuse,
            "limiter": args.limit,
        },
        "hbm_gbps_effective": round(info.alg_bytes / (ms_per_step * 1e-3) / 1e9, 1),
        "event_ms_per_step": ev_ms / args.steps,
        "phase_ms": {k: round(v, 4) for k, v in acc.items()},
        "roofline": roofline,
    }
    res["copy_ceiling"] = copy_ceiling(torch, dev, stream, w.npoints * isz)
    if args.copy_probe_mib:
        del ws
        a = torch.empty(args.copy_probe_mib << 17, dtype=torch.float64, device=dev).fill_(1.0)
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        res["copy_probe_bytes"] = a.numel() * 8
    if not args.no_cpu_baseline:
        print("# cpu baseline (oracle) ...", file=sys.stderr, flush=True)
        res["cpu_baseline"] = cpu_baseline(w, inp, args.cpu_seconds, args.limit, args.dparams)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
