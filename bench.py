"""Benchmark of the gs-SGD compression hot path on one MI355X.

One step = accumulate + sketch + merge + estimate/top-k + gather/reset (the fused gs_step)
over the P workers' gradients of one iteration, inputs resident in HBM. Default workload:
d = 25,600,000 (ResNet-50-sized), P = 8 workers, r x c = 5 x 256,000, k = 25,600, gradients
Laplace(0, b_s) with 53 log-uniform layer scales in [1e-5, 1e-2] (synthetic, seeded).

Prints one JSON line with
  value        gradient coordinates per second, P*d / (mean time per step over the timed steps);
               the median and minimum step times are reported beside it
  copy_frac    algorithmic GB/s as a fraction of a plain device copy timed in the same run
  roofline     the dominant stage's algorithmic bytes / its mean duration (HIP events the
               library records between the stages, on the stream the kernels run on, in as
               many further steps after the timed region, which carries no events inside a
               step) against MI355X's 8 TB/s HBM peak
  cpu_baseline the plain CPU oracle (single thread) timed on a bounded sample
Algorithmic bytes per step: B = 20*P*d + 8*r*c + 12*P*k + 8*k (vector state; the fused step
never writes the P per-worker tables); with --state sketch (momentum and error kept in the
sketch) B = 4*P*d + 24*r*c + 8*k.

The roofline object names the dominant kernel: of the stages within 10% of the longest one,
the one furthest below the HBM peak in algorithmic bytes. It also carries every such
co-dominant stage and the whole step's fraction (B / time per step / 8 TB/s).
"""
from __future__ import annotations

import argparse
import glob
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MI355X_CUS = 256  # compute units, when no device is visible to ask
METRIC = "gradient coords/sec per full sketch+unsketch+top-k step; % of HBM peak"


def stage_bytes(w, state: str = "vector") -> dict:
    """Algorithmic bytes each stage must move (not what an implementation happens to move)."""
    P, d, r, c, k = w.P, w.d, w.r, w.c, w.k
    if state == "sketch":
        return {
            "interleave": 0,                      # implementation only (g is read by the sketch)
            "sketch": 4 * P * d + 4 * r * c,      # read g, write the merged table (merged in the tiles)
            "merge": 0,                           # no kernel
            "select": 4 * r * c + 16 * r * c + 4 * r * c + 4 * k,  # read S; U, E read+written; E read
            "state_update": 8 * k,                # values and the correction of touched cells
        }
    # the fused step never writes the P per-worker tables: its tiles merge their own cells
    return {
        "accumulate": 20 * P * d,            # read g, u, v; write u, v
        "sketch": 4 * P * d + 4 * r * c,     # read v once, write the merged table
        "merge": 0,                          # no kernel: merged inside the sketch's tiles
        "select": 4 * r * c + 4 * k,         # read the merged table, write k indices
        "gather_reset": 12 * P * k + 4 * k,  # read v, zero u and v at k coordinates; write k values
    }


def step_bytes(w, state: str = "vector") -> int:
    """Algorithmic bytes of one fused step. Vector state: read g, u, v and write u, v
    (20 P d); the merged table written and read (8 r c); at the k selected coordinates v
    read, u and v zeroed (12 P k); idx and values written (8 k). The P per-worker tables
    never reach memory in the fused step, so they are not counted. Sketch state: read g
    (4 P d); merged written (4 r c); U, E read and written (16 r c); E read for the
    estimates (4 r c); idx and values (8 k)."""
    P, d, r, c, k = w.P, w.d, w.r, w.c, w.k
    if state == "sketch":
        return 4 * P * d + 4 * r * c + 16 * r * c + 4 * r * c + 8 * k
    return 20 * P * d + 8 * r * c + 12 * P * k + 8 * k


def roofline_of(stages: list, step_bytes_: int, step_ms: float):
    """The roofline object of the bench line. `stages`: per stage {stage, kernel, mean_ms,
    bytes_per_launch, achieved, frac, traffic, traffic_frac}. The dominant kernel is, among
    the stages within 10% of the longest one (co-dominant), the one furthest below the HBM
    peak in algorithmic bytes per second; every co-dominant stage and the whole step's
    fraction are reported beside it."""
    if not stages:
        return None
    longest = max(e["mean_ms"] for e in stages)
    co_dominant = [e for e in stages if e["mean_ms"] >= 0.9 * longest]
    p = min(co_dominant, key=lambda e: e["frac"])
    t = step_ms * 1e-3
    return {"bound": "hbm", "kernel": p["kernel"], "stage": p["stage"], "achieved": p["achieved"],
            "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": p["frac"], "traffic": p["traffic"],
            "traffic_unit": "bytes per launch", "bytes_per_launch": p["bytes_per_launch"], "mean_ms": p["mean_ms"],
            "co_dominant": co_dominant,
            "step": {"bytes": step_bytes_, "ms": step_ms, "achieved": step_bytes_ / t / 1e9,
                     "frac": step_bytes_ / t / 1e9 / HBM_PEAK_GBS}}


def log(msg):
    print(msg, file=sys.stderr, flush=True)


CSRC = os.path.join(ROOT, "paper_2108_06004_amd", "csrc")
# launch configuration and shared device helpers: a change there can change any kernel
SHARED_SOURCES = ("gs_api.hip", "gs_internal.hpp", "gs_device.hpp")


def file_sha256(path: str) -> str:
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def kernel_source_file(name: str):
    """The HIP source that defines kernel `name` (template arguments ignored), or None."""
    base = name.split("<")[0].strip()
    for p in sorted(glob.glob(os.path.join(CSRC, "*.hip"))):
        if re.search(r"__global__[^;{]*\b" + re.escape(base) + r"\s*\(", open(p).read()):
            return os.path.basename(p)
    return None


def num_cus() -> int:
    """Compute units of device 0 (the library sizes its grids by the device's count)."""
    try:
        import torch

        if torch.cuda.is_available():
            return torch.cuda.get_device_properties(0).multi_processor_count
    except Exception:
        pass
    return MI355X_CUS


def stage_kernels(w, layout: str = "interleaved", plan: dict = None) -> dict:
    """The kernels each stage of the fused step launches (names as rocprofv3 reports them).
    `plan` is the context's gs_describe; without it the library's size rule is assumed (list
    segments only for small sketches)."""
    if layout == "interleaved":
        ragged = "true" if w.d % (64 // (w.P // 4)) else "false"  # the last chunk of 64 / G coordinates
        acc = [f"k_accumulate_il<{w.P // 4}, {ragged}>"]
    elif w.P == 1:
        acc = ["k_accumulate4"]
    else:
        acc = [f"k_vi_il<{w.P}, true>"]
    tail = ["k_digit2", "k_select2", "k_mark", "k_emit"]
    # the full estimate's form: two coordinates per thread per pass up to 8 * 256 * (CUs)
    unsketch = f"k_unsketch<{w.r}, {2 if w.d <= 8 * 256 * num_cus() else 1}>"
    if w.d * w.r > 2_000_000:  # pruned selection (the library's choice above 2,000,000 cells of d*r)
        select = [f"k_sample<{w.r}, false>", "k_heavy", f"k_pruned<{w.r}, false, 0>", f"k_survivors<{w.r}, false>",
                  unsketch] + tail
    else:  # every coordinate estimated
        select = [unsketch] + tail
    segmented = plan["segments"] > 1 if plan is not None else w.d <= 1_000_000
    return {
        "accumulate": acc,
        # packed lists (the library's choice here); one worker in the worker-major layout: its
        # plain state vector gathered directly (the last template argument)
        "sketch": [f"k_pull<{w.P}, {4 if w.P <= 4 else 6}, true, "
                   f"{'true' if w.P == 1 and layout == 'worker_major' else 'false'}>"],
        # the tiles merge their own cells; small sketches' tiles, split into list segments,
        # are summed here
        "merge": [f"k_merge_partials<{w.P}>"] if segmented else [],
        "select": select,
        "gather_reset": [f"k_gather_reset<{w.P}>"],
    }


def measured_traffic(w, stage: str, layout: str = "interleaved"):
    """HBM-side bytes per launch of `stage` from the committed counter summary, or None when
    there is none for this workload and state layout, or when a source file the stage's kernels
    depend on (their own file and the shared ones) differs from the one the counters ran."""
    path = os.path.join(ROOT, "profiles", f"traffic_gs_step_{w.name}_{layout}.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    recorded = dict(re.findall(r"source_sha256\[([\w.]+)\]: ([0-9a-f]{64})", text))
    table = {name.strip(): float(val) for name, val in re.findall(r"traffic: (.+?) \| ([0-9.]+)", text)}
    names = stage_kernels(w, layout).get(stage)
    if not names or not all(n in table for n in names):
        return None
    for n in names:
        f = kernel_source_file(n)
        if f is None:
            return None
        for dep in (f,) + SHARED_SOURCES:
            if recorded.get(dep) != file_sha256(os.path.join(CSRC, dep)):
                return None
    return sum(table[n] for n in names)


def cpu_baseline(w, g, budget_s: float, min_s: float = 10.0) -> dict:
    """Time the oracle (as it stands), single-threaded, on consecutive steps of the same workload
    from zero state (the given gradients every step, the state carried over): steps are added
    until at least min_s has passed, and none is started that would pass budget_s."""
    import oracle
    import synth

    hp = synth.hash_params(w)
    u = np.zeros_like(g)
    v = np.zeros_like(g)
    n, dt = 0, 0.0
    while n == 0 or (dt < min_s and dt + dt / n <= budget_s and n < 1000):
        t0 = time.perf_counter()
        oracle.step(g, u, v, hp, w.c, w.k, rho=w.rho, want_tables=False, want_est=False)
        dt += time.perf_counter() - t0
        n += 1
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"value": n * w.P * w.d / dt, "unit": "coords/s", "cores": 1, "kind": "oracle",
            "sample": f"{n} consecutive full step(s) of {w.name} (P*d = {w.P * w.d} coordinates each) from zero "
                      f"state, the step-0 gradients every step, {dt:.1f} s single-threaded", "seconds": round(dt, 3),
            "steps": n,
            "host_nproc": os.cpu_count(), "host_cpu": model}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="laplace53-d25.6M-P8")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--profile-steps", type=int, default=None,
                    help="steps run after the timed region with stage events recorded between the "
                         "stages, for the stage breakdown and the roofline (default: as many as timed; 0: none)")
    ap.add_argument("--selection", choices=("topk", "heavymix"), default="topk",
                    help="topk: deterministic top-k by |estimate| (gs_step); heavymix: HEAVYMIX as printed with a "
                         "seeded random fill (gs_step_heavymix)")
    ap.add_argument("--state", choices=("vector", "sketch"), default="vector",
                    help="vector: per-worker u, v d-vectors (gs_step / gs_step_heavymix); sketch: momentum and error "
                         "kept in the merged sketch (gs_step_sketch_momentum; deterministic top-k)")
    ap.add_argument("--state-layout", choices=("interleaved", "worker_major"), default="interleaved",
                    help="layout of the per-worker state u, v: interleaved [d][P] rows (the sketch gathers them "
                         "directly) or worker-major [P][d] (the accumulation also writes an interleaved copy)")
    ap.add_argument("--compare-layout", action=argparse.BooleanOptionalAction, default=True,
                    help="also time the same steps with the other state layout (reported under other_layout)")
    ap.add_argument("--calibration-copy", action="store_true",
                    help="before warm-up, run one plain device copy of the gradient buffer (P*d*4 bytes read and "
                         "written) to calibrate rocprofv3 FETCH_SIZE / WRITE_SIZE counters")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (the P workers are simulated on one device); --gpus {args.gpus} "
              f"is not supported", file=sys.stderr)
        sys.exit(2)

    import torch

    import synth
    import paper_2108_06004_amd as gs

    w = synth.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    hp = synth.hash_params(w)
    log(f"[bench] generating inputs for {w.name}")
    nb = min(2, w.steps)
    g_host = [synth.gradients(w, t) for t in range(nb)]
    g_dev = [torch.from_numpy(x).to(dev) for x in g_host]
    merged = torch.empty((w.r, w.c), dtype=torch.float32, device=dev)
    idx = torch.empty(w.k, dtype=torch.int32, device=dev)
    vals = torch.empty(w.k, dtype=torch.float32, device=dev)
    layout = args.state_layout if args.state == "vector" else "worker_major"
    torch.cuda.synchronize()
    c_t0 = time.perf_counter()
    ctx = gs.GsContext(w.d, w.P, w.r, w.c, w.k, hp, rho=w.rho, state_layout=layout)
    torch.cuda.synchronize()
    create_ms = (time.perf_counter() - c_t0) * 1e3  # gs_create: scratch and the static tile lists
    plan = ctx.describe()
    u = torch.zeros(ctx.state_shape, dtype=torch.float32, device=dev)
    v = torch.zeros_like(u)
    if args.state == "sketch":
        if args.selection != "topk":
            print("--state sketch uses the deterministic top-k selection", file=sys.stderr)
            sys.exit(2)
        U_s = torch.zeros((w.r, w.c), dtype=torch.float32, device=dev)
        E_s = torch.zeros_like(U_s)

        def run_step(s_):
            ctx.step_sketch_momentum(g_dev[s_ % nb], U_s, E_s, w.k, merged, idx, vals)
    elif args.selection == "heavymix":
        # one set of fill draws per gradient batch (fresh draws each step in real use)
        rnd_dev = [torch.from_numpy(synth.fill_draws(w, t).view(np.int32)).to(dev) for t in range(nb)]

        def run_step(s_):
            ctx.step_heavymix(g_dev[s_ % nb], u, v, w.k, rnd_dev[s_ % nb], merged, idx, vals)
    else:
        def run_step(s_):
            ctx.step(g_dev[s_ % nb], u, v, w.k, merged, idx, vals)
    torch.cuda.synchronize()
    if args.calibration_copy:
        scratch = torch.empty_like(g_dev[0])
        scratch.copy_(g_dev[0])
        torch.cuda.synchronize()
        log(f"[bench] calibration copy: {g_dev[0].numel() * 4} bytes read and written")
        del scratch

    log(f"[bench] warmup {args.warmup}")
    for s in range(args.warmup):
        run_step(s)
    torch.cuda.synchronize()

    # the timed region: K steps on the caller's stream, step events by torch around them and
    # nothing recorded inside a step
    nprof = max(0, args.profile_steps if args.profile_steps is not None else args.steps)
    log(f"[bench] timing {args.steps} steps")
    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    ev[0].record(stream)
    for s in range(args.steps):
        run_step(s)
        ev[s + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms = ev[0].elapsed_time(ev[-1]) / args.steps
    per_step = sorted(ev[s].elapsed_time(ev[s + 1]) for s in range(args.steps))
    ms_median = per_step[len(per_step) // 2] if len(per_step) % 2 else \
        0.5 * (per_step[len(per_step) // 2 - 1] + per_step[len(per_step) // 2])
    # the stage breakdown: further steps with HIP events recorded by the library between the
    # stages (on the stream the kernels run on, without synchronizing); each event costs a few
    # microseconds, so these steps are kept out of the timed region
    if nprof > 0:
        log(f"[bench] {nprof} more steps with stage events")
        ctx.timing_start(nprof)
        for s in range(nprof):
            run_step(args.steps + s)
        torch.cuda.synchronize()
        stage_ms, n_timed = ctx.timing_stop()
    else:
        stage_ms, n_timed = {st: 0.0 for st in gs.STAGES}, 0
    if args.state == "sketch":  # stages of the sketch-space step
        stage_ms = {"interleave": stage_ms["accumulate"], "sketch": stage_ms["sketch"], "merge": stage_ms["merge"],
                    "select": stage_ms["select"], "state_update": stage_ms["gather_reset"]}
    sb = stage_bytes(w, args.state)
    kern = stage_kernels(w, layout, plan)
    stages = []
    for st, st_ms in stage_ms.items():
        if n_timed == 0 or st_ms <= 0 or sb.get(st, 0) <= 0:
            continue
        ach = sb[st] / (st_ms * 1e-3) / 1e9
        tr = measured_traffic(w, st, layout) if args.state == "vector" else None
        stages.append({"stage": st, "kernel": " + ".join(kern.get(st, [st])), "mean_ms": st_ms,
                       "bytes_per_launch": sb[st], "achieved": ach, "frac": ach / HBM_PEAK_GBS, "traffic": tr,
                       "traffic_frac": (tr / (st_ms * 1e-3) / 1e9 / HBM_PEAK_GBS) if tr else None})
    ctx.close()
    del u, v

    other_ms = None
    if args.compare_layout and args.state == "vector" and args.selection == "topk":
        other = "worker_major" if layout == "interleaved" else "interleaved"
        log(f"[bench] timing {args.steps} steps with the {other} state layout")
        ctx2 = gs.GsContext(w.d, w.P, w.r, w.c, w.k, hp, rho=w.rho, state_layout=other)
        u2 = torch.zeros(ctx2.state_shape, dtype=torch.float32, device=dev)
        v2 = torch.zeros_like(u2)
        for s in range(args.warmup):
            ctx2.step(g_dev[s % nb], u2, v2, w.k, merged, idx, vals)
        o0, o1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        o0.record(stream)
        for s in range(args.steps):
            ctx2.step(g_dev[s % nb], u2, v2, w.k, merged, idx, vals)
        o1.record(stream)
        torch.cuda.synchronize()
        other_ms = {"state_layout": other, "ms_per_step": o0.elapsed_time(o1) / args.steps}
        ctx2.close()
        del u2, v2

    # device copy bandwidth in the same run (read + write of one P*d fp32 buffer)
    src = g_dev[0]
    dst = torch.empty_like(src)
    dst.copy_(src)
    c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ncopy = 10
    torch.cuda.synchronize()
    c0.record(stream)
    for _ in range(ncopy):
        dst.copy_(src)
    c1.record(stream)
    torch.cuda.synchronize()
    copy_gbs = 2 * src.numel() * 4 / (c0.elapsed_time(c1) / ncopy * 1e-3) / 1e9
    del dst

    B = step_bytes(w, args.state)
    t = ms * 1e-3
    roofline = roofline_of(stages, B, ms)
    out = {
        "metric": METRIC,
        "value": w.P * w.d / t,
        "unit": "coords/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "ms_per_step_median": ms_median,
        "ms_per_step_min": per_step[0],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "d": w.d, "P": w.P, "r": w.r, "c": w.c, "k": w.k,
                   "selection": args.selection, "state": args.state, "state_layout": layout,
                   "gradients": w.note},
        "other_layout": other_ms,
        "coords_per_s_per_worker": w.d / t,
        "algorithmic_bytes_per_step": B,
        "achieved_gbs": B / t / 1e9,
        "hbm_frac": B / t / 1e9 / HBM_PEAK_GBS,
        "copy_gbs": copy_gbs,
        "copy_frac": B / t / 1e9 / copy_gbs,
        "wall_s_timed": wall,
        "stage_ms": stage_ms,
        "stage_ms_from": f"HIP events recorded between the stages of {n_timed} further steps after the timed region",
        "roofline": roofline,
        "create_ms": create_ms,
        "plan": plan,
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        log("[bench] CPU baseline (oracle steps, 10-30 s)")
        out["cpu_baseline"] = cpu_baseline(w, g_host[0], 30.0)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
