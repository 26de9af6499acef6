#!/usr/bin/env python3
"""Benchmark: one fwd+bwd training step of a sampled-subgraph GCN on one MI355X.

Workload (default): 2-layer GCN on a 65,536-vertex R-MAT subgraph (average
degree 50, 3,276,800 stored edges, mean-normalised CSR), H_in 65536x512,
hidden 512 per branch (concat 1024), linear PREDICT + softmax-CE over 100
classes; synthetic seeded inputs, random Glorot weights.  One step = CSR
transpose + both layers forward + loss head + both layers backward, inputs
resident in HBM.  Prints one JSON line.

  value        whole-step edge-features/s (sum over aggregation passes of
               nnz x width, divided by the step time)
  roofline     the kernel class with the most time in the timed region, timed
               with HIP events on its launch stream (library profiler)
  cpu_baseline the CPU oracle on the same workload, whole steps timed for at
               least --cpu-seconds on the host's cores
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "GCN layer fwd+bwd: subgraph edge-features/s and GFLOP/s; % HBM/MFMA peak"
PEAK_HBM_GBS = 8000.0
PEAK_TFLOPS = {"f32": 157.3, "bf16": 2500.0}
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


KERNEL_SOURCES = {"gemm": ["gemm.hip", "common.h"], "spmm": ["spmm.hip", "common.h"]}


def kernel_source_hash(kernel: str) -> str:
    """Hash of the source files the kernel class is built from."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_1810_11899_amd", "csrc")
    for f in KERNEL_SOURCES["gemm" if kernel.startswith("gemm") else "spmm"]:
        h.update(open(os.path.join(csrc, f), "rb").read())
    return h.hexdigest()[:16]


def traffic_for(kernel: str, config: str):
    """HBM bytes per launch (FETCH_SIZE + WRITE_SIZE, copy-calibrated) from the
    committed counter runs, or None when they are missing or the kernel's
    source has changed since they were taken."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    try:
        t = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    e = t.get(config, {}).get(kernel)
    if not e or e.get("source_hash") != kernel_source_hash(kernel):
        return None
    return e.get("bytes_per_launch")


def cpu_baseline(cfg: int, synth, step_work, B, min_seconds: float = 10.0, max_reps: int = 20):
    """The CPU oracle on the same workload: whole fwd+bwd steps, repeated until
    at least `min_seconds` of CPU work have been timed (bounded by max_reps)."""
    import oracle
    wl = synth.config(cfg)
    L = len(wl.layers)
    dims = [(l.f_in, l.h) for l in wl.layers]
    need = [li > 0 for li in range(L)] if L > 1 else [True]
    orders = [B.gcn_layer_pick_order(f, h, d) for (f, h), d in zip(dims, need)]
    work = step_work(wl.n, wl.graph.nnz, dims, orders, need,
                     wl.spec.classes if wl.spec.head else 0)
    oracle.step(synth.config(cfg, n=1024))  # warm the thread pool on a tiny instance
    reps, dt = 0, 0.0
    while reps < max_reps and (reps == 0 or dt < min_seconds):
        t0 = time.perf_counter()
        oracle.step(wl)
        dt += time.perf_counter() - t0
        reps += 1
    return {"value": work["edge_features"] * reps / dt, "unit": "edge-features/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": f"{reps} full fwd+bwd step(s) of the same workload (n={wl.n}, nnz={wl.graph.nnz}), "
                      f"{dt:.1f} s in total; float64 oracle, OpenMP aggregation + BLAS dense products"}


def measure_peaks(B, torch) -> dict:
    """Measured ceilings next to the datasheet ones: a streaming read of a
    2 GiB array and back-to-back matrix-core products (gcn_peaks.h), each the
    best of a few launch shapes, timed with events on the launch stream."""
    stream = torch.cuda.current_stream()
    ev = lambda: torch.cuda.Event(enable_timing=True)

    def timed(fn, reps):
        fn()
        a, b = ev(), ev()
        torch.cuda.synchronize()
        a.record(stream)
        for _ in range(reps):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps

    n = (2 << 30) // 4
    x = torch.ones(n, dtype=torch.float32, device="cuda")
    sink = torch.empty(256 * 16384, dtype=torch.float32, device="cuda")
    best_bw, best_blocks = 0.0, 0
    for blocks in (2048, 4096, 8192, 16384):
        ms = timed(lambda: B.gcn_peak_stream_read(x, sink, blocks), 5)
        bw = n * 4 / (ms / 1e3) / 1e9
        if bw > best_bw:
            best_bw, best_blocks = bw, blocks
    del x
    out = {"stream_read_gbs": round(best_bw, 1), "stream_read_blocks": best_blocks}
    for prec, iters in (("f32", 4000), ("bf16", 4000)):
        best, bb = 0.0, 0
        for blocks in (256, 512, 1024):
            fl = [0.0]

            def run():
                fl[0] = B.gcn_peak_mfma(B.PREC[prec], blocks, iters, sink)
            ms = timed(run, 3)
            tf = fl[0] / (ms / 1e3) / 1e12
            if tf > best:
                best, bb = tf, blocks
        out[f"mfma_{prec}_tflops"] = round(best, 1)
        out[f"mfma_{prec}_blocks"] = bb
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--prec", default="f32", choices=["f32", "bf16"])
    ap.add_argument("--config", type=int, default=3)
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="minimum CPU time of the oracle baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-profile", action="store_true", help="skip the per-kernel event timing")
    ap.add_argument("--no-peaks", action="store_true", help="skip the measured machine ceilings")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="only run a plain device copy of this size (for counter calibration)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only: this build has no multi-GPU path "
              f"(asked for --gpus {args.gpus}, WORLD_SIZE={world}).", file=sys.stderr)
        sys.exit(2)

    import torch
    if args.copy_calibration_mib:
        n = args.copy_calibration_mib * (1 << 20) // 4
        a = torch.ones(n, dtype=torch.float32, device="cuda")
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_each_way": n * 4}))
        return

    from paper_1810_11899_amd import binding as B
    from paper_1810_11899_amd import synth
    from paper_1810_11899_amd.runner import StepRunner, step_work

    B.lib()
    prec = B.PREC[args.prec]
    wl = synth.config(args.config)
    spec = synth.CONFIGS[args.config]
    runner = StepRunner(wl, prec=prec)
    work = runner.work()
    stream = torch.cuda.current_stream()

    for _ in range(args.warmup):
        runner.step()
    torch.cuda.synchronize()

    if not args.no_profile:
        B.gcn_profile_reset()
        B.gcn_profile_enable(True)
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for _ in range(args.steps):
        runner.step()
    stop.record(stream)
    torch.cuda.synchronize()
    B.gcn_profile_enable(False)
    ms_total = start.elapsed_time(stop)
    ms_step = ms_total / args.steps
    ef_per_s = work["edge_features"] / (ms_step / 1e3)
    gflops = (work["gemm_flops"] + work["spmm_flops"]) / (ms_step / 1e3) / 1e9

    kernels = {}
    roof = None
    config_name = spec.name + ("" if args.prec == "f32" else "_bf16")
    if not args.no_profile:
        prof = B.gcn_profile_read_all()
        for name, (ms, launches, flops, bytes_) in prof.items():
            if launches == 0:
                continue
            e = {"ms_per_step": round(ms / args.steps, 4), "launches_per_step": launches / args.steps}
            if flops > 0 and name.startswith("gemm"):
                e["tflops"] = round(flops / (ms / 1e3) / 1e12, 2)
            if bytes_ > 0:
                e["gbs"] = round(bytes_ / (ms / 1e3) / 1e9, 1)
            kernels[name] = e
        dom = max(((n, v) for n, v in prof.items() if v[1] > 0), key=lambda kv: kv[1][0])
        name, (ms, launches, flops, bytes_) = dom
        per_launch_ms = ms / launches
        if name.startswith("gemm"):
            achieved = flops / (ms / 1e3) / 1e12
            peak = PEAK_TFLOPS[args.prec]
            roof = {"bound": "mfma", "kernel": name, "achieved": round(achieved, 2), "peak": peak,
                    "unit": "TFLOP/s", "frac": round(achieved / peak, 4)}
        else:
            achieved = bytes_ / (ms / 1e3) / 1e9
            roof = {"bound": "hbm", "kernel": name, "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                    "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4)}
        roof["avg_launch_ms"] = round(per_launch_ms, 4)
        roof["launches_per_step"] = launches / args.steps
        roof["traffic"] = traffic_for(name, config_name)
        spm = prof.get("spmm")
        if spm and spm[1]:
            kernels["spmm"]["hbm_frac_gather_model"] = round(spm[3] / (spm[0] / 1e3) / 1e9 / PEAK_HBM_GBS, 4)

    out = {
        "metric": METRIC, "value": round(ef_per_s, 1), "unit": "edge-features/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32" if args.prec == "f32" else "bf16",
        "data": "synthetic (seeded R-MAT subgraph, N(0,1) features, Glorot weights, uniform labels)",
        "config": {"workload": config_name, "n": wl.n, "nnz": wl.graph.nnz,
                   "layers": [list(d) for d in runner.dims],
                   "orders": ["aggregate_first" if o == B.GCN_AGGREGATE_FIRST else "transform_first"
                              for o in runner.orders],
                   "head": spec.head, "classes": spec.classes, "parallelism": "single GPU"},
        "gflops": round(gflops, 1),
        "edge_features_per_step": work["edge_features"], "gemm_gflop_per_step": work["gemm_flops"] / 1e9,
        "roofline": roof, "kernels": kernels,
    }
    if not args.no_peaks:
        peaks = measure_peaks(B, torch)
        out["measured_peaks"] = peaks
        if roof is not None:
            key = "stream_read_gbs" if roof["bound"] == "hbm" else f"mfma_{args.prec}_tflops"
            roof["measured_peak"] = peaks[key]
            roof["frac_of_measured_peak"] = round(roof["achieved"] / peaks[key], 4)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(args.config, synth, step_work, B, min_seconds=args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
