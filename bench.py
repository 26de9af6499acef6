#!/usr/bin/env python3
"""Benchmark: one fwd+bwd training step of a sampled-subgraph GCN on one MI355X.

Other workloads (--workload): the frontier sampler, the sampled-subgraph
training loop, and the 200-subgraph epoch stream; --config picks the other
layer workloads.

Workload (default): 2-layer GCN on a 65,536-vertex R-MAT subgraph (average
degree 50, 3,276,800 stored edges, mean-normalised CSR), H_in 65536x512,
hidden 512 per branch (concat 1024), linear PREDICT + softmax-CE over 100
classes; synthetic seeded inputs, random Glorot weights.  One step = CSR
transpose + both layers forward + loss head + both layers backward, inputs
resident in HBM.  Prints one JSON line.

  value        whole-step edge-features/s (sum over aggregation passes of
               nnz x width, divided by the step time)
  roofline     the kernel class with the most time in a second, profiled pass
               of the same steps, each launch timed with HIP events on its
               launch stream (library profiler); the timed pass that gives
               `value` runs without those events
  cpu_baseline the CPU oracle on the same workload, whole steps timed for at
               least --cpu-seconds on the host's cores
"""
import argparse
import hashlib
import json
import re
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
    """Hash of the source files the kernel class is built from, with comments
    and blank space left out (a comment edit does not make counters stale)."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_1810_11899_amd", "csrc")
    for f in KERNEL_SOURCES["gemm" if kernel.startswith("gemm") else "spmm"]:
        text = open(os.path.join(csrc, f), encoding="utf-8").read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
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


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(cfg: int, synth, step_work, B, min_seconds: float = 10.0, max_reps: int = 20,
                 threads: int = 0, self_loops: bool = False):
    """The CPU oracle on the same workload: whole fwd+bwd steps, repeated until
    at least `min_seconds` of CPU work have been timed (bounded by max_reps).
    threads > 0: that many threads for the oracle's aggregation and BLAS (a
    serial run is the analogue of the paper's single-core baseline)."""
    import contextlib
    import oracle
    limit = contextlib.nullcontext()
    prev = oracle.num_threads()
    if threads > 0:
        from threadpoolctl import threadpool_limits
        limit = threadpool_limits(limits=threads)
        oracle.set_num_threads(threads)
    try:
        with limit:
            return _cpu_baseline(cfg, synth, step_work, B, min_seconds, max_reps, self_loops)
    finally:
        if threads > 0:
            oracle.set_num_threads(prev)


def _cpu_baseline(cfg, synth, step_work, B, min_seconds, max_reps, self_loops=False):
    import oracle
    wl = synth.config(cfg, self_loops=self_loops)
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
            "kind": "oracle", "cpu_model": cpu_model(),
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


def measure_gather(B, torch, wl) -> dict:
    """Measured row-gather ceilings (gcn_peak_gather): the rate at which this
    GPU delivers gathered row bytes to the CUs, best over a few launch shapes.
      uniform_<R>B_<size>  uniformly random rows of R bytes from an array of
                           that size (64 MiB fits the 256 MB Infinity Cache;
                           4 GiB does not, so most rows come from HBM)
      csr_fp32_rows        the workload's CSR column indices in order, rows of
                           the float32 features (k = the first layer's width,
                           rounded up to a row size the probe takes)
      csr_bf16_rows        the same with bfloat16 rows (half the bytes)
    A 16 KiB array stays in every CU's L1, so its rate is the CU's
    vector-memory path with every row a hit: no gather of that row size with
    16-byte lane loads runs faster, and it is the ceiling the propagation
    kernels are measured against.  2 MiB sits in every XCD's 4 MB L2.  The
    csr_* cases are one aggregation pass's gathers in plain CSR order over
    all CUs (no slice schedule, no arithmetic, no CSR or output traffic): a
    reference point for what the kernels' schedules add, not a ceiling."""
    stream = torch.cuda.current_stream()
    blocks_list = (2048, 4096, 8192)
    sink = torch.empty(max(blocks_list) * 256, dtype=torch.float32, device="cuda")
    out = {}

    def best(X, row_bytes, idx):
        bb, best_gbs = 0, 0.0
        for blocks in blocks_list:
            B.gcn_peak_gather(X, row_bytes, idx, sink, blocks)
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            a.record(stream)
            for _ in range(3):
                B.gcn_peak_gather(X, row_bytes, idx, sink, blocks)
            b.record(stream)
            torch.cuda.synchronize()
            gbs = idx.numel() * row_bytes * 3 / (a.elapsed_time(b) / 1e3) / 1e9
            if gbs > best_gbs:
                best_gbs, bb = gbs, blocks
        return {"gbs": round(best_gbs, 1), "blocks": bb, "rows": int(idx.numel()), "row_bytes": row_bytes}

    g = torch.Generator(device="cuda")
    g.manual_seed(181011899)
    for row_bytes in (256, 512, 1024):
        for size, tag in ((16 << 10, "16KiB"), (2 << 20, "2MiB"), (64 << 20, "64MiB"), (4 << 30, "4GiB")):
            rows = size // row_bytes
            X = torch.ones((rows, row_bytes // 4), dtype=torch.float32, device="cuda")
            count = (2 << 30) // row_bytes        # 2 GiB gathered per launch
            idx = torch.randint(0, rows, (count,), dtype=torch.int32, device="cuda", generator=g)
            out[f"uniform_{row_bytes}B_{tag}"] = best(X, row_bytes, idx)
            del X, idx
    k = wl.layers[0].f_in
    idx = torch.from_numpy(wl.graph.indices).cuda()

    def probe_row(nbytes):   # the probe's row sizes: 16 B times a power of two up to 1 KB, 2 KB, 4 KB
        r = 16
        while r < nbytes and r < 4096:
            r *= 2
        return r
    rb = probe_row(4 * k)
    X = torch.ones((wl.n, rb // 4), dtype=torch.float32, device="cuda")
    out["csr_order_fp32_rows"] = best(X, rb, idx)
    rb = probe_row(2 * k)
    X16 = torch.ones((wl.n, rb // 2), dtype=torch.bfloat16, device="cuda")
    out["csr_order_bf16_rows"] = best(X16, rb, idx)
    del X, X16
    return out


def chase_latency_ns(B, torch, n: int, chains: int, steps: int = 4000, seed: int = 0) -> float:
    """Latency of one dependent load, ns, over an int32 random cycle of n
    elements walked by `chains` wavefronts at once (gcn_peak_chase)."""
    import numpy as np
    rng = np.random.default_rng(seed)
    perm = rng.permutation(n).astype(np.int64)
    nxt = np.empty(n, dtype=np.int32)
    nxt[perm] = np.roll(perm, -1).astype(np.int32)
    assert nxt.min() >= 0 and nxt.max() < n
    d_next = torch.from_numpy(nxt).cuda()
    sink = torch.empty(chains, dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()
    B.gcn_peak_chase(d_next, 200, chains, sink)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    a.record(stream)
    B.gcn_peak_chase(d_next, steps, chains, sink)
    b.record(stream)
    torch.cuda.synchronize()
    return a.elapsed_time(b) * 1e6 / steps


def bench_sampler(args, B, torch):
    """Frontier sampling (Sec. IV, Alg. 2-4) of S runs at once on a
    Reddit-shaped R-MAT training graph, then the induced subgraphs of the batch
    and one subgraph's feature gather.  One JSON line."""
    import numpy as np
    from paper_1810_11899_amd import synth
    from oracle import sampler as OS  # cpu_baseline leg only
    spec = synth.TRAINING_GRAPHS["reddit_like"]
    t0 = time.perf_counter()
    tg = synth.training_graph(**spec, seed=0)
    gen_s = time.perf_counter() - t0
    g = tg.graph
    m, n, cap, eta = 1000, 8000, 30, 2.0
    params = B.gcn_sampler_plan(g.indptr, m, n, eta=eta, cap=cap, seed=1)
    S = args.sampler_runs
    G = B.DeviceCSR.from_host(g.n, g.n, g.indptr, g.indices, g.vals)
    X = torch.from_numpy(tg.X).cuda()
    stream = torch.cuda.current_stream()
    ev = lambda: torch.cuda.Event(enable_timing=True)
    verts = torch.empty((S, n), dtype=torch.int32, device="cuda")
    counts = torch.empty(S, dtype=torch.int32, device="cuda")
    status = torch.empty(S, dtype=torch.int32, device="cuda")
    for w in range(args.warmup):
        B.gcn_frontier_sample(G, params, 10 ** 9 + w * S, S, verts, counts, status)
    torch.cuda.synchronize()
    a, b = ev(), ev()
    a.record(stream)
    for k in range(args.steps):
        B.gcn_frontier_sample(G, params, k * S, S, verts, counts, status)
    b.record(stream)
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / args.steps
    st = status.cpu().numpy()
    c = counts.cpu().numpy()
    sampled = float(c.sum())
    # induced subgraphs of the last batch, and the feature gather of one of them
    ws = B.Workspace("cuda")
    ib = B.InducedBatch(S, n, int(S * n * 30), "cuda")
    B.gcn_induce_subgraphs(G, verts, counts, ib, ws)
    torch.cuda.synchronize()
    if int(ib.status.item()) != 0:
        ib = B.InducedBatch(S, n, int(ib.edge_offsets[-1].item()), "cuda")
    a2, b2 = ev(), ev()
    a2.record(stream)
    B.gcn_induce_subgraphs(G, verts, counts, ib, ws)
    b2.record(stream)
    torch.cuda.synchronize()
    induce_ms = a2.elapsed_time(b2)
    n_sub = ib.n_sub.cpu().numpy()
    nnz_sub = np.diff(ib.edge_offsets.cpu().numpy())
    H0 = torch.empty((n, X.shape[1]), dtype=torch.float32, device="cuda")
    a3, b3 = ev(), ev()
    a3.record(stream)
    for _ in range(10):
        B.gcn_gather_rows(X, ib.vsub[0], int(n_sub[0]), H0)
    b3.record(stream)
    torch.cuda.synchronize()
    gather_ms = a3.elapsed_time(b3) / 10
    # latency bound: two dependent global loads per step, measured on a random
    # cycle the size of G's neighbour array, at the same concurrency
    lat = chase_latency_ns(B, torch, g.nnz, S)
    steps_per_run_s = (n - m) / (ms / 1e3)
    peak_steps = 1e9 / (2 * lat)
    out = {
        "metric": "frontier sampling (Dashboard, Alg. 2-4): sampled vertices/s",
        "value": round(sampled / (ms / 1e3), 1), "unit": "sampled vertices/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "int32", "data": "synthetic (seeded R-MAT training graph)",
        "config": {"workload": f"frontier_{tg.name}_m{m}_n{n}_cap{cap}_runs{S}", "n_vertices": g.n, "nnz": g.nnz,
                   "m": m, "n": n, "eta": eta, "cap": cap, "runs_per_launch": S,
                   "db_entries": params.db_entries, "ia_slots": params.ia_slots,
                   "lds_bytes_per_run": 12 * params.ia_slots + 2 * params.db_entries,
                   "parallelism": "single GPU"},
        "statuses": {B.SAMPLE_STATUS[int(k)]: int((st == k).sum()) for k in np.unique(st)},
        "subgraphs_per_s": round(S / (ms / 1e3), 1),
        "induce": {"ms_per_batch": round(induce_ms, 4), "subgraphs": S,
                   "mean_vertices": float(n_sub.mean()), "mean_edges": float(nnz_sub.mean())},
        "gather": {"ms_per_subgraph": round(gather_ms, 4), "rows": int(n_sub[0]), "width": int(X.shape[1]),
                   "gbs": round(2 * 4 * int(n_sub[0]) * X.shape[1] / (gather_ms / 1e3) / 1e9, 1)},
        "roofline": {"bound": "latency", "kernel": "frontier_sample", "achieved": round(steps_per_run_s, 1),
                     "peak": round(peak_steps, 1), "unit": "steps/s per run", "frac": round(steps_per_run_s / peak_steps, 4),
                     "dependent_load_ns": round(lat, 1), "traffic": None},
        "graph_generation_s": round(gen_s, 1),
    }
    if not args.no_cpu_baseline:
        reps, dt, tot = 0, 0.0, 0
        while dt < args.cpu_seconds and reps < 100000:
            t1 = time.perf_counter()
            v, _ = OS.frontier_sample(g.indptr, g.indices, m, n, params.db_entries, params.ia_slots, cap=cap,
                                      p=64, seed=1, sampler_id=reps)
            dt += time.perf_counter() - t1
            tot += v.size
            reps += 1
        out["cpu_baseline"] = {"value": round(tot / dt, 1), "unit": "sampled vertices/s", "cores": 1,
                               "cpu_model": cpu_model(),
                               "kind": "oracle",
                               "sample": f"{reps} runs of the same sampler on the same graph, {dt:.1f} s; "
                                         f"sequential C oracle (one thread)"}
    print(json.dumps(out), flush=True)


def _stream_subgraph(s: int):
    """Subgraph s of the epoch stream (a worker process draws it)."""
    from paper_1810_11899_amd import synth
    return synth.config(4, s=s)


STREAM_ORACLE_SUBSET = (0, 1, 2, 50, 100, 150, 198, 199)


def bench_stream(args, torch):
    """The epoch stream: fwd+bwd on each of `--stream-subgraphs` independent
    subgraphs (50,000 vertices, R-MAT, degree drawn from 30..50 per subgraph,
    3 layers 200 -> 2x512 -> 2x512 -> 2x512, softmax-CE over 50 classes), the
    device activations, gradients, workspace and streams reused across
    subgraphs.  The subgraphs are drawn on the host by a process pool (the
    analogue of Alg. 5's pool), then streamed: each goes through pinned host
    buffers on a copy stream into one of two device input slots while the
    previous subgraph's step runs on the compute stream.  value =
    edge-features / summed compute-stream step time; the end-to-end wall time
    of the pipelined stream (host buffers to finished steps, uploads
    included) is reported beside it, with the same stream through one input
    slot (uploads not overlapped) for comparison."""
    import numpy as np
    from concurrent.futures import ProcessPoolExecutor
    from paper_1810_11899_amd import synth
    from paper_1810_11899_amd.runner import EpochPipeline, StepRunner
    S = args.stream_subgraphs
    spec = synth.WORKLOADS[4]
    workers = max(1, min(16, len(os.sched_getaffinity(0))))
    # the worker processes are forked before this process first touches the
    # GPU; they only draw subgraphs with numpy
    import multiprocessing
    t0 = time.perf_counter()
    with ProcessPoolExecutor(max_workers=workers, mp_context=multiprocessing.get_context("fork")) as ex:
        subgraphs = []
        for s, wl in enumerate(ex.map(_stream_subgraph, range(S))):
            subgraphs.append(wl)
            if (s + 1) % 25 == 0:
                print(f"stream: {s + 1}/{S} subgraphs drawn", file=sys.stderr, flush=True)
    gen_s = time.perf_counter() - t0
    from paper_1810_11899_amd import binding as B
    B.lib()
    nnzs = [wl.graph.nnz for wl in subgraphs]
    cap = spec.n * spec.d_range[1]
    assert max(nnzs) <= cap
    symmetric = [B.gcn_csr_pattern_symmetric_host(wl.graph.indptr, wl.graph.indices) for wl in subgraphs]
    runner = StepRunner(subgraphs[0], prec=B.PREC[args.prec], nnz_capacity=cap)
    stream = torch.cuda.current_stream()
    losses = torch.zeros(S, dtype=torch.float32, device="cuda")

    def run(slots, timed):
        pipe = EpochPipeline(runner, cap, slots=slots, compute_stream=stream)
        for s in range(min(args.warmup, S)):
            pipe.submit(subgraphs[s], symmetric[s])
        torch.cuda.synchronize()
        evs, ef = [], 0.0
        t1 = time.perf_counter()
        for s, wl in enumerate(subgraphs):
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)] if timed else None
            runner.model.set_loss(losses[s:s + 1])
            pipe.submit(wl, symmetric[s], events=ev)
            evs.append(ev)
            ef += runner.work()["edge_features"]
        torch.cuda.synchronize()
        wall = time.perf_counter() - t1
        runner.model.set_loss(runner.loss)
        return wall, evs, ef, pipe.slots[0].bytes

    wall, evs, ef, _ = run(2, True)
    step_ms = [e[2].elapsed_time(e[3]) for e in evs]
    up_ms = [e[0].elapsed_time(e[1]) for e in evs]
    up_bytes = 0
    for wl in subgraphs:
        g = wl.graph
        up_bytes += 4 * (g.n + 1) + 8 * g.nnz + wl.H.nbytes + (wl.labels.nbytes if wl.labels is not None else 0)
    wall_1, _, _, _ = run(1, False)
    total_s = sum(step_ms) / 1e3
    work = runner.work()
    gpu_losses = losses.cpu().numpy()
    out = {
        "metric": "GCN layer fwd+bwd over an epoch stream of subgraphs: edge-features/s",
        "value": round(ef / total_s, 1), "unit": "edge-features/s", "n_gpus": 1, "steps": S,
        "warmup": min(args.warmup, S),
        "ms_per_step": round(1e3 * total_s / S, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": args.prec, "data": "synthetic (seeded R-MAT subgraphs, N(0,1) features, "
                                                      "Glorot weights shared by the stream, uniform labels)",
        "config": {"workload": spec.name + ("" if args.prec == "f32" else "_bf16"), "n": spec.n,
                   "subgraphs": S, "nnz_min": int(min(nnzs)), "nnz_max": int(max(nnzs)),
                   "nnz_mean": float(np.mean(nnzs)), "layers": [list(d) for d in runner.dims],
                   "parallelism": "single GPU"},
        "compute_stream_s_total": round(total_s, 4),
        "step_ms_min_median_max": [round(min(step_ms), 4), round(float(np.median(step_ms)), 4),
                                   round(max(step_ms), 4)],
        "gemm_gflop_last_subgraph": work["gemm_flops"] / 1e9,
        "end_to_end": {
            "what": "host-resident subgraphs to finished steps: pinned staging, uploads on a copy stream "
                    "into two input slots, steps on the compute stream",
            "wall_s": round(wall, 4), "edge_features_per_s": round(ef / wall, 1),
            "upload_gb": round(up_bytes / 1e9, 3), "upload_s_total_copy_stream": round(sum(up_ms) / 1e3, 4),
            "upload_gbs": round(up_bytes / (sum(up_ms) / 1e3) / 1e9, 1),
            "wall_s_one_slot": round(wall_1, 4),
            "note": "value is the compute-stream rate (inputs resident in HBM); this is the PCIe-inclusive rate"},
        "host_generation_s": round(gen_s, 1), "host_generation_workers": workers,
    }
    if not args.no_cpu_baseline:
        import oracle
        subset = [s for s in STREAM_ORACLE_SUBSET if s < S]
        dt, ef_c, errs = 0.0, 0.0, []
        for s in subset:
            wl = subgraphs[s]
            t1 = time.perf_counter()
            r = oracle.step(wl)
            dt += time.perf_counter() - t1
            errs.append(abs(float(gpu_losses[s]) - r.loss) / abs(r.loss))
            L = len(wl.layers)
            dims = [(l.f_in, l.h) for l in wl.layers]
            need = [li > 0 for li in range(L)]
            from paper_1810_11899_amd.runner import step_work
            ef_c += step_work(wl.n, wl.graph.nnz, dims, runner.orders, need, spec.classes)["edge_features"]
        out["cpu_baseline"] = {"value": round(ef_c / dt, 1), "unit": "edge-features/s",
                               "cores": oracle.num_threads(), "kind": "oracle", "cpu_model": cpu_model(),
                               "sample": f"subgraphs {list(subset)} of the stream, {dt:.1f} s, "
                                         f"{dt / len(subset):.2f} s per subgraph; the whole stream would take "
                                         f"about {dt / len(subset) * S:.0f} s (x{S} extrapolated)",
                               "loss_rel_err_max_vs_gpu": float(max(errs))}
    print(json.dumps(out), flush=True)


PHASES = {  # the time breakdown of Sec. VI-C (Fig. 3): sampling, propagation, weights
    "sampling": ("frontier_sample", "induce_subgraphs"),
    "feature_propagation": ("spmm", "spmm_fixup", "spmm_bf16"),
    "weight_application": ("gemm_nn", "gemm_tn", "gemm_nt", "splitk_reduce", "gemm_nn_bf16", "gemm_tn_bf16",
                           "gemm_nt_bf16", "gemm_nt_bf16_big", "gemm_nt_bf16_big_masked", "gemm_tn_bf16_big"),
}


def bench_train(args, B, torch):
    """Alg. 5 on one GPU: frontier-sampled subgraphs of a Reddit-shaped
    training graph, 2-layer GCN (602 -> 2x128 -> 2x128, softmax-CE over 41
    classes), ADAM; pools of subgraphs sampled on a side stream while the
    compute stream trains.  One JSON line."""
    import numpy as np
    import oracle
    from oracle import optim as OO
    from oracle import sampler as OS
    from paper_1810_11899_amd import synth
    from paper_1810_11899_amd.train import SamplerConfig, Trainer
    spec = synth.TRAINING_GRAPHS["reddit_like"]
    tg = synth.training_graph(**spec, seed=0)
    dims = [(602, 128), (256, 128)]
    cfg = SamplerConfig(m=1000, n=8000, eta=2.0, cap=30, pool=args.pool, seed=1)
    tr = Trainer(tg, dims, cfg, lr=0.01, prec=B.PREC[args.prec])
    for _ in range(args.train_warmup):
        tr.step()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    verts = edges = 0
    host = 0.0
    wait0 = tr.wait_s
    t0 = time.perf_counter()
    a.record(stream)
    for _ in range(args.train_iters):
        th = time.perf_counter()
        ns, nnz = tr.step()
        host += time.perf_counter() - th
        verts += ns
        edges += nnz
    b.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    K = args.train_iters
    if not args.no_profile:   # a second, profiled pass for the per-kernel breakdown
        B.gcn_profile_reset()
        B.gcn_profile_enable(True)
        for _ in range(K):
            tr.step()
        torch.cuda.synchronize()
        B.gcn_profile_enable(False)
    ms_it = wall * 1e3 / K
    losses = tr.loss_history()
    ef = 0.0   # edge-features of the iterations (aggregation widths of the orders used)
    for (f_in, h), o, li in zip(dims, tr.orders, range(len(dims))):
        if o == B.GCN_AGGREGATE_FIRST:
            ef += f_in + (min(f_in, h) if li > 0 else 0)
        else:
            ef += 2 * h
    phases, kernels = {}, {}
    if not args.no_profile:
        prof = B.gcn_profile_read_all()
        for name, (ms, launches, flops, bytes_) in prof.items():
            if launches:
                kernels[name] = {"ms_per_iteration": round(ms / K, 4), "launches_per_iteration": launches / K}
        for ph, names in PHASES.items():
            phases[ph] = round(sum(prof[nm][0] for nm in names if nm in prof) / K, 4)
        phases["other"] = round(sum(v["ms_per_iteration"] for v in kernels.values()) - sum(phases.values()), 4)
    out = {
        "metric": "GCN training with frontier sampling (Alg. 5): iterations/s",
        "value": round(K / wall, 2), "unit": "iterations/s", "n_gpus": 1, "steps": K,
        "warmup": args.train_warmup, "ms_per_step": round(ms_it, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": args.prec, "data": "synthetic (seeded R-MAT training graph, random labels)",
        "config": {"workload": f"train_{tg.name}_602-128-128_ce41_m1000_n8000_pool{args.pool}",
                   "n_vertices": tg.graph.n, "nnz": tg.graph.nnz, "layers": [list(d) for d in dims],
                   "orders": ["aggregate_first" if o == B.GCN_AGGREGATE_FIRST else "transform_first"
                              for o in tr.orders], "parallelism": "single GPU"},
        "mean_subgraph_vertices": verts / K, "mean_subgraph_edges": edges / K,
        "edge_features_per_s": round(edges * ef / wall, 1),
        "compute_stream_ms_per_iteration": round(a.elapsed_time(b) / K, 4),
        # host time spent issuing one iteration (library calls return once
        # their kernels are queued), without the waits for pool refills: the
        # host runs ahead of the GPU until the next pool is not ready yet, so
        # those waits are the GPU's backpressure.  Near ms_per_step would mean
        # the host paces the GPU.
        "host_issue_ms_per_iteration": round((host - (tr.wait_s - wait0)) * 1e3 / K, 4),
        "host_wait_for_pools_ms_per_iteration": round((tr.wait_s - wait0) * 1e3 / K, 4),
        "phases_ms_per_iteration": phases, "kernels": kernels,
        "loss_first_last": [float(losses[0]), float(losses[-1])],
    }
    if not args.no_cpu_baseline:
        # the oracle pipeline on the same graph: sample, induce, fwd/bwd, ADAM
        g = tg.graph
        P = {k: v.astype(np.float64) for k, v in tr.model.host_tensors().items()}
        M = {k: np.zeros_like(v) for k, v in P.items()}
        V = {k: np.zeros_like(v) for k, v in P.items()}
        sp = synth.Spec("train", 0, "rmat", 0, dims, "ce", tg.classes)
        reps, dt = 0, 0.0
        while dt < args.cpu_seconds and reps < 50:
            t1 = time.perf_counter()
            v, _ = OS.frontier_sample(g.indptr, g.indices, cfg.m, cfg.n, tr.params.db_entries, tr.params.ia_slots,
                                      cap=cfg.cap, p=64, seed=cfg.seed, sampler_id=10 ** 6 + reps)
            vs, ip, ix, vals = OS.induce(g.indptr, g.indices, v)
            layers = [synth.Layer(P[f"W_self{i}"].astype(np.float32), P[f"W_neigh{i}"].astype(np.float32),
                                  P[f"bias{i}"].astype(np.float32)) for i in range(len(dims))]
            wl = synth.Workload(sp, 0, synth.Graph(vs.size, ip, ix, vals), OS.gather_rows(tg.X, vs), layers,
                                W_pred=P["W_pred"].astype(np.float32), b_pred=P["b_pred"].astype(np.float32),
                                labels=OS.gather_rows(tg.labels, vs))
            r = oracle.step(wl)
            grads = {"W_pred": r.dW_pred, "b_pred": r.db_pred}
            for i in range(len(dims)):
                grads[f"W_self{i}"], grads[f"W_neigh{i}"], grads[f"bias{i}"] = r.dW_self[i], r.dW_neigh[i], r.db[i]
            for k in P:
                P[k], M[k], V[k] = OO.adam(P[k], grads[k], M[k], V[k], reps + 1, 0.01)
            dt += time.perf_counter() - t1
            reps += 1
        out["cpu_baseline"] = {"value": round(reps / dt, 4), "unit": "iterations/s", "cores": oracle.num_threads(),
                               "cpu_model": cpu_model(),
                               "kind": "oracle",
                               "sample": f"{reps} iterations of the oracle pipeline (sampler, induced subgraph, "
                                         f"float64 fwd/bwd, ADAM) on the same graph, {dt:.1f} s"}
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--prec", default="f32", choices=["f32", "bf16"])
    ap.add_argument("--config", type=int, default=3)
    ap.add_argument("--index-bits", type=int, default=32, choices=[16, 32],
                    help="column-index width of the subgraph's CSR (16: uint16, at most 65,536 vertices)")
    ap.add_argument("--self-loops", action="store_true", help="add a self-connection to every vertex")
    ap.add_argument("--orders", default="tuned", choices=["tuned", "rule"],
                    help="layer groupings: measured per workload (tuned) or gcn_layer_pick_order's width rule")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="minimum CPU time of the oracle baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-profile", action="store_true", help="skip the per-kernel event timing")
    ap.add_argument("--no-peaks", action="store_true", help="skip the measured machine ceilings")
    ap.add_argument("--no-variants", action="store_true",
                    help="skip the bfloat16 variant that the default (float32, 65,536-vertex) run also measures")
    ap.add_argument("--workload", default="step", choices=["step", "sampler", "train", "stream"],
                    help="step: one fwd+bwd step of the layer (default); sampler: the frontier sampler; "
                         "train: the sampled-subgraph training loop")
    ap.add_argument("--pool", type=int, default=256, help="subgraphs per pool refill (train)")
    ap.add_argument("--stream-subgraphs", type=int, default=200, help="subgraphs of the epoch stream (stream)")
    ap.add_argument("--train-iters", type=int, default=600)
    ap.add_argument("--train-warmup", type=int, default=40)
    ap.add_argument("--sampler-runs", type=int, default=512, help="sampler runs per launch")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="only run a plain device copy of this size (for counter calibration)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only: the library has no multi-GPU path "
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

    if args.workload == "stream":   # forks its generator processes before loading the library
        bench_stream(args, torch)
        return
    from paper_1810_11899_amd import binding as B
    from paper_1810_11899_amd import synth
    from paper_1810_11899_amd.runner import step_work

    B.lib()
    if args.workload == "sampler":
        bench_sampler(args, B, torch)
        return
    if args.workload == "train":
        bench_train(args, B, torch)
        return
    wl = synth.config(args.config, self_loops=args.self_loops)
    # a bfloat16 step keeps its activations as bfloat16 end to end (the
    # configuration of the bfloat16 variant below), where the library allows
    # it (an output gradient that arrives unmasked needs the float32 Y)
    fo = args.prec == "f32" or args.config != 3
    out = bench_step(args, args.prec, wl, B, torch, synth, index_bits=args.index_bits, float_outputs=fo)
    out["float_outputs"] = fo
    variants = {}
    if args.config == 3 and args.prec == "f32" and args.index_bits == 32 and not args.no_variants:
        # the bfloat16-operand variant of the same workload, and the float32
        # step with uint16 column indices, measured the same way
        keys = ("value", "unit", "ms_per_step", "dtype", "gflops", "step_ms_min_median", "host_issue_ms_per_step",
                "roofline", "kernels", "csr_bytes", "index_bits")
        # the bfloat16 step keeps activations as bfloat16 end to end (each
        # layer's output only as the next consumer's bfloat16 operand rows)
        v = bench_step(args, "bf16", wl, B, torch, synth, float_outputs=False)
        variants["bf16"] = {k: v[k] for k in keys if k in v}
        variants["bf16"]["float_outputs"] = False
        variants["bf16"]["config"] = {k: v["config"][k] for k in ("workload", "orders", "order_choice", "order_step_ms")
                                      if k in v["config"]}
        v = bench_step(args, "f32", wl, B, torch, synth, index_bits=16,
                       orders=[B.GCN_AGGREGATE_FIRST if o == "aggregate_first" else B.GCN_TRANSFORM_FIRST
                               for o in out["config"]["orders"]])
        variants["uint16"] = {k: v[k] for k in keys if k in v and k != "kernels"}
        variants["uint16"]["kernels"] = {k: v["kernels"][k] for k in ("spmm", "transpose_symmetric")
                                         if k in v["kernels"]}
        variants["uint16"]["config"] = {"workload": v["config"]["workload"]}
        variants["uint16"]["csr_bytes_saved"] = out["csr_bytes"] - v["csr_bytes"]
    if variants:
        out["variants"] = variants
    if not args.no_peaks:
        peaks = measure_peaks(B, torch)
        peaks["gather"] = measure_gather(B, torch, wl)
        out["measured_peaks"] = peaks
        for o in [out] + list(variants.values()):
            roof = o.get("roofline")
            if roof is not None and roof["bound"] == "gather":
                ref = peaks["gather"].get(f"uniform_{roof['gather_row_bytes']}B_16KiB")
                if ref:
                    roof["peak"] = ref["gbs"]
                    roof["frac"] = round(roof["achieved"] / ref["gbs"], 4)
            elif roof is not None:
                prec_o = "f32" if o["dtype"] == "f32" else "bf16"
                key = "stream_read_gbs" if roof["bound"] == "hbm" else f"mfma_{prec_o}_tflops"
                roof["measured_peak"] = peaks[key]
                roof["frac_of_measured_peak"] = round(roof["achieved"] / peaks[key], 4)
            spmm_vs_gather(o, peaks["gather"])
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(args.config, synth, step_work, B, min_seconds=args.cpu_seconds,
                                           self_loops=args.self_loops)
        if args.config in (0, 1, 2):   # the serial oracle as well (small workloads only)
            out["cpu_baseline_serial"] = cpu_baseline(args.config, synth, step_work, B,
                                                      min_seconds=args.cpu_seconds, max_reps=5, threads=1,
                                                      self_loops=args.self_loops)
    print(json.dumps(out), flush=True)


def spmm_vs_gather(o: dict, gather: dict):
    """The aggregation kernels against the measured gather rates: the rate at
    which they deliver gathered row bytes (one row of the aggregated width per
    stored edge) over the probe's rate for random rows of the size each
    kernel's lane groups read, from an L2-resident array (the ceiling: every
    row an L2 hit), from one that fits only the Infinity Cache, and from one
    that comes mostly from HBM (above 1: the kernel's locality beats random
    rows from that level)."""
    # per lane group on the XCD-sliced schedules both kernels gather
    # 512-byte pieces of a row (128 float32 or 256 bfloat16 columns)
    for cls, row in (("spmm", 512), ("spmm_bf16", 512)):
        k = o.get("kernels", {}).get(cls)
        if not k or "gather_gbs" not in k:
            continue
        for tag, name in (("16KiB", "frac_of_l1_gather_ceiling"), ("2MiB", "vs_l2_gather"),
                          ("64MiB", "vs_infinity_cache_gather"), ("4GiB", "vs_hbm_gather")):
            ref = gather.get(f"uniform_{row}B_{tag}")
            if ref:
                k[name] = round(k["gather_gbs"] / ref["gbs"], 4)


def bench_step(args, prec_name: str, wl, B, torch, synth, index_bits: int = 32, orders=None,
               float_outputs: bool = True) -> dict:
    """Time one workload's fwd+bwd step at one precision: the whole step with
    events around the timed steps (no per-kernel events in them), then a
    second, profiled pass of as many steps for the per-kernel breakdown and
    the roofline of the dominant kernel class."""
    from paper_1810_11899_amd.runner import StepRunner
    prec = B.PREC[prec_name]
    spec = wl.spec
    if orders is None:
        orders = None if args.orders == "rule" else "tuned"
    runner = StepRunner(wl, prec=prec, index_bits=index_bits, orders=orders, float_outputs=float_outputs)
    timings = getattr(runner, "order_timings", None)
    work = runner.work()
    stream = torch.cuda.current_stream()

    for _ in range(args.warmup):
        runner.step()
    torch.cuda.synchronize()

    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    host = 0.0
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    start.record(stream)
    for i in range(args.steps):
        th = time.perf_counter()
        runner.step()
        host += time.perf_counter() - th
        marks[i].record(stream)   # per-step times (no synchronization in the loop)
    stop.record(stream)
    torch.cuda.synchronize()
    step_ms = sorted([start.elapsed_time(marks[0])] +
                     [marks[i - 1].elapsed_time(marks[i]) for i in range(1, args.steps)])
    if not args.no_profile:
        B.gcn_profile_reset()
        B.gcn_profile_enable(True)
        for _ in range(args.steps):
            runner.step()
        torch.cuda.synchronize()
        B.gcn_profile_enable(False)
    ms_total = start.elapsed_time(stop)
    ms_step = ms_total / args.steps
    ef_per_s = work["edge_features"] / (ms_step / 1e3)
    gflops = (work["gemm_flops"] + work["spmm_flops"]) / (ms_step / 1e3) / 1e9

    kernels = {}
    roof = None
    config_name = wl.spec.name + ("" if prec_name == "f32" else "_bf16") + ("_uint16" if index_bits == 16 else "")
    if not args.no_profile:
        prof = B.gcn_profile_read_all()
        for name, (ms, launches, flops, bytes_) in prof.items():
            if launches == 0:
                continue
            e = {"ms_per_step": round(ms / args.steps, 4), "launches_per_step": launches / args.steps}
            if flops > 0 and name.startswith("gemm"):
                e["tflops"] = round(flops / (ms / 1e3) / 1e12, 2)
                # fraction of the time the class would take at the datasheet
                # peaks (matrix cores or moving its bytes once, the larger)
                t_bound = max(flops / (PEAK_TFLOPS[prec_name] * 1e12), bytes_ / (PEAK_HBM_GBS * 1e9))
                e["roofline_time_frac"] = round(t_bound / (ms / 1e3), 4)
            if bytes_ > 0:
                e["gbs"] = round(bytes_ / (ms / 1e3) / 1e9, 1)
            kernels[name] = e
        # dominant kernel: the one with the most time (the large-tile bf16
        # product's two classes, plain and masked epilogue, are one kernel)
        groups = {}
        for n, v in prof.items():
            if v[1] == 0:
                continue
            key = "gemm_nt_bf16_big" if n.startswith("gemm_nt_bf16_big") else n
            groups[key] = tuple(a + b for a, b in zip(groups.get(key, (0.0, 0, 0.0, 0.0)), v))
        name, (ms, launches, flops, bytes_) = max(groups.items(), key=lambda kv: kv[1][0])
        per_launch_ms = ms / launches
        if name.startswith("gemm"):
            # a product is bound by the matrix cores or by moving its operands
            # and output once, whichever takes longer at the datasheet peaks
            peak = PEAK_TFLOPS[prec_name]
            t_mfma = flops / (peak * 1e12)
            t_hbm = bytes_ / (PEAK_HBM_GBS * 1e9)
            if t_mfma >= t_hbm:
                achieved = flops / (ms / 1e3) / 1e12
                roof = {"bound": "mfma", "kernel": name, "achieved": round(achieved, 2), "peak": peak,
                        "unit": "TFLOP/s", "frac": round(achieved / peak, 4)}
            else:
                achieved = bytes_ / (ms / 1e3) / 1e9
                roof = {"bound": "hbm", "kernel": name, "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                        "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4)}
            roof["mfma_frac"] = round(flops / (ms / 1e3) / 1e12 / peak, 4)
            roof["hbm_frac_algorithmic"] = round(bytes_ / (ms / 1e3) / 1e9 / PEAK_HBM_GBS, 4)
        elif name in ("spmm", "spmm_bf16"):
            # a gather: bound by the CU's vector-memory path, which takes every
            # gathered 16-byte lane vector wherever it hits (L2, Infinity
            # Cache, HBM).  `achieved` is the gathered row bytes per second
            # (one row of the aggregated width per stored edge); the peak is
            # the measured rate of random row gathers of the size its lane
            # groups read (on the sliced schedules, 512-byte pieces: 128
            # float32 or 256 bfloat16 columns) from an L1-resident array
            # (filled in once the machine ceilings are measured).  The gather-model bytes over
            # 8 TB/s are kept beside it: above 1, since the caches serve most
            # gathers, so not a DRAM fraction.
            esz = 4 if name == "spmm" else 2
            achieved = work["edge_features"] * esz * args.steps / (ms / 1e3) / 1e9
            roof = {"bound": "gather", "kernel": name, "achieved": round(achieved, 1), "peak": None,
                    "unit": "GB/s", "frac": None, "peak_source": "measured L1-resident random-row gather",
                    "gather_row_bytes": 512,
                    "hbm_frac_gather_model": round(bytes_ / (ms / 1e3) / 1e9 / PEAK_HBM_GBS, 4)}
        else:
            achieved = bytes_ / (ms / 1e3) / 1e9
            roof = {"bound": "hbm", "kernel": name, "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                    "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4)}
        roof["avg_launch_ms"] = round(per_launch_ms, 4)
        roof["launches_per_step"] = launches / args.steps
        roof["traffic"] = traffic_for(name, config_name)
        for cls, esz in (("spmm", 4), ("spmm_bf16", 2)):
            spm = prof.get(cls)
            if not (spm and spm[1]):
                continue
            t_s = spm[0] / 1e3
            # bytes the aggregation delivers to the CUs under the gather model
            # (one row of the aggregated width per stored edge, plus the CSR
            # and the output rows): a cache-served rate, not a DRAM one
            kernels[cls]["gather_model_gbs"] = round(spm[3] / t_s / 1e9, 1)
            kernels[cls]["gather_gbs"] = round(work["edge_features"] * esz * args.steps / t_s / 1e9, 1)
            # compulsory model: every feature row read once, plus CSR and
            # output: a lower bound on DRAM traffic, as a fraction of 8 TB/s
            passes = spm[1] / args.steps
            k_sum = work["edge_features"] / max(wl.graph.nnz, 1)
            comp = args.steps * (wl.n * k_sum * (esz + 4) + passes * (8.0 * wl.graph.nnz + 4.0 * (wl.n + 1)))
            kernels[cls]["hbm_frac_compulsory_model"] = round(comp / t_s / 1e9 / PEAK_HBM_GBS, 4)

    return {
        "metric": METRIC, "value": round(ef_per_s, 1), "unit": "edge-features/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32" if prec_name == "f32" else "bf16",
        "data": "synthetic (seeded R-MAT subgraph, N(0,1) features, Glorot weights, uniform labels)",
        "csr_bytes": runner.csr_bytes(), "index_bits": index_bits,
        "config": {"workload": config_name, "n": wl.n, "nnz": wl.graph.nnz,
                   "layers": [list(d) for d in runner.dims],
                   "orders": ["aggregate_first" if o == B.GCN_AGGREGATE_FIRST else "transform_first"
                              for o in runner.orders],
                   "head": spec.head, "classes": spec.classes, "parallelism": "single GPU",
                   "order_choice": "measured" if timings else ("given" if isinstance(orders, list) else "width rule"),
                   **({"order_step_ms": {"+".join("af" if o == B.GCN_AGGREGATE_FIRST else "tf" for o in k):
                                         round(v, 4) for k, v in timings.items()}} if timings else {})},
        "gflops": round(gflops, 1),
        "step_ms_min_median": [round(step_ms[0], 4), round(step_ms[len(step_ms) // 2], 4)],
        "host_issue_ms_per_step": round(host * 1e3 / args.steps, 4),
        "edge_features_per_step": work["edge_features"], "gemm_gflop_per_step": work["gemm_flops"] / 1e9,
        "roofline": roof, "kernels": kernels,
    }


if __name__ == "__main__":
    main()
