#!/usr/bin/env python3
"""Benchmark of the dual-sparse SpMSpV on one MI355X.

Default workload: y = W x with W 4096 x 4096 fp16 at 70 % unstructured
weight sparsity and x (Laplace) thresholded to 70 % activation sparsity,
batch 1 -- the "70 % dual sparsity" point.  One step = one celty_spmspv call
(selection, compressed-column walk, LDS accumulation, merge, fp16 output: a
single kernel launch).

Cold cache: the encoded matrix is copied to enough distinct device buffers
that the steps, rotating over them, read at least 1 GiB (beyond the 256 MiB
Infinity Cache and the L2s) between two reads of the same copy -- counted in
the bytes a call reads, its active columns, not in the copy's size -- so
every step streams its weights from HBM (--cold-bytes sets the 1 GiB).
Before every timed replay of the K steps (outside the timed events) 1 GiB
of another buffer is read, so the first copies a replay reads are not left
in a cache by the replay before it, whatever the step count, and one call
on a spare copy re-warms the code and the small buffers.

Timing: HIP events on the launch stream around the K steps, which are
launched back to back and all enqueued while the GPU is still busy with the
cache-clearing reads before the start event, so neither the host nor a graph
launch sits inside the timed region; the same K steps as one graph replay
are reported beside it.

Printed (one JSON line): µs per SpMSpV (value, lower is better), effective
GB/s on algorithmic bytes, the roofline of the kernel (the timing above; the
profiler's kernel durations and HBM traffic from the committed records), the
time of a plain read of the same bytes in one launch (read_floor), the dense
fp16 GEMV (torch F.linear, i.e. hipBLASLt/rocBLAS) on the same shape under
the same cold protocol and timing, the floor of a near-empty kernel, eager
per-call times, and the CPU oracle timed on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0   # MI355X HBM3E, published
METRIC = "µs/SpMSpV + effective HBM GB/s (% peak), 4096×4096 at 70% dual sparsity"
COLD_BYTES = 1 << 30
KERNEL_SOURCE = os.path.join(ROOT, "paper_2608_01536_amd", "csrc", "spmspv.hip")
PROFILES = os.path.join(ROOT, "profiles")
CALIBRATION_BYTES = 256 << 20


def traffic_file(workload_key: str) -> str:
    return os.path.join(PROFILES, f"spmspv_{workload_key}_traffic.json")


def kernel_trace_file(workload_key: str) -> str:
    return os.path.join(PROFILES, f"spmspv_{workload_key}_kernel_trace.json")


def kernel_source_code(text: str) -> str:
    """The kernel source with comments removed and whitespace collapsed
    (string and character literals kept as they are)."""
    out, i, n = [], 0, len(text)
    while i < n:
        ch = text[i]
        if text.startswith("//", i):
            j = text.find("\n", i)
            i = n if j < 0 else j
        elif text.startswith("/*", i):
            j = text.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        elif ch in "\"'":
            j = i + 1
            while j < n and text[j] != ch:
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        else:
            out.append(ch)
            i += 1
    return " ".join("".join(out).split())


def kernel_source_sha() -> str:
    """sha256 of the kernel source's code: a comment edit does not void the
    counter profiles, a code edit does."""
    import hashlib
    with open(KERNEL_SOURCE, encoding="utf-8") as f:
        return hashlib.sha256(kernel_source_code(f.read()).encode()).hexdigest()


def measured_traffic(workload_key: str):
    """HBM bytes per launch from the committed counter profile, or None when
    the profile is missing, for another workload, or older than the kernel."""
    try:
        with open(traffic_file(workload_key)) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_sha256") != kernel_source_sha() or rec.get("workload_key") != workload_key:
        return None
    return rec.get("traffic_bytes_per_launch")


def recorded_kernel_trace(workload_key: str):
    """Dispatch durations of the SpMSpV kernel from the committed kernel-trace
    record, or None when it is missing, for another workload, or older than
    the kernel."""
    try:
        with open(kernel_trace_file(workload_key)) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_sha256") != kernel_source_sha() or rec.get("workload_key") != workload_key:
        return None
    return rec


def record_kernel_trace(workload_key: str, trace_csv: str, command: str) -> int:
    """Turns a rocprofv3 --kernel-trace CSV of this benchmark into the record
    recorded_kernel_trace() reads: the mean and median duration of the
    SpMSpV dispatches of the timed (queued) replays: the last 5 * steps
    dispatches, which also hold four of the single re-warm calls between the
    replays; the warm-up, eager and graph-replay calls come first.  Under the
    tracer the host's launches slow down enough that the queued kernels run
    with idle time between them, each on its own; the tracer's timestamps
    for graph-replayed kernels are not used, as they run the end of one
    kernel into the start of the next."""
    import csv
    import statistics
    durs = []
    with open(trace_csv) as f:
        for row in csv.DictReader(f):
            if "spmspv_kernel" in row["Kernel_Name"]:
                durs.append((int(row["Start_Timestamp"]), int(row["End_Timestamp"]) - int(row["Start_Timestamp"])))
    if not durs:
        print("record-kernel-trace: no SpMSpV dispatches in the trace", file=sys.stderr)
        return 1
    durs.sort()
    steps = int(command.split("--steps")[1].split()[0]) if "--steps" in command else 1000
    tail = [d for _, d in durs[-5 * steps:]]
    rec = {"workload_key": workload_key, "kernel_source_sha256": kernel_source_sha(),
           "dispatches": len(tail), "mean_ns": round(statistics.fmean(tail), 1),
           "median_ns": float(statistics.median(tail)), "min_ns": min(tail), "max_ns": max(tail),
           "command": command}
    with open(kernel_trace_file(workload_key), "w") as f:
        json.dump(rec, f, indent=1)
        f.write("\n")
    print(json.dumps(rec))
    return 0


def _counter_per_dispatch(csv_path: str, name_parts) -> list:
    """Per-dispatch sums of a rocprofv3 counter CSV for kernels whose name
    contains any of name_parts."""
    import csv
    vals = {}
    with open(csv_path) as f:
        for row in csv.DictReader(f):
            if any(n in row["Kernel_Name"] for n in name_parts):
                vals[row["Dispatch_Id"]] = vals.get(row["Dispatch_Id"], 0.0) + float(row["Counter_Value"])
    return list(vals.values())


def record_traffic(workload_key: str, paths, commands) -> int:
    """Turns four rocprofv3 --pmc runs (FETCH_SIZE and WRITE_SIZE of this
    benchmark, then of the plain copy) into HBM bytes per launch: each
    counter's median per SpMSpV dispatch, scaled by the bytes the copy moved
    over what the same counter read for it.  Writes the record that
    measured_traffic() reads."""
    import statistics
    fetch, write, cfetch, cwrite = paths
    k_f = _counter_per_dispatch(fetch, ["spmspv_kernel"])
    k_w = _counter_per_dispatch(write, ["spmspv_kernel"])
    c_f = _counter_per_dispatch(cfetch, ["elementwise_kernel", "copy"])
    c_w = _counter_per_dispatch(cwrite, ["elementwise_kernel", "copy"])
    if not (k_f and k_w and c_f and c_w):
        print("record-traffic: a counter file has no matching dispatches", file=sys.stderr)
        return 1
    fk, wk = statistics.median(k_f), statistics.median(k_w)
    cf, cw = statistics.median(c_f), statistics.median(c_w)
    ff, wf = CALIBRATION_BYTES / (cf * 1024.0), CALIBRATION_BYTES / (cw * 1024.0)
    rec = {"workload_key": workload_key, "kernel_source_sha256": kernel_source_sha(),
           "fetch_kib_per_dispatch": fk, "write_kib_per_dispatch": wk, "dispatches": [len(k_f), len(k_w)],
           "copy_fetch_kib": cf, "copy_write_kib": cw, "copy_bytes": CALIBRATION_BYTES,
           "fetch_factor": ff, "write_factor": wf,
           "traffic_bytes_per_launch": int(round(fk * 1024.0 * ff + wk * 1024.0 * wf)),
           "commands": commands}
    with open(traffic_file(workload_key), "w") as f:
        json.dump(rec, f, indent=1)
        f.write("\n")
    print(json.dumps(rec))
    return 0


def _encode_layer(job):
    """Host worker: draw the 7 projections of one layer (its own seeds, x and
    tau) and encode them; also the stacked encodings of the projections that
    share an x (q/k/v, gate/up), which the fused schedule launches as one
    taller matrix.  Returns plain host data for the parent to upload."""
    cfg, layer, as_, fused = job
    import paper_2608_01536_amd as celty
    import workloads

    probs = workloads.layer_problems(cfg, 0, layer, as_)
    encs = [celty.celty_encode(p.W, p.mask, celty.default_tile_rows(*p.W.shape)) for p in probs]
    alg = [algorithmic_bytes_from_encoding(e, p.x, p.tau)[0] for e, p in zip(encs, probs)]
    groups = _x_groups(cfg)
    xs = {workloads.CONFIGS[cfg]["layers"][g[0]].x_group: probs[g[0]].x for g in groups}
    taus = [p.tau for p in probs]
    stacked = []
    if fused:
        for g in groups:
            if len(g) == 1:
                stacked.append(None)
                continue
            Wst = np.concatenate([probs[i].W for i in g], axis=0)
            Mst = np.concatenate([probs[i].mask for i in g], axis=0)
            stacked.append(celty.celty_encode(Wst, Mst, celty.default_tile_rows(*Wst.shape)))
            del Wst, Mst
    dense_shapes = [p.W.shape for p in probs]
    del probs
    return layer, encs, stacked, xs, taus, alg, dense_shapes


def _x_groups(cfg):
    """Runs of consecutive projections that read the same x."""
    import workloads
    groups, prev = [], None
    for i, pr in enumerate(workloads.CONFIGS[cfg]["layers"]):
        if pr.x_group == prev:
            groups[-1].append(i)
        else:
            groups.append([i])
        prev = pr.x_group
    return groups


def sequence_bench(args) -> int:
    """One decode step of config 3, 4 or 5: the 7 projections of every layer,
    timed as one HIP graph per schedule.  Every layer is its own draw (seeds
    per layer and projection, its own activations and thresholds), encoded on
    the host by a pool of worker processes and uploaded to HBM, so a step
    streams all of its distinct weights from HBM.  When the step reads less
    than the cold threshold (1 GiB) the graph runs it several times over,
    each time on its own device copy of the layers (and the caches are
    cleared before each timed replay)."""
    import concurrent.futures as cf
    import multiprocessing as mp

    import workloads

    cfg = args.sequence
    c = workloads.CONFIGS[cfg]
    as_ = args.seq_as if args.seq_as is not None else (c["as_"] if not isinstance(c["as_"], tuple) else 60)
    n_layers = args.layers or c["n_layers"]
    fused_on = not args.no_fused
    groups = _x_groups(cfg)
    names = [pr.name for pr in c["layers"]]
    workers = max(1, min(args.workers or 16, len(os.sched_getaffinity(0)), n_layers))
    print(f"[sequence] config {cfg}: {n_layers} distinct layers at as{as_:g}, {workers} host workers",
          file=sys.stderr, flush=True)
    # the pool starts before this process touches the GPU
    pool = cf.ProcessPoolExecutor(max_workers=workers, mp_context=mp.get_context("fork"))
    futs = [pool.submit(_encode_layer, (cfg, l, as_, fused_on)) for l in range(n_layers)]

    import torch
    import torch.nn.functional as F

    import paper_2608_01536_amd as celty

    dev = torch.device("cuda:0")
    layers = [None] * n_layers          # per layer: device encodings of the 7 projections
    fused = [None] * n_layers           # per layer: one device encoding per x-group
    xs = [None] * n_layers              # per layer: device x of each projection
    taus = [None] * n_layers
    alg_step = 0.0
    algs = [None] * n_layers            # per layer: algorithmic bytes of the 7 projections
    stored_step = 0
    dense_shapes = None
    done = 0
    for fut in cf.as_completed(futs):
        layer, encs, stacked, xh, tl, alg, dense_shapes = fut.result()
        layers[layer] = [e.to_device(dev) for e in encs]
        if fused_on:
            fused[layer] = [layers[layer][g[0]] if st is None else st.to_device(dev)
                            for g, st in zip(groups, stacked)]
        xd = {k: torch.from_numpy(v.view(np.int16)).to(dev) for k, v in xh.items()}
        xs[layer] = [xd[pr.x_group] for pr in c["layers"]]
        taus[layer] = tl
        algs[layer] = alg
        alg_step += sum(alg)
        stored_step += sum(stored_bytes(e) for e in encs)
        del encs, stacked
        done += 1
        if done % 8 == 0 or done == n_layers:
            print(f"[sequence] {done}/{n_layers} layers encoded and uploaded", file=sys.stderr, flush=True)
    pool.shutdown()
    flush = CacheFlush(torch)
    ys = [torch.empty(pr.M, dtype=torch.int16, device=dev) for pr in c["layers"]]
    wss = [celty.new_workspace(W, dev) for W in layers[0]]
    bws = [celty.new_batch_workspace([layers[0][i] for i in g], dev) for g in groups]
    if fused_on:
        fys = [torch.empty(f.M, dtype=torch.int16, device=dev) for f in fused[0]]
        fws = [celty.new_workspace(f, dev) for f in fused[0]]
    # a step that reads less than the cold threshold is repeated within one
    # graph, each repeat on its own device copy of every layer, so that no
    # layer is read again before COLD_BYTES of other reads
    reps = max(1, -(-COLD_BYTES // max(1, int(alg_step))))
    lay_r = [layers] + [[[e.clone_to() for e in L] for L in layers] for _ in range(reps - 1)]
    fus_r = [fused] + [[[e.clone_to() for e in F_] for F_ in fused] for _ in range(reps - 1)] if fused_on else None

    def step_sequential(s):
        for l in range(n_layers):
            L = lay_r[s % reps][l]
            for i in range(len(L)):
                celty.celty_spmspv(L[i], xs[l][i], taus[l][i], ys[i], wss[i])

    def step_batched(s):
        for l in range(n_layers):
            L = lay_r[s % reps][l]
            for g, w in zip(groups, bws):
                celty.celty_spmspv_batch([L[i] for i in g], [xs[l][i] for i in g], [taus[l][i] for i in g],
                                         [ys[i] for i in g], w)

    def step_fused(s):
        for l in range(n_layers):
            for j, g in enumerate(groups):
                celty.celty_spmspv(fus_r[s % reps][l][j], xs[l][g[0]], taus[l][g[0]], fys[j], fws[j])

    out = {"sequence": cfg, "name": c["name"], "activation_sparsity_pct": as_, "layers": n_layers,
           "distinct_layers": True, "data": "synthetic",
           "alg_bytes_per_step": int(alg_step), "stored_bytes_per_step": int(stored_step),
           "graph_repeats_of_the_step": reps}
    schedules = [("sequential", step_sequential, len(names)), ("batched", step_batched, len(groups))]
    if fused_on:
        schedules.append(("fused", step_fused, len(groups)))
    for label, fn, launches in schedules:
        for i in range(2):
            fn(i)
        torch.cuda.synchronize()
        us, samples = time_graph(torch, fn, reps, replays=3, flush=flush)
        out[label] = {"us_per_step": round(us, 2), "launches_per_step": n_layers * launches,
                      "GBps": round(alg_step / us / 1e3, 1),
                      "pct_peak_hbm": round(100 * alg_step / us / 1e3 / PEAK_HBM_GBPS, 2)}
        print(f"[sequence] {label}: {us:.1f} us/step", file=sys.stderr, flush=True)
    if not args.no_dense:
        dense = {}
        for (M, K) in sorted(set(dense_shapes)):
            Wf = torch.zeros(M, K, dtype=torch.float16, device=dev)
            Wf.normal_(0.0, 0.02)
            nd = max(2, -(-COLD_BYTES // (2 * M * K)))
            dc = [Wf] + [Wf.clone() for _ in range(nd - 1)]
            xd = torch.zeros(1, K, dtype=torch.float16, device=dev)
            for j in range(5):
                F.linear(xd, dc[j % nd])
            dense[(M, K)], _ = time_graph(torch, lambda j: F.linear(xd, dc[j % nd]), max(nd, 100), replays=3,
                                          flush=flush)
            del dc, Wf
            torch.cuda.empty_cache()
        d_step = n_layers * sum(dense[sh] for sh in dense_shapes)
        out["dense_gemv_us_per_step"] = round(d_step, 2)
        out["dense_note"] = ("sum over the layer's shapes of F.linear fp16 batch-1 times (cold copies, caches "
                             "cleared before each timed replay) x layers")
        out["speedup_vs_dense"] = {k: round(d_step / out[k]["us_per_step"], 3) for k, _, _ in schedules}
    if fused_on and not args.no_read_floor:
        # the fused schedule's launches as plain reads of their algorithmic
        # bytes (one launch per x-group and layer, in order, distinct bytes)
        del layers, fused, lay_r, fus_r
        torch.cuda.empty_cache()
        sizes = [[max(16, int(sum(algs[l][i] for i in g)) // 16 * 16) for g in groups] for l in range(n_layers)]
        per_step = sum(sum(s) for s in sizes)
        buf = torch.empty(reps * per_step, dtype=torch.uint8, device=dev)   # distinct bytes per repeat
        buf.fill_(1)
        sink = torch.empty(1024, dtype=torch.int32, device=dev)

        def step_read(s):
            off = (s % reps) * per_step
            for l in range(n_layers):
                for nb in sizes[l]:
                    celty.celty_bench_stream_read(buf[off:off + nb], nb, sink, 512, 512)
                    off += nb

        step_read(0)
        torch.cuda.synchronize()
        us, _ = time_graph(torch, step_read, reps, replays=3, flush=flush)
        out["read_floor"] = {"us_per_step": round(us, 2), "GBps": round(alg_step / us / 1e3, 1),
                             "pct_peak_hbm": round(100 * alg_step / us / 1e3 / PEAK_HBM_GBPS, 2),
                             "fused_vs_floor": round(us / out["fused"]["us_per_step"], 3),
                             "op": "the fused schedule's launches as plain streaming reads of their algorithmic "
                                   "bytes (celty_bench_stream_read, 512 x 512 lanes)"}
        print(f"[sequence] read floor: {us:.1f} us/step", file=sys.stderr, flush=True)
    print(json.dumps(out))
    return 0


def format_study(args) -> int:
    """Host only: stored size of a 4096x4096 fp16 matrix in this library's
    RLC-CSC (4-bit runs, Section 3.2) against a bitmap format and dense fp16,
    across weight sparsity (the paper's compression-efficiency comparison).
    RLC-CSC is counted three ways: 2.5 B per stored entry (values + runs, the
    paper's accounting), plus the 8-entry alignment of each segment, plus the
    group pointers.  The bitmap is its theoretical size: one bit per position
    and 2 B per non-zero."""
    import paper_2608_01536_amd as celty
    import workloads

    M = K = 4096
    dense = 2 * M * K
    rows = []
    for ws in (10, 20, 30, 40, 50, 60, 70, 80, 90):
        p = workloads.make_problem(2, M, K, ws, 50, "laplace", seed=0, proj=workloads.PROJ_IDS["w"])
        for R in ([512, 4096] if ws in (50, 70) else [512]):
            enc = celty.celty_encode(p.W, p.mask, R)
            entries = 2.5 * (enc.n_nnz + enc.n_pad)
            aligned = 2 * 8 * enc.n_groups + 4 * enc.n_groups
            stored = aligned + 4 * (enc.T * K + 1)
            bitmap = M * K / 8.0 + 2.0 * enc.n_nnz
            rows.append({"weight_sparsity_pct": ws, "R": R, "nnz": int(enc.n_nnz), "padding": int(enc.n_pad),
                         "rlc_entry_ratio": round(entries / dense, 4), "rlc_aligned_ratio": round(aligned / dense, 4),
                         "rlc_stored_ratio": round(stored / dense, 4), "bitmap_ratio": round(bitmap / dense, 4)})
            print(json.dumps(rows[-1]), flush=True)
    return 0


def encode_throughput(args) -> int:
    """Host only: throughput of the library's RLC-CSC encoder (offline in the
    paper, Section 3.2) on the benchmark matrices, in dense entries scanned
    and stored entries written per second, for several thread counts."""
    import paper_2608_01536_amd as celty
    import workloads

    cpus = len(os.sched_getaffinity(0))
    for (M, K, ws) in ((4096, 4096, 70), (4096, 4096, 50), (28672, 8192, 50)):
        p = workloads.make_problem(2, M, K, ws, 50, "laplace", seed=0, proj=workloads.PROJ_IDS["w"])
        R = celty.default_tile_rows(M, K)
        for threads in sorted({1, 4, cpus}):
            best = float("inf")
            for _ in range(3):
                t = time.perf_counter()
                enc = celty.celty_encode(p.W, p.mask, R, n_threads=threads)
                best = min(best, time.perf_counter() - t)
            print(json.dumps({"M": M, "K": K, "weight_sparsity_pct": ws, "R": R, "threads": threads,
                              "seconds": round(best, 4), "dense_entries_per_s": round(M * K / best / 1e6, 1),
                              "stored_entries_per_s": round(enc.n_entries / best / 1e6, 1),
                              "unit": "millions per second", "host_cpus": cpus}), flush=True)
    return 0


def copy_calibration() -> int:
    """A plain device copy of CALIBRATION_BYTES (reads and writes that many
    bytes once): run under the FETCH_SIZE / WRITE_SIZE counters to scale them."""
    import torch
    a = torch.ones(CALIBRATION_BYTES, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": CALIBRATION_BYTES, "copies": 3}))
    return 0


def algorithmic_bytes_from_encoding(enc, x: np.ndarray, tau: float) -> tuple:
    """B_alg = 2.5 * E_A + 2K + 2M from the encoded arrays the kernel reads.

    E_A counts, over the active columns, every entry up to the last stored
    value of each segment (stored values + run-length padding); the trailing
    8-entry alignment is excluded.  Returns (B_alg, E_A, groups_A)."""
    active = np.abs(x.astype(np.float32)) > np.float32(tau)
    G = enc.n_groups
    gptr = enc.gptr.astype(np.int64)
    if G == 0:
        return 2.0 * enc.K + 2.0 * enc.M, 0, 0
    vals = enc.values.reshape(G, 8)
    nz = vals & np.uint16(0x7FFF) != 0
    last_in_group = np.where(nz.any(axis=1), 7 - np.argmax(nz[:, ::-1], axis=1), -1)
    last_entry = np.where(last_in_group >= 0, 8 * np.arange(G) + last_in_group, -1)
    seg_len = np.diff(gptr)
    nonempty = np.flatnonzero(seg_len > 0)
    seg_last = np.full(gptr.size - 1, -1, dtype=np.int64)
    seg_last[nonempty] = np.maximum.reduceat(last_entry, gptr[nonempty])
    n_seg = np.where(seg_last >= 0, seg_last - 8 * gptr[:-1] + 1, 0).reshape(enc.T, enc.K)
    e_a = int(n_seg[:, active].sum())
    g_a = int(seg_len.reshape(enc.T, enc.K)[:, active].sum())
    return 2.5 * e_a + 2.0 * enc.K + 2.0 * enc.M, e_a, g_a


def fetched_bytes_from_encoding(enc, g_a: int, plan: dict, group_bytes: int = 20) -> tuple:
    """Bytes the kernel's own loads and stores request (merge atomics aside).

    compressed: every 8-entry group of an active column's segments (16 B of
    values + 4 B of runs, or 16 B of row offsets in the 16-bit row layout:
    group_bytes; the trailing alignment entries included) plus the
    group pointers (each workgroup reads the Kc + 1 pointers of its slice in
    its row tile, so T * (K + KC) words).  total adds x and the column maxima
    of each workgroup's slice (2 + 2 B per column, once per row tile) and y
    (2 B * M).  Returns (compressed, total)."""
    KC = -(-enc.K // plan["cols_per_block"])
    compressed = group_bytes * g_a + 4 * enc.T * (enc.K + KC)
    return compressed, compressed + 4 * enc.T * enc.K + 2 * enc.M


def stored_bytes(enc) -> int:
    return 2 * enc.values.size + 4 * enc.runs.size + 4 * enc.gptr.size + 2 * enc.colmax.size


def time_loop(torch, fn, steps: int) -> float:
    """Wall time per call (µs) of `steps` back-to-back calls, HIP events."""
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    s.record()
    for i in range(steps):
        fn(i)
    e.record()
    torch.cuda.synchronize()
    return s.elapsed_time(e) * 1e3 / steps


class CacheFlush:
    """Reads COLD_BYTES of other device memory with ordinary (allocating)
    loads: run before a timed replay (outside its events), it evicts whatever
    the previous replay left in the L2s and the Infinity Cache and leaves only
    clean lines behind.  (Overwriting the buffer instead leaves dirty lines
    whose write-back then competes with the first calls of the replay: at 20
    calls per replay it added 10-20 % to the measured time.)"""

    def __init__(self, torch):
        self.torch = torch
        self.buf = torch.ones(COLD_BYTES // 8, dtype=torch.int64, device="cuda")

    def __call__(self):
        self.torch.amax(self.buf.view(-1, 4096), dim=1)


def time_graph(torch, fn, steps: int, replays: int = 5, flush=None, rewarm=None) -> tuple:
    """Capture `steps` calls in one HIP graph; return (µs per call of the timed
    replay, per-replay µs-per-call samples).  Replaying removes host launch
    overhead, so each call's time is its kernel plus the graph's inter-kernel
    gap (and, amortised over the steps, the replay's own start).  flush, if
    given, runs before every replay, outside the timed events; then rewarm, if
    given: one untimed call on data the replay does not read, which restores
    the kernel's code and the small per-call buffers to the caches, as in a
    running decode loop, while the timed calls' weights stay cold.  A short
    device-side wait precedes the start event, so that the replay's kernels
    are already queued when timing starts (otherwise the host's submission of
    a replay can leave the GPU idle inside the timed region)."""
    g = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        for i in range(steps):
            fn(i)
    if flush is not None:
        flush()
    g.replay()
    torch.cuda.synchronize()
    samples = []
    for _ in range(replays):
        if flush is not None:
            flush()
        if rewarm is not None:
            rewarm()
        torch.cuda._sleep(200000)   # about 0.1 ms of device time, outside the events
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        g.replay()
        e.record()
        torch.cuda.synchronize()
        samples.append(s.elapsed_time(e) * 1e3 / steps)
    del g
    return float(np.median(samples)), samples


def cold_copies(enc, p) -> int:
    """Copies of enc to rotate so that a copy is read again only after at
    least COLD_BYTES of other reads.  Counted in the bytes one call reads
    (its algorithmic bytes: the active columns' entries, x and y), not in the
    copy's stored size: a call reads the same active columns of every copy,
    so a rotation sized by stored bytes would bring each copy's read part
    back after far less traffic than COLD_BYTES, within reach of the
    Infinity Cache."""
    read = algorithmic_bytes_from_encoding(enc, p.x, p.tau)[0]
    return max(2, -(-COLD_BYTES // max(1, int(read))))


def time_queued(torch, fn, steps: int, replays: int = 5, flush=None, rewarm=None) -> tuple:
    """µs per call of `steps` calls launched one after another on the launch
    stream and all queued before the timed region starts: before each timed
    replay (outside the events) the GPU streams reads of the cache-clearing
    buffer for as long as the host needs to enqueue the replay (rather than
    idling: after milliseconds of idling, the next milliseconds of this
    kernel run measurably slower, while a plain read does not), then the
    rewarm call and the short wait of time_graph; the GPU then runs the
    steps back to back, with no host gap and no graph launch inside the
    events.  (A graph replay adds a fixed cost of about 11 µs between its
    start event and its first kernel, the same for a one-element fill as for
    this kernel; queued launches have about 2.5 µs.)  Returns (median µs per
    call, per-replay samples, info): info holds the host's µs per launch and
    whether every replay's launches were all enqueued before the GPU reached
    them (queued_ahead)."""
    torch.cuda.synchronize()
    n = max(1, min(steps, 50))
    t0 = time.perf_counter()
    for i in range(n):
        fn(i)
    host_us = (time.perf_counter() - t0) * 1e6 / n
    torch.cuda.synchronize()
    wait_us = 200.0 + 2.0 * host_us * steps
    if flush is not None:
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        flush()
        e.record()
        torch.cuda.synchronize()
        busy_us = max(1.0, s.elapsed_time(e) * 1e3)
        reads = max(1, int(wait_us // busy_us) + 1)
    else:   # no cache clearing (a hot run): an idle wait instead
        busy_us, reads = wait_us, 0
    samples, ahead = [], True
    for _ in range(replays):
        for _ in range(reads):
            flush()
        if reads == 0:
            torch.cuda._sleep(int(wait_us * 2400))   # shader-clock cycles, at most 2.4 GHz
        if rewarm is not None:
            rewarm()
        torch.cuda._sleep(200000)   # as time_graph, about 0.1 ms
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        t0 = time.perf_counter()
        for i in range(steps):
            fn(i)
        enq = (time.perf_counter() - t0) * 1e6
        e.record()
        torch.cuda.synchronize()
        ahead = ahead and enq < max(1, reads) * busy_us
        samples.append(s.elapsed_time(e) * 1e3 / steps)
    return float(np.median(samples)), samples, {"host_us_per_launch": round(host_us, 2), "queued_ahead": ahead,
                                                "reads_before_each_replay": reads}


def cold_spmspv(torch, celty, enc, p, launch, steps: int, warmup: int, hot: bool = False, flush=None) -> dict:
    """µs per celty_spmspv_ex call (time_queued, and time_graph beside it) on
    rotated device copies of enc (cold_copies of them, so every call streams
    its part of W from HBM; with flush, the caches are also cleared before
    every timed replay, then one untimed call on a spare copy that the replay
    does not read re-warms the code and the small buffers)."""
    dev = torch.device("cuda:0")
    ncopies = 1 if hot else cold_copies(enc, p)
    base = enc.to_device(dev)
    # ncopies rotated by the steps, plus one spare (the last) for the re-warm call
    copies = [base] + [base.clone_to() for _ in range(ncopies)]
    x = torch.from_numpy(p.x.view(np.int16)).to(dev)
    y = torch.empty(enc.M, dtype=torch.int16, device=dev)
    ws = celty.new_workspace(base, dev)

    def step(i):
        # stream = None: the binding launches on torch's current stream, which
        # is the capture stream while a graph is being recorded
        celty.celty_spmspv_ex(copies[i % ncopies], x, p.tau, y, ws, launch)

    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    eager_us = time_loop(torch, step, steps)
    # the same eager loop through prepared calls (arguments checked once)
    preps = [celty.PreparedSpMSpV(c, x, y, ws, launch) for c in copies]
    eager_prepared_us = time_loop(torch, lambda i: preps[i % ncopies](p.tau), steps)
    del preps
    # the timed region: the steps launched back to back on the launch stream,
    # all enqueued while the GPU still runs the cache-clearing reads; one step
    # is exactly one kernel launch
    spare = copies[-1]
    rewarm = None if hot else (lambda: celty.celty_spmspv_ex(spare, x, p.tau, y, ws, launch))
    # first, for comparison, the same steps as one HIP graph replay
    g_us, g_samples = time_graph(torch, step, steps, flush=None if hot else flush, rewarm=rewarm)
    us, samples, info = time_queued(torch, step, steps, flush=None if hot else flush, rewarm=rewarm)
    out = {"us": us, "samples": samples, "queued": info, "graph_us": g_us, "graph_samples": g_samples,
           "eager_us": eager_us, "eager_prepared_us": eager_prepared_us, "copies": ncopies}
    del copies, base
    torch.cuda.empty_cache()
    return out


READ_SHAPES = ((256, 1024), (512, 512), (1024, 256))


def read_floor(torch, celty, nbytes: float, steps: int, flush=None) -> dict:
    """What the memory system gives one launch that reads nbytes: the
    library's measurement reference (celty_bench_stream_read, a plain
    streaming read) timed on rotated cold buffers under the same
    protocol as the product, best of three launch shapes."""
    nb = max(16, int(nbytes) // 16 * 16)
    nc = max(2, -(-COLD_BYTES // nb))
    bufs = [torch.empty(nb, dtype=torch.uint8, device="cuda") for _ in range(nc + 1)]   # the last one spare
    for b in bufs:
        b.fill_(1)
    sink = torch.empty(1024, dtype=torch.int32, device="cuda")
    best = None
    for blocks, threads in READ_SHAPES:
        us, _, _ = time_queued(torch, lambda i: celty.celty_bench_stream_read(bufs[i % nc], nb, sink, blocks, threads),
                               steps, replays=3, flush=flush,
                               rewarm=lambda: celty.celty_bench_stream_read(bufs[-1], nb, sink, blocks, threads))
        if best is None or us < best[0]:
            best = (us, blocks, threads)
    del bufs
    torch.cuda.empty_cache()
    return {"us": round(best[0], 3), "bytes": nb, "GBps": round(nb / best[0] / 1e3, 1),
            "launch": f"{best[1]} workgroups x {best[2]} lanes",
            "op": "celty_bench_stream_read: one launch streaming the same number of bytes, 16-byte loads"}


def cold_dense(torch, F, p, steps: int, hot: bool = False, flush=None) -> dict:
    """The dense reference: F.linear fp16 at batch 1 on the masked W and the
    thresholded x, same cold rotation, cache clearing, re-warm call on a spare
    copy and queued-launch timing."""
    dev = torch.device("cuda:0")
    M, K = p.W.shape
    Wf = torch.from_numpy(np.where(p.mask != 0, p.W, np.float16(0))).to(dev)
    nd = 1 if hot else max(2, -(-COLD_BYTES // (2 * M * K)))
    dcopies = [Wf] + [Wf.clone() for _ in range(nd)]   # nd rotated, the last one spare
    xd = torch.from_numpy(np.where(np.abs(p.x.astype(np.float32)) > p.tau, p.x, np.float16(0))).to(dev)[None]
    for i in range(20):
        F.linear(xd, dcopies[i % nd])
    dense_us, _, _ = time_queued(torch, lambda i: F.linear(xd, dcopies[i % nd]), steps,
                                 flush=None if hot else flush,
                                 rewarm=None if hot else (lambda: F.linear(xd, dcopies[-1])))
    del dcopies, Wf
    torch.cuda.empty_cache()
    return {"us": round(dense_us, 3), "GBps": round((2 * M * K + 2 * K + 2 * M) / dense_us / 1e3, 1),
            "op": "torch.nn.functional.linear fp16, batch 1 (hipBLASLt/rocBLAS)", "copies": nd,
            "timing": "queued launches, as the SpMSpV"}


VARIANT_SHAPES = ((4096, 4096, 70, 70), (4096, 4096, 30, 30), (5120, 5120, 60, 60), (13824, 5120, 60, 60),
                  (8192, 8192, 50, 60), (28672, 8192, 50, 40), (28672, 8192, 50, 60))


def variant_study(args) -> int:
    """The kernel's variants on the same products, in one process: the
    paper's 4-bit runs with the plain tile (the default), the same with the
    XOR-swizzled tile, 16-bit row offsets (no reconstruction) and the runs in
    lane-interleaved order.  Per shape: the three encodings on rotated cold
    copies, the four y checked bit-equal, then three rounds (alternating
    order) of queued-launch timing with the caches cleared before every
    replay; one JSON line per shape with the median µs of each variant."""
    import torch

    import paper_2608_01536_amd as celty
    import workloads

    dev = torch.device("cuda:0")
    flush = CacheFlush(torch)
    names = ("rlc", "swizzle", "rows16", "interleaved")
    for (M, K, ws, as_) in VARIANT_SHAPES:
        R = celty.default_tile_rows(M, K)
        p = workloads.make_problem(2, M, K, ws, as_, "laplace", seed=0, proj=workloads.PROJ_IDS["w"])
        encs = {"rlc": celty.celty_encode(p.W, p.mask, R),
                "rows16": celty.celty_encode(p.W, p.mask, R, layout=celty.LAYOUT_ROWS16),
                "interleaved": celty.celty_encode(p.W, p.mask, R, layout=celty.LAYOUT_INTERLEAVED)}
        copies = {}
        for k, e in encs.items():
            base = e.to_device(dev)
            # rotated copies, plus a spare (the last) for the re-warm call
            copies[k] = [base] + [base.clone_to() for _ in range(cold_copies(e, p))]
        copies["swizzle"] = copies["rlc"]
        launch = {v: (0, 0, 0, 1 if v == "swizzle" else 0) for v in names}
        x = torch.from_numpy(p.x.view(np.int16)).to(dev)
        y = torch.empty(M, dtype=torch.int16, device=dev)
        wsb = celty.new_workspace(copies["rlc"][0], dev)
        ys = []
        for v in names:
            celty.celty_spmspv_ex(copies[v][0], x, p.tau, y, wsb, launch[v])
            torch.cuda.synchronize()
            ys.append(y.cpu().numpy().copy())
        same = all(np.array_equal(ys[0], o) for o in ys[1:])
        res = {v: [] for v in names}
        for rnd in range(3):
            for v in (names if rnd % 2 == 0 else names[::-1]):
                cs = copies[v]
                n_rot = len(cs) - 1
                us, _, _ = time_queued(torch, lambda i, cs=cs, v=v: celty.celty_spmspv_ex(cs[i % n_rot], x, p.tau, y,
                                                                                         wsb, launch[v]),
                                       args.steps, replays=3, flush=flush,
                                       rewarm=lambda cs=cs, v=v: celty.celty_spmspv_ex(cs[-1], x, p.tau, y, wsb,
                                                                                       launch[v]))
                res[v].append(us)
        b_alg = algorithmic_bytes_from_encoding(encs["rlc"], p.x, p.tau)[0]
        med = {v: round(float(np.median(res[v])), 3) for v in names}
        print(json.dumps({"study": "kernel variants", "shape": f"{M}x{K}", "ws": ws, "as": as_, "R": R,
                          "us": med, "y_bit_equal": same, "algorithmic_bytes": b_alg,
                          "stored_bytes": {k: stored_bytes(e) for k, e in encs.items()}, "steps": args.steps}),
              flush=True)
        del copies, encs
        torch.cuda.empty_cache()
        if not same:
            return 1
    return 0


PAPER_SHAPES = ((4096, 4096), (4096, 11008), (5120, 5120), (5120, 13824), (7168, 7168), (7168, 28672))


def paper_shapes(args) -> int:
    """The six layer shapes of the paper's kernel evaluation (LLaMA-2-7B,
    LLaMA-2-13B and OPT-30B projections, Section 5) at 30, 50 and 70 % dual
    sparsity (weight = activation sparsity), each against the dense fp16
    GEMV under the same cold protocol; one JSON line per point, then the mean
    speedup per sparsity level (the paper reports its own means as context).
    The GPU test suite checks these same problems against the oracle."""
    import torch
    import torch.nn.functional as F

    import paper_2608_01536_amd as celty
    import workloads

    flush = CacheFlush(torch)
    speed = {}
    for pct in (30, 50, 70):
        for (M, K) in PAPER_SHAPES:
            p = workloads.make_problem(2, M, K, pct, pct, "laplace", seed=0, proj=workloads.PROJ_IDS["w"])
            R = celty.default_tile_rows(M, K)
            enc = celty.celty_encode(p.W, p.mask, R)
            plan = celty.celty_spmspv_plan(enc, None)
            b_alg, _, g_a = algorithmic_bytes_from_encoding(enc, p.x, p.tau)
            comp, _ = fetched_bytes_from_encoding(enc, g_a, plan)
            sp_ = cold_spmspv(torch, celty, enc, p, None, args.steps, args.warmup, flush=flush)
            d = cold_dense(torch, F, p, args.steps, flush=flush)
            speed.setdefault(pct, []).append(d["us"] / sp_["us"])
            print(json.dumps({"M": M, "K": K, "dual_sparsity_pct": pct, "R": R, "launch": plan,
                              "us": round(sp_["us"], 3), "alg_GBps": round(b_alg / sp_["us"] / 1e3, 1),
                              "pct_peak_alg": round(100 * b_alg / sp_["us"] / 1e3 / PEAK_HBM_GBPS, 2),
                              "pct_peak_fetched": round(100 * comp / sp_["us"] / 1e3 / PEAK_HBM_GBPS, 2),
                              "dense_us": d["us"], "speedup_vs_dense": round(d["us"] / sp_["us"], 3)}),
                  flush=True)
    print(json.dumps({"paper_shapes_mean_speedup_vs_dense": {str(k): round(float(np.mean(v)), 3)
                                                             for k, v in speed.items()},
                      "paper_shapes_max_speedup_vs_dense": {str(k): round(float(np.max(v)), 3)
                                                            for k, v in speed.items()},
                      "shapes": [f"{M}x{K}" for M, K in PAPER_SHAPES], "data": "synthetic"}))
    return 0


def cpu_baseline(p, budget_s: float) -> dict:
    """The CPU oracle as it stands, on this host's cores, over a bounded sample."""
    from oracle import spmspv as ref
    try:
        from threadpoolctl import threadpool_info
        threads = max([d.get("num_threads", 1) for d in threadpool_info()] + [1])
    except Exception:
        threads = 1
    runs, t0 = 0, time.perf_counter()
    best = float("inf")
    while True:
        a = time.perf_counter()
        ref.spmspv_dense_fp64(p.W, p.mask, p.x, p.tau)
        best = min(best, time.perf_counter() - a)
        runs += 1
        if time.perf_counter() - t0 > budget_s or runs >= 1000:
            break
    total = time.perf_counter() - t0
    # the oracle's second evaluation (fp64 CSC over the active columns, the
    # CSC matrix built from W and the mask inside each call, as it stands)
    runs2, t2 = 0, time.perf_counter()
    while True:
        ref.spmspv_csc_fp64(p.W, p.mask, p.x, p.tau)
        runs2 += 1
        if time.perf_counter() - t2 > budget_s / 2 or runs2 >= 1000:
            break
    total2 = time.perf_counter() - t2
    M, K = p.W.shape
    return {"value": round(total / runs * 1e6, 1), "unit": "µs/SpMSpV", "cores": int(threads),
            "kind": "oracle", "best_us": round(best * 1e6, 1),
            "sample": f"{runs} calls of the fp64 dense masked GEMV oracle on the same {M}x{K} problem "
                      f"({total:.1f} s), BLAS threads={threads}, host cpus={len(os.sched_getaffinity(0))}",
            "csc_fp64": {"value": round(total2 / runs2 * 1e6, 1), "unit": "µs/SpMSpV",
                         "sample": f"{runs2} calls of the oracle's fp64 CSC evaluation ({total2:.1f} s)"}}


def main() -> int:
    global COLD_BYTES
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1000)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--R", type=int, default=0, help="tile height (0 = library default)")
    ap.add_argument("--cols", type=int, default=0, help="columns per workgroup (0 = auto)")
    ap.add_argument("--waves", type=int, default=0, help="wavefronts per workgroup (0 = auto)")
    ap.add_argument("--ws", type=float, default=70.0, help="weight sparsity %%")
    ap.add_argument("--as", dest="as_", type=float, default=70.0, help="activation sparsity %%")
    ap.add_argument("--M", type=int, default=4096)
    ap.add_argument("--K", type=int, default=4096)
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--no-read-floor", action="store_true",
                    help="skip the plain-read reference of the same bytes (celty_bench_stream_read)")
    ap.add_argument("--sigma", type=float, default=0.0,
                    help="outlier input features: per-feature scales exp(sigma*N(0,1)) on W's columns and x, "
                         "per-row magnitude pruning (0 = the uniform-mask workload)")
    ap.add_argument("--hot", action="store_true", help="reuse one copy (cache-resident; diagnostic)")
    ap.add_argument("--cold-bytes", type=int, default=COLD_BYTES,
                    help="reads between two reads of the same data in the timed loops, and the size of the "
                         "cache-clearing read before each timed replay (default 1 GiB)")
    ap.add_argument("--layout", choices=("rlc", "rows16", "interleaved"), default="rlc",
                    help="row encoding of the matrix: the paper's 4-bit runs (default), 16-bit row offsets "
                         "(decode-free), or the runs in lane-interleaved order")
    ap.add_argument("--lds-swizzle", action="store_true", help="XOR-swizzled LDS tile (RLC layout)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain copy of a known size (counter calibration)")
    ap.add_argument("--record-traffic", nargs=4, metavar=("FETCH_CSV", "WRITE_CSV", "COPY_FETCH_CSV", "COPY_WRITE_CSV"),
                    help="host only: write this workload's HBM traffic record from rocprofv3 counter CSVs")
    ap.add_argument("--record-kernel-trace", metavar="TRACE_CSV",
                    help="host only: write this workload's kernel-duration record from a rocprofv3 "
                         "--kernel-trace CSV of this benchmark run with the same flags")
    ap.add_argument("--sequence", type=int, choices=(3, 4, 5),
                    help="time one decode step of config 3, 4 or 5 (its own JSON line)")
    ap.add_argument("--layers", type=int, default=0, help="layers of --sequence (0 = the config's)")
    ap.add_argument("--seq-as", type=float, default=None, help="activation sparsity of --sequence")
    ap.add_argument("--workers", type=int, default=0, help="host processes that encode --sequence layers (0 = 16)")
    ap.add_argument("--no-fused", action="store_true", help="--sequence without the stacked-encoding schedule")
    ap.add_argument("--format-study", action="store_true",
                    help="host only: RLC-CSC vs bitmap vs dense sizes across weight sparsity")
    ap.add_argument("--variant-study", action="store_true",
                    help="the kernel variants (swizzled tile, 16-bit rows, interleaved runs) against the default, "
                         "one process, seven shapes")
    ap.add_argument("--paper-shapes", action="store_true",
                    help="the paper's six kernel shapes at 30/50/70%% dual sparsity vs dense GEMV")
    ap.add_argument("--encode-throughput", action="store_true",
                    help="host only: encoder throughput on the benchmark matrices")
    args = ap.parse_args()
    COLD_BYTES = max(256 << 20, args.cold_bytes // 4096 * 4096)
    if args.copy_calibration:
        return copy_calibration()
    if args.format_study:
        return format_study(args)
    if args.encode_throughput:
        return encode_throughput(args)

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: the SpMSpV path here is single-GPU "
              "(row-sharding across GPUs is a design note, not built); use --gpus 1", file=sys.stderr)
        return 2

    if args.sequence:
        return sequence_bench(args)
    if args.paper_shapes:
        return paper_shapes(args)
    if args.variant_study:
        return variant_study(args)

    import torch
    import torch.nn.functional as F

    import paper_2608_01536_amd as celty
    import workloads

    M, K = args.M, args.K
    headline = (M, K, args.ws, args.as_) == (4096, 4096, 70.0, 70.0) and not args.sigma and \
        args.layout == "rlc" and not args.lds_swizzle
    if args.sigma:
        p = workloads.outlier_feature_problem(M, K, int(args.ws), args.as_, args.sigma)
    else:
        p = workloads.make_problem(2, M, K, args.ws, args.as_, "laplace", seed=0, proj=workloads.PROJ_IDS["w"])
    R = args.R or celty.default_tile_rows(M, K)
    layout = {"rlc": celty.LAYOUT_RLC, "rows16": celty.LAYOUT_ROWS16, "interleaved": celty.LAYOUT_INTERLEAVED}[args.layout]
    enc_rlc = celty.celty_encode(p.W, p.mask, R)
    enc = enc_rlc if layout == celty.LAYOUT_RLC else celty.celty_encode(p.W, p.mask, R, layout=layout)
    swz = 1 if args.lds_swizzle else 0
    launch = (args.cols, args.waves, 0, swz) if (args.cols or args.waves or swz) else None
    plan = celty.celty_spmspv_plan(enc, launch)
    variant = ("" if layout == celty.LAYOUT_RLC else f"-{args.layout}") + ("-swizzle" if swz else "")
    workload_key = (f"{M}x{K}-ws{args.ws:g}-as{args.as_:g}" + (f"-sigma{args.sigma:g}" if args.sigma else "") + f"-R{R}-"
                    f"{plan['cols_per_block']}x{plan['waves_per_block']}x{plan['groups_per_lane']}" + variant)
    variant_flags = (f" --layout {args.layout}" if layout != celty.LAYOUT_RLC else "") + \
                    (" --lds-swizzle" if swz else "")
    if args.record_traffic:
        flags = f" --M {M} --K {K} --ws {args.ws:g} --as {args.as_:g}" + (f" --R {args.R}" if args.R else "") + \
                (f" --sigma {args.sigma:g}" if args.sigma else "") + \
                (f" --cols {args.cols}" if args.cols else "") + (f" --waves {args.waves}" if args.waves else "") + \
                variant_flags
        cmds = [f"rocprofv3 --pmc {c} --output-format csv -d <out> -o run -- python3 bench.py "
                f"--steps 200 --warmup 20 --no-cpu --no-dense --no-read-floor{flags}" for c in ("FETCH_SIZE", "WRITE_SIZE")]
        cmds += [f"rocprofv3 --pmc {c} --output-format csv -d <out> -o run -- python3 bench.py --copy-calibration"
                 for c in ("FETCH_SIZE", "WRITE_SIZE")]
        return record_traffic(workload_key, args.record_traffic, cmds)
    if args.record_kernel_trace:
        flags = f" --M {M} --K {K} --ws {args.ws:g} --as {args.as_:g}" + (f" --R {args.R}" if args.R else "") + \
                (f" --sigma {args.sigma:g}" if args.sigma else "") + \
                (f" --cols {args.cols}" if args.cols else "") + (f" --waves {args.waves}" if args.waves else "") + \
                variant_flags
        cmd = (f"rocprofv3 --kernel-trace --stats --output-format csv -d <out> -o run -- python3 bench.py "
               f"--no-cpu --no-dense --no-read-floor --steps {args.steps} --warmup {args.warmup}{flags}")
        return record_kernel_trace(workload_key, args.record_kernel_trace, cmd)
    dev = torch.device("cuda:0")
    # algorithmic bytes are those of the paper's format (RLC) for every
    # variant; bytes requested are the variant's own
    b_alg, e_a, g_a = algorithmic_bytes_from_encoding(enc_rlc, p.x, p.tau)
    if layout == celty.LAYOUT_ROWS16:
        g_v = algorithmic_bytes_from_encoding(enc, p.x, p.tau)[2]
        comp_fetched, total_fetched = fetched_bytes_from_encoding(enc, g_v, plan, group_bytes=32)
    else:
        comp_fetched, total_fetched = fetched_bytes_from_encoding(enc, g_a, plan)
    print(f"[bench] {M}x{K} ws{args.ws:g} as{args.as_:g} R={R} plan={plan}", file=sys.stderr, flush=True)
    flush = None if args.hot else CacheFlush(torch)
    run = cold_spmspv(torch, celty, enc, p, launch, args.steps, args.warmup, args.hot, flush=flush)
    us_step, samples, eager_us, ncopies = run["us"], run["samples"], run["eager_us"], run["copies"]
    us_kernel = us_step
    print(f"[bench] timed: {us_step:.3f} us/step (queued launches), {run['graph_us']:.3f} (graph replay), "
          f"eager {eager_us:.2f} us/call", file=sys.stderr, flush=True)

    # floor: a near-empty kernel (one-element fill) under the same timing
    tiny = torch.zeros(1, device=dev)
    floor_wall = time_loop(torch, lambda i: tiny.fill_(1.0), args.steps)
    floor_kernel, _, _ = time_queued(torch, lambda i: tiny.fill_(1.0), args.steps, flush=flush)

    dense = None if args.no_dense else cold_dense(torch, F, p, args.steps, args.hot, flush=flush)
    floor_read = None if (args.hot or args.no_read_floor) else read_floor(torch, celty, b_alg, args.steps, flush)

    cpu = None
    if not args.no_cpu:
        print("[bench] cpu baseline", file=sys.stderr, flush=True)
        cpu = cpu_baseline(p, args.cpu_seconds)

    gbps_step = b_alg / us_step / 1e3
    achieved = b_alg / us_kernel / 1e3
    traffic = None if args.hot else measured_traffic(workload_key)
    ktrace = None if args.hot else recorded_kernel_trace(workload_key)
    workload = (f"{M}x{K} fp16 W (out x in), {args.ws:g}% unstructured weight sparsity + "
                f"{args.as_:g}% activation sparsity (Laplace x, magnitude threshold), batch 1")
    if args.sigma:
        workload += (f"; outlier input features (per-feature scale exp({args.sigma:g}*N(0,1)) on W's columns "
                     f"and x, per-row magnitude pruning)")
    out = {
        "metric": METRIC if headline else f"us/SpMSpV + effective HBM GB/s, {M}x{K} at ws{args.ws:g}/as{args.as_:g}",
        "value": round(us_step, 3),
        "unit": "µs/SpMSpV",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(us_step / 1e3, 6),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16 inputs, f32 products, i32/i64 fixed-point sums",
        "arithmetic": "fp16 W and x; every product exact in fp32; sums in int32 fixed point per workgroup on a "
                      "grid from n * max colmax*|x| over its n active columns; column slices merged with 64-bit "
                      "integer atomics on a fixed 2^-33 grid (partials clamped to +-4096, the excess added on "
                      "2^-8); y fp16 (RNE)",
        "data": "synthetic",
        "config": {"workload": workload, "workload_key": workload_key, "M": M, "K": K, "weight_sparsity_pct": args.ws,
                   "activation_sparsity_pct": args.as_, "tile_rows_R": R,
                   "storage": {"rlc": "fp16 values + 4-bit runs", "rows16": "fp16 values + 16-bit row offsets",
                               "interleaved": "fp16 values + 4-bit runs, lane-interleaved"}[args.layout] +
                              (", XOR-swizzled LDS tile" if swz else ""),
                   "cold_copies": ncopies, "launch": plan},
        "effective_GBps": round(gbps_step, 1),
        "pct_peak_hbm": round(100 * gbps_step / PEAK_HBM_GBPS, 2),
        "algorithmic_bytes": b_alg,
        "active_entries": e_a,
        "compressed_bytes_fetched": comp_fetched,
        "pct_peak_hbm_fetched": round(100 * comp_fetched / us_step / 1e3 / PEAK_HBM_GBPS, 2),
        "bytes_requested": total_fetched,
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                     "frac": round(achieved / PEAK_HBM_GBPS, 4), "traffic": traffic,
                     "kernel_us": round(us_kernel, 3), "kernel_us_replays": [round(v, 3) for v in samples],
                     "bytes_per_launch": b_alg,
                     "timing": "HIP events on the launch stream around the K steps, launched back to back, "
                               "all enqueued before the GPU reaches the start event",
                     "queued": run["queued"],
                     "graph_replay_us": round(run["graph_us"], 3),
                     "graph_replay_us_replays": [round(v, 3) for v in run["graph_samples"]],
                     "kernel_trace": None if ktrace is None else {
                         "mean_us": round(ktrace["mean_ns"] / 1e3, 3), "median_us": round(ktrace["median_ns"] / 1e3, 3),
                         "frac_mean": round(b_alg / ktrace["mean_ns"] / PEAK_HBM_GBPS, 4),
                         "frac_median": round(b_alg / ktrace["median_ns"] / PEAK_HBM_GBPS, 4),
                         "dispatches": ktrace["dispatches"],
                         "source": os.path.relpath(kernel_trace_file(workload_key), ROOT)}},
        "eager_us_per_call": round(eager_us, 3),
        "eager_us_per_call_prepared": round(run["eager_prepared_us"], 3),
        "launch_floor": {"queued_us": round(floor_kernel, 3), "eager_us": round(floor_wall, 3),
                         "op": "one-element torch fill kernel"},
        "read_floor": None if floor_read is None else dict(
            floor_read, kernel_vs_floor=round(floor_read["us"] / us_step, 3),
            note="a plain read of the algorithmic bytes in one launch; kernel_vs_floor > 1: the SpMSpV call "
                 "takes less time than that read"),
        "dense_gemv": dense,
        "speedup_vs_dense": round(dense["us"] / us_step, 3) if dense else None,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out))
    return 0


if __name__ == "__main__":
    sys.exit(main())
