"""Throughput of calling-context-tree construction on one MI355X.

One step = one cct_build (ingest, exact dedup, exclusive aggregation, publish,
canonical sort, node emission with exclusive and inclusive sums) of the whole batch,
inputs already resident in HBM, followed by cct_free.  Prints one JSON line.

With --workload merge, one step = the 32 cct_merge calls that fold 32 chunks of
2,097,152 events into a tree built (untimed) from an 8,388,608-event base; the rate
is chunk events per second of merge time.

With --workload activity, one step = 8 cct_merge_activity calls into a tree built
(untimed) from the same base: each joins one flush of activity records (every launch
of a 2,097,152-path registry once, in shuffled order, 10% repeated records, 2% records
with unregistered IDs) with the registry by correlation ID and merges the result; the
rate is records per second.

With --workload bottom_up, one step = one cct_bottom_up computation (the view is
recomputed: every step starts from a tree built untimed from the 16M-event trace); the
rate is tree nodes per second.

    python bench.py [--gpus 1] [--steps 20] [--warmup 3] [--workload layered_16m]
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

METRIC = "call-path events aggregated/sec into CCT + achieved HBM GB/s (fraction of peak)"
HBM_PEAK_GBPS = 8000.0
DESCRIPTIONS = {
    "layered_16m": "16,777,216 events, 200,000 frame ids, depth 16-128, 90% under 8 training-loop roots, "
                   "2 uint64 metrics, Zipf 1.1",
    "layered_1m": "1,048,576 events, 50,000 frame ids, depth 8-64, 3 uint64 metrics, Zipf 1.2",
    "deep_recursion": "4,194,304 events, 20,000 frame ids, depth 256-512 recursion of a 12-frame cycle, "
                      "1 uint64 metric",
    "tiny": "10,000 events on a random call-site tree, 1 uint64 metric",
    "merge": "8,388,608-event base (layered_16m program, 60% of its paths) + 32 merged chunks of 2,097,152 events "
             "(20% from paths new to the chunk), 4 uint64 metrics (one full-range)",
    "bottom_up": "bottom-up view of the layered_16m tree (4,407,055 nodes, 2 uint64 metrics): per frame, exclusive "
                 "sums and inclusive sums counted once per path",
    "filter": "ratio filter over the layered_16m tree (4,407,055 nodes, 2 uint64 metrics): nodes whose incl "
              "metric 0 per unit of incl metric 1 is below the root's ratio (the shape of the kernel-fusion and "
              "CPU-latency analyses), exact 128-bit products, ids listed in preorder",
    "stats": "layered_16m built with per-node statistics (16,777,216 events, 2 uint64 metrics): sample counts, "
             "minima and sums of squares kept per path, then every node's exclusive and inclusive count, min, sum of "
             "squares, mean and population deviation",
    "query": "1,048,576 query paths (the first events' paths of the layered_16m trace, so every one is a node, "
             "plus 1,024 absent ones) looked up in the layered_16m tree (4,407,055 nodes, 2 uint64 metrics): node "
             "ids and both sums; the tree's prefix index is built by the first (warm-up) call",
    "activity": "8,388,608-event base (as merge) + 8 activity flushes, each a registry of 2,097,152 call paths "
                "(a merge chunk) under distinct correlation IDs and 2,348,810 records (every ID once, shuffled, "
                "+10% repeated IDs, +2% unregistered IDs), 4 uint64 metrics",
}
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "ingest_traffic.json")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_digest():
    h = hashlib.sha256()
    for name in ("ingest.hip", "common.h"):
        with open(os.path.join(ROOT, "paper_2411_02797_amd", "csrc", name), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(workload):
    """HBM bytes per ingest launch from the committed rocprofv3 counter summary, or
    None when there is none for this workload or the kernel changed since."""
    try:
        with open(TRAFFIC_FILE) as fh:
            rec = json.load(fh)
    except (OSError, ValueError):
        return None
    r = rec.get(workload)
    if not r or r.get("kernel_digest") != kernel_source_digest():
        return None
    return r.get("bytes_per_launch")


def host_cpu():
    """Host CPU model and the logical CPUs this process may run on."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return model, len(os.sched_getaffinity(0)), os.cpu_count()


def achievable_read(torch, buf):
    """Same-run achievable read bandwidth: the best of five plain coalesced 16-byte buffer-load
    reads of `buf` (libcct_readbw.so), as context for the 8 TB/s denominator."""
    import ctypes
    path = os.path.join(ROOT, "paper_2411_02797_amd", "libcct_readbw.so")
    if not os.path.exists(path):
        return None
    lib = ctypes.CDLL(path)
    lib.cctbw_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int,
                               ctypes.POINTER(ctypes.c_float)]
    lib.cctbw_read.restype = ctypes.c_int
    sink = torch.zeros(4096, dtype=torch.int32, device=buf.device)
    nbytes = buf.numel() * buf.element_size()
    best = ctypes.c_float(0)
    rc = lib.cctbw_read(ctypes.c_void_p(buf.data_ptr()), nbytes, ctypes.c_void_p(sink.data_ptr()),
                        ctypes.c_void_p(torch.cuda.current_stream().cuda_stream), 5, ctypes.byref(best))
    if rc != 0 or best.value <= 0:
        return None
    gbps = nbytes / (best.value * 1e-3) / 1e9
    return {"gbps": gbps, "frac_of_peak": gbps / HBM_PEAK_GBPS, "bytes": nbytes, "best_ms": best.value,
            "kernel": "plain coalesced read of the frames buffer, best of 5, same run"}


def cpu_baseline(offsets, frames, metrics, sample_events):
    import oracle
    n = min(sample_events, offsets.size - 1)
    o = offsets[: n + 1]
    f = frames[: int(o[-1])]
    w = metrics[:n]
    t0 = time.perf_counter()
    orc = oracle.Oracle(w.shape[1])
    orc.ingest(o, f, w)
    orc.tree()
    dt = time.perf_counter() - t0
    orc.close()
    model, nproc, ncpu = host_cpu()
    return {"value": n / dt, "unit": "events/s", "cores": 1, "kind": "oracle",
            "sample": f"first {n:,} events ({int(o[-1]):,} frames) of the same trace, std::map trie "
                      f"(single thread, g++ -O2), {dt:.1f} s",
            "nproc": nproc, "host_cpus": ncpu, "cpu_model": model}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="layered_16m", choices=sorted(DESCRIPTIONS))
    ap.add_argument("--cpu-sample", type=int, default=1 << 24, help="events timed on the oracle")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibrate", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB five times (the reference kernel that "
                         "scales the HBM byte counters) and exit")
    ap.add_argument("--read-calibrate", type=int, default=0, metavar="MIB",
                    help="only run the plain 16-byte buffer-load read of MIB MiB five times (a second "
                         "reference kernel for the fetched-byte counter) and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "bench.py measures one GPU; sharding across GPUs is a design only, nothing here runs on several",
                          "n_gpus": args.gpus}))
        sys.exit(2)

    import torch
    # the library's calls go to the stream they are given; the bench gives them a stream of
    # its own, as a caller would, rather than the legacy default stream (on which a call
    # on the 1M-event workload measured about 0.04 ms slower)
    torch.cuda.set_stream(torch.cuda.Stream(device=0))
    if args.copy_calibrate:
        n = args.copy_calibrate << 20
        src = torch.ones(n // 4, dtype=torch.int32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "launches": 5}))
        return
    if args.read_calibrate:
        buf = torch.ones((args.read_calibrate << 20) // 4, dtype=torch.int32, device="cuda")
        torch.cuda.synchronize()
        r = achievable_read(torch, buf)
        if r is None:
            sys.exit("read calibration failed: libcct_readbw.so missing or the read kernel failed")
        print(json.dumps({"read_bytes": r["bytes"], "launches": 5, "best_ms": r["best_ms"], "gbps": r["gbps"]}))
        return
    import tracegen
    import paper_2411_02797_amd as cct

    cct.load_library()
    dev = torch.device("cuda", 0)
    t0 = time.perf_counter()
    if args.workload == "merge":
        return bench_merge(args, torch, tracegen, cct, dev)
    if args.workload == "activity":
        return bench_activity(args, torch, tracegen, cct, dev)
    if args.workload == "bottom_up":
        return bench_bottom_up(args, torch, tracegen, cct, dev)
    if args.workload == "filter":
        return bench_filter(args, torch, tracegen, cct, dev)
    if args.workload == "stats":
        return bench_stats(args, torch, tracegen, cct, dev)
    if args.workload == "query":
        return bench_query(args, torch, tracegen, cct, dev)
    o, f, w = tracegen.generate(args.workload)
    N, F, M = o.size - 1, f.size, w.shape[1]
    log(f"generated {args.workload}: N={N:,} F={F:,} M={M} in {time.perf_counter() - t0:.1f}s")
    to = torch.from_numpy(o).to(dev)
    tf = torch.from_numpy(f.view(np.int32)).to(dev)
    tw = torch.from_numpy(w.view(np.int64)).to(dev)
    torch.cuda.synchronize()

    for i in range(args.warmup):
        tree = cct.build(to, tf, tw)
        U, _, D = tree._info()
        tree.free()
        log(f"warmup {i}: U={U:,} D={D:,} phases(ms)={['%.3f' % x for x in cct.last_timings()]}")
    torch.cuda.synchronize()
    phases, step_wall = [], []
    t_start = time.perf_counter()
    for _ in range(args.steps):
        t_step = time.perf_counter()
        tree = cct.build(to, tf, tw)  # returns once the stream has finished the build
        phases.append(cct.last_timings())
        tree.free()
        step_wall.append((time.perf_counter() - t_step) * 1000.0)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    ms = wall * 1000.0 / args.steps
    ph = np.array(phases)
    ingest_ms = float(ph[:, 0].mean())
    log(f"timed {args.steps} steps: {ms:.3f} ms/step; mean phases(ms) ingest/publish/sort/emit/total = "
        f"{['%.3f' % x for x in ph.mean(axis=0)]}")

    # algorithmic bytes.  The dominant kernel (ingest: validate, hash, exact dedup) must
    # read the offsets and every frame once; the whole call must in addition read the
    # metrics once and write every output array once.
    b_ingest = 8 * (N + 1) + 4 * F
    b_alg = b_ingest + 8 * M * N + U * (12 + 16 * M)
    achieved = b_ingest / (ingest_ms * 1e-3) / 1e9
    traffic = measured_traffic(args.workload)
    line = {
        "metric": METRIC,
        "value": N / (ms * 1e-3),
        "unit": "events/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u64",
        "data": "synthetic",
        "config": {"workload": f"{args.workload}: {DESCRIPTIONS[args.workload]}", "events": N, "frames": F,
                   "metrics": M, "distinct_paths": D, "nodes": U},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS, "traffic": traffic,
                     "kernel": "ingest_kernel (validate offsets, hash paths, exact dedup into the table)",
                     "bytes_per_launch": b_ingest, "avg_launch_ms": ingest_ms},
        "effective_hbm_gbps": b_alg / (ms * 1e-3) / 1e9,
        "effective_frac_of_peak": b_alg / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS,
        "phase_ms": {"ingest": ingest_ms, "publish": float(ph[:, 1].mean()), "sort": float(ph[:, 2].mean()),
                     "emit": float(ph[:, 3].mean()), "call": float(ph[:, 4].mean())},
        "step_ms": {"mean": ms, "median": float(np.median(step_wall)), "min": float(np.min(step_wall))},
        "call_ms": {"mean": float(ph[:, 4].mean()), "median": float(np.median(ph[:, 4])),
                    "min": float(np.min(ph[:, 4]))},
        "achievable_read": achievable_read(torch, tf),
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(o, f, w, args.cpu_sample)
    print(json.dumps(line), flush=True)


def bench_merge(args, torch, tracegen, cct, dev):
    def to_dev(o, f, w):
        return (torch.from_numpy(o).to(dev), torch.from_numpy(f.view(np.int32)).to(dev),
                torch.from_numpy(w.view(np.int64)).to(dev))
    t0 = time.perf_counter()
    base = to_dev(*tracegen.generate("merge_base"))
    chunks = []
    n_chunk_events = n_chunk_frames = 0
    for c in range(32):
        o, f, w = tracegen.generate("merge_chunk", chunk=c)
        n_chunk_events += o.size - 1
        n_chunk_frames += f.size
        chunks.append(to_dev(o, f, w))
    M = chunks[0][2].shape[1]
    torch.cuda.synchronize()
    log(f"generated merge: base N={base[0].numel() - 1:,}, 32 chunks N={n_chunk_events:,} "
        f"F={n_chunk_frames:,} in {time.perf_counter() - t0:.1f}s")
    merge_ms, phases, base_ms = [], [], []
    U = D = 0
    sizes = []  # (U before, U after) of every merge of the last step
    for step in range(args.warmup + args.steps):
        tree = cct.build(*base)
        base_ms.append(cct.last_timings()[4])
        torch.cuda.synchronize()
        t_seq = time.perf_counter()
        ph, sz = [], []
        u_prev = tree.n_nodes
        for ch in chunks:
            tree.merge(*ch)
            ph.append(cct.last_timings())
            u_now = tree.n_nodes  # host-side (cct_info reads no device memory)
            sz.append((u_prev, u_now))
            u_prev = u_now
        torch.cuda.synchronize()
        wall = (time.perf_counter() - t_seq) * 1000.0
        U, _, D = tree._info()
        tree.free()
        sizes = sz
        if step >= args.warmup:
            merge_ms.append(wall)
            phases.extend(ph)
        log(f"{'warmup' if step < args.warmup else 'step'} {step}: 32 merges {wall:.2f} ms, U={U:,} D={D:,}")
    ms = float(np.mean(merge_ms))
    ph = np.array(phases)
    ingest_ms = float(ph[:, 0].mean())
    b_ingest = 8 * (n_chunk_events // 32 + 1) + 4 * (n_chunk_frames // 32)
    achieved = b_ingest / (ingest_ms * 1e-3) / 1e9
    # whole-merge algorithmic bytes of the 32 merges of a step: each reads its chunk's
    # offsets, frames and metrics and the old nodes' exclusive sums, and writes every
    # node's parent, frame, depth, exclusive and inclusive sums
    b_merge = (8 * (n_chunk_events + 32) + 4 * n_chunk_frames + 8 * M * n_chunk_events
               + sum(u1 * (12 + 16 * M) + u0 * 8 * M for u0, u1 in sizes))
    eff = b_merge / (ms * 1e-3) / 1e9
    line = {
        "metric": METRIC, "value": n_chunk_events / (ms * 1e-3), "unit": "events/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "u64", "data": "synthetic",
        "config": {"workload": f"merge: {DESCRIPTIONS['merge']}", "chunk_events": n_chunk_events,
                   "chunk_frames": n_chunk_frames, "metrics": M, "distinct_paths": D, "nodes": U,
                   "base_build_ms": float(np.mean(base_ms))},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS, "traffic": None,
                     "kernel": "ingest_kernel of one merge (validate, hash, exact dedup against the tree)",
                     "bytes_per_launch": b_ingest, "avg_launch_ms": ingest_ms},
        "phase_ms_per_merge": {"ingest": ingest_ms, "publish": float(ph[:, 1].mean()),
                               "sort": float(ph[:, 2].mean()), "emit": float(ph[:, 3].mean()),
                               "call": float(ph[:, 4].mean())},
        "effective_hbm_gbps": eff,
        "effective_frac_of_peak": eff / HBM_PEAK_GBPS,
        "step_ms": {"mean": ms, "median": float(np.median(merge_ms)), "min": float(np.min(merge_ms))},
        "merge_call_ms": {"median": float(np.median(ph[:, 4])), "min": float(np.min(ph[:, 4]))},
        "achievable_read": achievable_read(torch, chunks[0][1]),
    }
    print(json.dumps(line), flush=True)



def activity_flush(tracegen, c):
    """Flush c: the registry is merge chunk c (its call paths, registered at launch under
    distinct IDs), the records name every registered ID once in shuffled order, plus 10%
    repeated IDs and 2% IDs never registered."""
    o, f, w = tracegen.generate("merge_chunk", chunk=c)
    n, m = o.size - 1, w.shape[1]
    rng = np.random.default_rng(1000 + c)
    ids = (np.uint64(c + 1) << np.uint64(40)) + rng.permutation(n).astype(np.uint64)
    order = rng.permutation(n)
    rep = rng.integers(0, n, size=n // 10)
    rec = np.concatenate([ids[order], ids[rep], (np.uint64(1) << np.uint64(63)) + np.arange(n // 50, dtype=np.uint64)])
    met = np.concatenate([w[order], w[rep], w[: n // 50]])
    perm = rng.permutation(rec.size)
    return o, f, ids, rec[perm], np.ascontiguousarray(met[perm])


def bench_activity(args, torch, tracegen, cct, dev):
    def t64(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int64)).to(dev)
    t0 = time.perf_counter()
    bo, bf, bw = tracegen.generate("merge_base")
    base = (torch.from_numpy(bo).to(dev), torch.from_numpy(bf.view(np.int32)).to(dev), t64(bw))
    flushes = []
    n_rec = n_reg = n_reg_frames = 0
    for c in range(8):
        o, f, ids, rec, met = activity_flush(tracegen, c)
        n_rec += rec.size
        n_reg += o.size - 1
        n_reg_frames += f.size
        flushes.append((torch.from_numpy(o).to(dev), torch.from_numpy(f.view(np.int32)).to(dev), t64(ids), t64(rec),
                        t64(met)))
    M = flushes[0][4].shape[1]
    torch.cuda.synchronize()
    log(f"generated activity: 8 flushes, {n_reg:,} registered paths ({n_reg_frames:,} frames), {n_rec:,} records "
        f"in {time.perf_counter() - t0:.1f}s")
    step_ms, phases = [], []
    unmatched = U = D = 0
    for step in range(args.warmup + args.steps):
        tree = cct.build(*base)
        torch.cuda.synchronize()
        t_seq = time.perf_counter()
        ph, un = [], 0
        for fl in flushes:
            un += tree.merge_activity(*fl)
            ph.append(cct.last_timings())
        torch.cuda.synchronize()
        wall = (time.perf_counter() - t_seq) * 1000.0
        U, _, D = tree._info()
        tree.free()
        unmatched = un
        if step >= args.warmup:
            step_ms.append(wall)
            phases.extend(ph)
        log(f"{'warmup' if step < args.warmup else 'step'} {step}: 8 flushes {wall:.2f} ms, unmatched {un:,}, "
            f"U={U:,} D={D:,}")
    ms = float(np.mean(step_ms))
    ph = np.array(phases)
    join_ms = float(ph[:, 5].mean())
    # algorithmic bytes of the join per flush: registry offsets and IDs read, records'
    # IDs and metrics read, the per-path sums written.  Every registered path is named by
    # a record here, so the registry is the merged batch and no frame is copied.
    per = n_reg // 8, n_rec // 8
    b_join = 8 * (per[0] + 1) + 8 * per[0] + 8 * per[1] * (1 + M) + 8 * per[0] * M
    achieved = b_join / (join_ms * 1e-3) / 1e9
    line = {
        "metric": METRIC, "value": n_rec / (ms * 1e-3), "unit": "records/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "u64", "data": "synthetic",
        "config": {"workload": f"activity: {DESCRIPTIONS['activity']}", "records": n_rec, "registered_paths": n_reg,
                   "registered_frames": n_reg_frames, "unmatched_records": unmatched, "metrics": M,
                   "distinct_paths": D, "nodes": U},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS, "traffic": None,
                     "kernel": "correlation-ID join of one flush (table, join, per-path sums, compaction)",
                     "bytes_per_launch": b_join, "avg_launch_ms": join_ms},
        "phase_ms_per_flush": {"join": join_ms, "ingest": float(ph[:, 0].mean()), "publish": float(ph[:, 1].mean()),
                               "sort": float(ph[:, 2].mean()), "emit": float(ph[:, 3].mean()),
                               "merge_call": float(ph[:, 4].mean())},
    }
    print(json.dumps(line), flush=True)


def bench_bottom_up(args, torch, tracegen, cct, dev):
    o, f, w = tracegen.generate("layered_16m")
    to = torch.from_numpy(o).to(dev)
    tf = torch.from_numpy(f.view(np.int32)).to(dev)
    tw = torch.from_numpy(w.view(np.int64)).to(dev)
    M = w.shape[1]
    view_ms, wall_ms = [], []
    U = K = 0
    for step in range(args.warmup + args.steps):
        tree = cct.build(to, tf, tw)
        U = tree.n_nodes
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        v = tree.bottom_up()
        torch.cuda.synchronize()
        wall = (time.perf_counter() - t0) * 1000.0
        K = v["frames"].numel()
        ms = cct.last_timings()[6]
        tree.free()
        del v
        if step >= args.warmup:
            view_ms.append(ms)
            wall_ms.append(wall)
        log(f"{'warmup' if step < args.warmup else 'step'} {step}: view {ms:.3f} ms (call {wall:.3f} ms), "
            f"U={U:,} K={K:,}")
    ms = float(np.mean(view_ms))
    # algorithmic bytes: every node's frame, subtree end and sums read once, the view written once
    b_alg = U * (4 + 4 + 16 * M) + K * (4 + 16 * M)
    achieved = b_alg / (ms * 1e-3) / 1e9
    line = {
        "metric": METRIC, "value": U / (ms * 1e-3), "unit": "nodes/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "u64", "data": "synthetic",
        "config": {"workload": f"bottom_up: {DESCRIPTIONS['bottom_up']}", "nodes": U, "frames_in_view": K,
                   "metrics": M, "call_ms_with_copy_out": float(np.mean(wall_ms))},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS, "traffic": None,
                     "kernel": "bottom-up view (radix sort by frame, max-scan, prefix sums)",
                     "bytes_per_launch": b_alg, "avg_launch_ms": ms},
    }
    print(json.dumps(line), flush=True)

def bench_filter(args, torch, tracegen, cct, dev):
    o, f, w = tracegen.generate("layered_16m")
    tree = cct.build(torch.from_numpy(o).to(dev), torch.from_numpy(f.view(np.int32)).to(dev),
                     torch.from_numpy(w.view(np.int64)).to(dev))
    U, M = tree.n_nodes, w.shape[1]
    root = tree.to_tensors(device="cpu")["incl"][0].numpy().view(np.uint64)
    p, q = int(root[0]), max(int(root[1]), 1)  # the root's ratio of metric 0 to metric 1
    del o, f, w
    filt_ms, hot_ms, wall_ms = [], [], []
    K = H = 0
    for step in range(args.warmup + args.steps):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ids = tree.filter(0, -1, p, q, den="metric", den_metric=1)
        wall = (time.perf_counter() - t0) * 1000.0
        K, ms = ids.numel(), cct.last_timings()[7]
        H = tree.hotspots(0, 1, 1000).numel()  # leaves above 0.1% of the root's metric 0
        hot = cct.last_timings()[7]
        del ids
        if step >= args.warmup:
            filt_ms.append(ms)
            hot_ms.append(hot)
            wall_ms.append(wall)
        log(f"{'warmup' if step < args.warmup else 'step'} {step}: filter {ms * 1000:.1f} us (call {wall * 1000:.1f} us), "
            f"K={K:,}; hotspots {hot * 1000:.1f} us, {H:,} leaves")
    tree.free()
    ms = float(np.mean(filt_ms))
    # algorithmic bytes: both sums of every node read once, each match's id written once
    b_alg = U * 16 + K * 8
    achieved = b_alg / (ms * 1e-3) / 1e9
    line = {
        "metric": METRIC, "value": U / (ms * 1e-3), "unit": "nodes/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "u64", "data": "synthetic",
        "config": {"workload": f"filter: {DESCRIPTIONS['filter']}", "nodes": U, "metrics": M, "matches": K,
                   "threshold": [p, q], "call_ms_with_count_readback": float(np.mean(wall_ms)),
                   "hotspot_ms": float(np.mean(hot_ms)), "hotspot_leaves": H},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS, "traffic": None,
                     "kernel": "ratio filter (predicate mask, scan of tile counts, id write)",
                     "bytes_per_launch": b_alg, "avg_launch_ms": ms},
    }
    print(json.dumps(line), flush=True)


def bench_stats(args, torch, tracegen, cct, dev):
    o, f, w = tracegen.generate("layered_16m")
    N, F, M = o.size - 1, f.size, w.shape[1]
    to = torch.from_numpy(o).to(dev)
    tf = torch.from_numpy(f.view(np.int32)).to(dev)
    tw = torch.from_numpy(w.view(np.int64)).to(dev)
    del o, f, w
    build_ms, kept_ms, node_ms, plain_ms = [], [], [], []
    U = 0
    for step in range(args.warmup + args.steps):
        tree = cct.build(to, tf, tw)  # the same build without statistics, for the overhead
        plain = cct.last_timings()[4]
        tree.free()
        tree = cct.build(to, tf, tw, stats=True)
        t = cct.last_timings()
        U = tree.n_nodes
        st = tree.stats()
        node = cct.last_timings()[9]
        del st
        tree.free()
        if step >= args.warmup:
            build_ms.append(t[4])
            kept_ms.append(t[8])
            node_ms.append(node)
            plain_ms.append(plain)
        log(f"{'warmup' if step < args.warmup else 'step'} {step}: build with statistics {t[4]:.3f} ms "
            f"(statistics {t[8]:.3f} ms; plain build {plain:.3f} ms), node statistics {node:.3f} ms, U={U:,}")
    ms = float(np.mean(build_ms))
    kept = float(np.mean(kept_ms))
    # algorithmic bytes of the kept statistics: every event's slot id and metric row read once
    b_alg = N * (4 + 8 * M)
    achieved = b_alg / (kept * 1e-3) / 1e9
    line = {
        "metric": METRIC, "value": N / (ms * 1e-3), "unit": "events/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "u64", "data": "synthetic",
        "config": {"workload": f"stats: {DESCRIPTIONS['stats']}", "events": N, "frames": F, "metrics": M,
                   "nodes": U, "statistics_ms": kept, "plain_build_ms": float(np.mean(plain_ms)),
                   "node_statistics_ms": float(np.mean(node_ms))},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS, "traffic": None,
                     "kernel": "statistics kept by the build (per-slot samples, fold into the paths)",
                     "bytes_per_launch": b_alg, "avg_launch_ms": kept},
    }
    print(json.dumps(line), flush=True)


def bench_query(args, torch, tracegen, cct, dev):
    o, f, w = tracegen.generate("layered_16m")
    tree = cct.build(torch.from_numpy(o).to(dev), torch.from_numpy(f.view(np.int32)).to(dev),
                     torch.from_numpy(w.view(np.int64)).to(dev))
    U, M = tree.n_nodes, w.shape[1]
    Q = 1 << 20
    absent = 1024
    qo = np.concatenate([o[:Q + 1], o[Q] + 3 * np.arange(1, absent + 1, dtype=np.int64)])
    qf = np.concatenate([f[:o[Q]], np.full(3 * absent, 0xFFFFFFF0, np.uint32)])
    del o, f, w
    tqo, tqf = torch.from_numpy(qo).to(dev), torch.from_numpy(qf.view(np.int32)).to(dev)
    nq, nf = qo.size - 1, int(qo[-1])
    q_ms, wall_ms = [], []
    index_ms = 0.0
    for step in range(args.warmup + args.steps):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ids, ex, inc = tree.query(tqo, tqf)
        wall = (time.perf_counter() - t0) * 1000.0
        ms = cct.last_timings()[10]
        if step == 0:
            index_ms = cct.last_timings()[11]  # the first query builds the tree's prefix index
        found = int((ids >= 0).sum().item())
        del ids, ex, inc
        if step >= args.warmup:
            q_ms.append(ms)
            wall_ms.append(wall)
        log(f"{'warmup' if step < args.warmup else 'step'} {step}: lookup {ms:.3f} ms (call {wall:.3f} ms), "
            f"{found:,} of {nq:,} found")
    tree.free()
    ms = float(np.mean(q_ms))
    # algorithmic bytes: every query's offsets and frames read once, its id and sums written once
    b_alg = 8 * (nq + 1) + 4 * nf + nq * (8 + 16 * M)
    achieved = b_alg / (ms * 1e-3) / 1e9
    line = {
        "metric": METRIC, "value": nq / (ms * 1e-3), "unit": "queries/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "u32", "data": "synthetic",
        "config": {"workload": f"query: {DESCRIPTIONS['query']}", "queries": nq, "query_frames": nf, "nodes": U,
                   "metrics": M, "call_ms_with_readback": float(np.mean(wall_ms)),
                   "index_build_ms_first_query": index_ms},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS, "traffic": None,
                     "kernel": "query_kernel (prefix-index probe, exact verification against the stored path)",
                     "bytes_per_launch": b_alg, "avg_launch_ms": ms},
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
