"""Throughput of batched tree-ensemble scoring on one MI355X.

Default workload: the GBDT binary classifier of 500 perfect trees of depth 8
over 28 features (sigmoid of the summed leaves), scoring a resident batch of
1,000,000 rows into scores and per-tree leaf ids, with the strategy the
selector picks. One step is one hb_predict over the whole batch.

Prints one JSON line with rows/s, the roofline of the dominant kernel (its
average launch time measured with HIP events on the launch stream), the other
two strategies timed on the same workload, and the CPU oracle's rate on a
bounded sample of the same workload.
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

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "rows/sec scored, 500-tree depth-8 ensemble, 1M rows; % HBM / MFMA peak"
HBM_PEAK = 8.0e12   # B/s, MI355X HBM3E
INT8_PEAK = 5.0e15  # dense int8 MFMA ops/s, MI355X


def kernel_label(h, strat, n, ws_bytes=0):
    """The kernels a call of n rows launches, as the library's own launch
    plan reports them (hb_plan): "name grid=(x,y) block=b" per launch."""
    return "; ".join(f"{p['kernel']} grid={p['grid']} block={p['block']}" for p in h.plan(n, strat, ws_bytes))


PROFILES = os.path.join(ROOT, "profiles")
CSRC = os.path.join(ROOT, "paper_2010_04804_amd", "csrc")


def kernel_source_sha() -> str:
    """Hash of the library sources: counter summaries recorded against another
    hash describe a different kernel and are not reported."""
    h = hashlib.sha256()
    for p in sorted(glob.glob(os.path.join(CSRC, "*"))):
        with open(p, "rb") as fh:
            h.update(os.path.basename(p).encode())
            h.update(fh.read())
    return h.hexdigest()[:16]


def recorded_traffic(config: int, strategy: str, rows: int, leaves: bool):
    """HBM bytes per launch from a committed rocprofv3 counter summary, or None."""
    sha = kernel_source_sha()
    pat = re.compile(r"traffic_record: config=(\d+) strategy=(\w+) rows=(\d+) leaves=(\d) "
                     r"source_sha=(\w+) fetch_bytes=(\d+) write_bytes=(\d+)")
    for p in glob.glob(os.path.join(PROFILES, "*.md")):
        for m in pat.finditer(open(p).read()):
            if (int(m[1]), m[2], int(m[3]), int(m[4]), m[5]) == (config, strategy, rows, int(leaves), sha):
                return int(m[6]) + int(m[7])
    return None


def algorithmic_bytes(info, n, leaves, strategy):
    """HBM bytes one launch must move: X read once, scores (and leaf ids)
    written once, the strategy's compiled tables read once."""
    K, T, F = info["n_outputs"], info["n_trees"], info["n_features"]
    b = n * F * 4 + n * K * 4 + info["table_bytes"][strategy]
    if leaves:
        b += n * T * 4
    return b


def gemm_ops(model, n):
    """2 n sum_t |I_t| |L_t|: the path-matrix contraction of Algorithm 1 only
    (the feature selection and the leaf gather count as zero operations)."""
    off = model["tree_node_offset"]
    tot = 0
    for t in range(model["n_trees"]):
        f = model["feature"][off[t]:off[t + 1]]
        i = int((f >= 0).sum())
        tot += i * (f.size - i)
    return 2 * n * tot


def cpu_baseline(model, cfg, seconds_target=15.0):
    """The oracle as it stands, timed on this host on the first rows of the
    same workload (bounded to about seconds_target of CPU time)."""
    import oracle
    from paper_2010_04804_amd import synth

    cores = min(len(os.sched_getaffinity(0)), 16)
    probe = synth.make_rows(cfg, 2000)
    t0 = time.perf_counter()
    oracle.predict(model, probe, leaves=True, n_threads=cores)
    dt = max(time.perf_counter() - t0, 1e-6)
    n = int(min(max(2000 * seconds_target / dt, 2000), 1_000_000))
    X = synth.make_rows(cfg, n)
    t0 = time.perf_counter()
    oracle.predict(model, X, leaves=True, n_threads=cores)
    dt = time.perf_counter() - t0
    # one thread on a 10,000-row slice, for a per-core figure
    t1 = time.perf_counter()
    oracle.predict(model, X[:10_000], leaves=True, n_threads=1)
    dt1 = time.perf_counter() - t1
    cpu_model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    cpu_model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"value": n / dt, "unit": "rows/s", "cores": cores, "kind": "oracle",
            "sample": f"first {n} rows of the same workload (scores and leaf ids), "
                      f"{dt:.1f} s on {cores} threads",
            "single_thread_rows_per_s": min(10_000, n) / dt1, "cpu_model": cpu_model,
            "host_cpus": os.cpu_count()}


def mfma_peak_measured():
    """Sustained dense int8 matrix-core rate of this GPU in ops/s, from the
    probe library built beside libhb.so (None if it is not built)."""
    import ctypes
    path = os.path.join(ROOT, "paper_2010_04804_amd", "libhb_probe.so")
    if not os.path.exists(path):
        return None
    lib = ctypes.CDLL(path)
    lib.hb_probe_mfma_i8.restype = ctypes.c_int
    lib.hb_probe_mfma_i8.argtypes = [ctypes.c_int, ctypes.POINTER(ctypes.c_double)]
    v = ctypes.c_double(0.0)
    rc = lib.hb_probe_mfma_i8(0, ctypes.byref(v))
    return v.value if rc == 0 else None


LDS_READS = ["b32, each lane its own word", "b32, hashed slot of 256 (1 KiB)", "b64, each lane its own word pair",
             "b64, hashed slot of 256 (2 KiB)", "u16, each lane its own half-word", "b128, each lane its own 16 bytes",
             "b128, hashed slot of 64 (1 KiB)", "b64 hashed of 256 and b32 own, alternating"]


def run_lds_probe():
    """Nanoseconds per wave-wide LDS read instruction per CU for the read
    shapes of the traversal walks (16 waves per CU, eight reads in flight per
    wave), from the probe library built beside libhb.so: one JSON line per
    shape."""
    import ctypes
    path = os.path.join(ROOT, "paper_2010_04804_amd", "libhb_probe.so")
    if not os.path.exists(path):
        print(json.dumps({"error": "libhb_probe.so is not built (run the package build)"}))
        sys.exit(1)
    lib = ctypes.CDLL(path)
    lib.hb_probe_lds_read.restype = ctypes.c_int
    lib.hb_probe_lds_read.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.POINTER(ctypes.c_double)]
    for mode, name in enumerate(LDS_READS):
        v = ctypes.c_double(0.0)
        rc = lib.hb_probe_lds_read(0, mode, ctypes.byref(v))
        if rc:
            print(json.dumps({"error": f"hb_probe_lds_read({mode}) returned {rc}"}))
            sys.exit(1)
        print(json.dumps({"lds_read": name, "mode": mode, "ns_per_read_per_cu": v.value}), flush=True)


def end_to_end(hb, h, X, n, info, leaves, strategy, dev, reps=3):
    """The whole request from host memory: X copied in from pinned host
    memory, the scoring call, scores (and leaf ids) copied back to pinned host
    memory, one stream, timed from the first copy's start to the last copy's
    end (HIP events), median of a few repetitions; the three parts are timed
    by events between them. The paper times whole runs of its frameworks the
    same way (processor time), Sec. 6."""
    import torch
    stream = torch.cuda.current_stream(dev)
    Xh = torch.from_numpy(X).pin_memory()
    K, T = info["n_outputs"], info["n_trees"]
    sh = torch.empty((n, K), dtype=torch.float32).pin_memory()
    ih = torch.empty((n, T), dtype=torch.int32).pin_memory() if leaves else None
    Xd = torch.empty_like(Xh, device=dev)
    sd = torch.empty((n, K), dtype=torch.float32, device=dev)
    idd = torch.empty((n, T), dtype=torch.int32, device=dev) if leaves else None
    runs = []
    for _ in range(reps):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        ev[0].record(stream)
        Xd.copy_(Xh, non_blocking=True)
        ev[1].record(stream)
        hb.predict_ptr(h, Xd.data_ptr(), n, sd.data_ptr(), idd.data_ptr() if leaves else None, strategy,
                       stream.cuda_stream)
        ev[2].record(stream)
        sh.copy_(sd, non_blocking=True)
        if leaves:
            ih.copy_(idd, non_blocking=True)
        ev[3].record(stream)
        torch.cuda.synchronize()
        runs.append([ev[0].elapsed_time(ev[3]), ev[0].elapsed_time(ev[1]), ev[1].elapsed_time(ev[2]),
                     ev[2].elapsed_time(ev[3])])
    runs.sort()
    tot, h2d, kern, d2h = runs[len(runs) // 2]
    del Xh, sh, ih, Xd, sd, idd
    torch.cuda.empty_cache()
    return {"ms": tot, "rows_per_s": n / (tot * 1e-3), "h2d_ms": h2d, "kernel_ms": kern, "d2h_ms": d2h,
            "note": "inputs from and outputs to pinned host memory over PCIe; not the bench value"}


def _event_ms(stream, fn, reps):
    """Average time of ``reps`` back-to-back calls of fn, HIP events on ``stream``."""
    import torch
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for _ in range(reps):
        fn()
    ev1.record(stream)
    torch.cuda.synchronize()
    return ev0.elapsed_time(ev1) / reps


def run_sweep():
    """Strategy crossover: every feasible strategy on 100-tree forests of depth
    3, 7, 11 and 12 over 200 or 28 features, at batch sizes 1 to 1M (scores
    only, as a scoring service would call it), each with and without a
    tree-split workspace. One JSON line per point, then a summary of the
    fastest strategy per (model, batch) beside the selector's choice."""
    import torch

    import paper_2010_04804_amd as hb
    from paper_2010_04804_amd import synth

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    nmax = max(synth.SWEEP["batches"])
    scores = torch.empty((nmax, 1), dtype=torch.float32, device=dev)
    table = {}
    xs = {}
    for kind in synth.SWEEP["models"]:
        F = synth.sweep_features(kind)
        if F not in xs:
            xs.clear()
            torch.cuda.empty_cache()
            xs[F] = torch.from_numpy(synth.sweep_rows(nmax, F)).to(dev)
        X = xs[F]
        h = hb.compile(synth.sweep_model(kind), device=0)
        info = h.info()
        for n in synth.SWEEP["batches"]:
            row = {}
            for s in ("gemm", "ptt", "tt"):
                if not info["feasible"][s]:
                    continue
                # each strategy as hb_predict, and as hb_predict_ws with the
                # workspace it can use (the better of the two counts)
                nws = hb.workspace_bytes(h, n, s)
                ws = torch.empty(max(nws, 1), dtype=torch.uint8, device=dev)
                best_ms = None
                for use_ws in ((False, True) if nws else (False,)):
                    fn = lambda: hb.predict_ptr(h, X.data_ptr(), n, scores.data_ptr(), None, s,
                                                stream.cuda_stream, ws.data_ptr() if use_ws else None,
                                                nws if use_ws else 0)
                    fn()
                    torch.cuda.synchronize()
                    probe = _event_ms(stream, fn, 1)
                    reps = int(min(200, max(3, 100.0 / max(probe, 1e-3))))
                    # the best of three averages: at a few microseconds per
                    # call one average carries launch jitter of several percent
                    ms = min(_event_ms(stream, fn, reps) for _ in range(3))
                    print(json.dumps({"sweep": kind, "batch": n, "strategy": s, "workspace": use_ws,
                                      "us": round(ms * 1e3, 2), "rows_per_s": n / (ms * 1e-3), "reps": reps}),
                          flush=True)
                    best_ms = ms if best_ms is None else min(best_ms, ms)
                row[s] = best_ms
            best = min(row, key=row.get)
            table[f"{kind}/{n}"] = {"best": best, "auto": h.select(n),
                                    "us": {k: round(v * 1e3, 2) for k, v in row.items()}}
        h.close()
    print(json.dumps({"sweep_summary": table}), flush=True)


def run_latency(config, batches=(1, 10, 100, 1_000, 10_000, 30_000)):
    """Request-response latency on one workload's model at small batch sizes
    (scores only): back-to-back launches timed with HIP events, and one call
    plus a stream synchronisation timed on the host, both for the eager call
    and for a replay of it captured in a HIP graph. The selector's strategy
    runs with and without a tree-split workspace (hb_predict_ws), and GEMM
    beside it, also both ways."""
    import statistics

    import torch

    import paper_2010_04804_amd as hb
    from paper_2010_04804_amd import synth

    dev = torch.device("cuda:0")
    model = synth.make_model(config)
    h = hb.compile(model, device=0)
    info = h.info()
    K = info["n_outputs"]
    X = torch.from_numpy(synth.make_rows(config, max(batches))).to(dev)
    side = torch.cuda.Stream(dev)
    out = {}
    for n in batches:
        for strat, use_ws in (("auto", False), ("auto", True), ("gemm", False), ("gemm", True)):
            s_name = h.select(n) if strat == "auto" else strat
            if not info["feasible"][s_name]:
                continue
            nws = hb.workspace_bytes(h, n, s_name) if use_ws else 0
            if use_ws and not nws:
                continue
            ws = torch.empty(max(nws, 1), dtype=torch.uint8, device=dev)
            ws_ptr = ws.data_ptr() if nws else None
            scores = torch.empty((n, K), dtype=torch.float32, device=dev)
            with torch.cuda.stream(side):
                fn = lambda: hb.predict_ptr(h, X.data_ptr(), n, scores.data_ptr(), None, s_name,
                                            torch.cuda.current_stream(dev).cuda_stream, ws_ptr, nws)
                for _ in range(3):
                    fn()
                torch.cuda.synchronize()
                ref = scores.clone()
                reps = 200 if s_name != "gemm" else 20
                pipelined = _event_ms(side, fn, reps)
                rt = []
                for _ in range(reps):
                    t0 = time.perf_counter()
                    fn()
                    side.synchronize()
                    rt.append(time.perf_counter() - t0)
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=side):
                hb.predict_ptr(h, X.data_ptr(), n, scores.data_ptr(), None, s_name,
                               side.cuda_stream, ws_ptr, nws)
            grt = []
            for i in range(reps):
                scores.fill_(float("nan"))
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                g.replay()
                torch.cuda.synchronize()
                grt.append(time.perf_counter() - t0)
                if i < 3 and not torch.equal(scores, ref):
                    raise RuntimeError(f"graph replay {i} differs from the eager call (batch {n})")
            key = f"{n}/{s_name}" + ("+ws" if nws else "")
            out[key] = {"pipelined_us": round(pipelined * 1e3, 2),
                        "roundtrip_us_median": round(statistics.median(rt) * 1e6, 2),
                        "roundtrip_us_min": round(min(rt) * 1e6, 2),
                        "graph_roundtrip_us_median": round(statistics.median(grt) * 1e6, 2),
                        "graph_roundtrip_us_min": round(min(grt) * 1e6, 2)}
            print(json.dumps({"latency": key, **out[key]}), flush=True)
            del g
    h.close()
    print(json.dumps({"latency_summary": {"workload": synth.CONFIGS[config]["name"], "points": out}}),
          flush=True)


def run_pruning():
    """Feature selection injection on wide inputs: 500 perfect trees of depth
    8 over 2000-column rows whose decision nodes test 40, 120, 200 or all
    2000 columns, 100,000 rows, PTT with and without leaf ids. The kernels
    stage only the tested columns, so narrower use reaches the row-parallel
    kernel; rows are read whole from HBM either way (the algorithmic bytes)."""
    import torch

    import paper_2010_04804_amd as hb
    from paper_2010_04804_amd import synth

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    n = 100_000
    X = torch.from_numpy(synth.narrow_use_rows(2000, n, seed=3)).to(dev)
    scores = torch.empty((n, 1), dtype=torch.float32, device=dev)
    ids = torch.empty((n, 500), dtype=torch.int32, device=dev)
    for used in (40, 120, 200, 2000):
        h = hb.compile(synth.narrow_use_model(2000, used, 500, 8, seed=3), device=0)
        for leaves in (True, False):
            fn = lambda: hb.predict_ptr(h, X.data_ptr(), n, scores.data_ptr(),
                                        ids.data_ptr() if leaves else None, "ptt", stream.cuda_stream)
            fn()
            torch.cuda.synchronize()
            ms = _event_ms(stream, fn, 10)
            b = n * 2000 * 4 + n * 4 + (n * 500 * 4 if leaves else 0)
            print(json.dumps({"pruning": used, "n_used_features": h.info()["n_used_features"],
                              "leaf_ids": leaves, "ms": round(ms, 4), "rows_per_s": n / (ms * 1e-3),
                              "hbm_frac": b / (ms * 1e-3) / HBM_PEAK}), flush=True)
        h.close()


def run_configs():
    """Every workload (1-5) at its batch size, every feasible strategy, with
    and without leaf ids: ms per call (HIP events), rows/s, and the fraction
    of the roofline that bounds it (HBM for the traversals, int8 MFMA for
    GEMM). One JSON line per point."""
    import torch

    import paper_2010_04804_amd as hb
    from paper_2010_04804_amd import synth

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    for cfg in sorted(synth.CONFIGS) + ["rf2"]:
        if cfg == "rf2":  # beside the five: a binary random forest with vector leaves over narrow rows
            n, name = synth.RF_VECTOR["n_rows"], synth.RF_VECTOR["name"]
            model, rows = synth.rf_vector_model(), synth.rf_vector_rows(n)
        else:
            n, name = synth.CONFIGS[cfg]["n_rows"], synth.CONFIGS[cfg]["name"]
            model, rows = synth.make_model(cfg), synth.make_rows(cfg, n)
        h = hb.compile(model, device=0)
        info = h.info()
        X = torch.from_numpy(rows).to(dev)
        scores = torch.empty((n, info["n_outputs"]), dtype=torch.float32, device=dev)
        ids = torch.empty((n, info["n_trees"]), dtype=torch.int32, device=dev)
        auto = h.select(n)
        for s in ("ptt", "tt", "gemm"):
            if not info["feasible"][s]:
                continue
            for leaves in (True, False):
                fn = lambda: hb.predict_ptr(h, X.data_ptr(), n, scores.data_ptr(),
                                            ids.data_ptr() if leaves else None, s, stream.cuda_stream)
                fn()
                torch.cuda.synchronize()
                probe = _event_ms(stream, fn, 1)
                ms = _event_ms(stream, fn, int(min(20, max(2, 300.0 / max(probe, 1e-3)))))
                if s == "gemm":
                    frac = gemm_ops(model, n) / (ms * 1e-3) / INT8_PEAK
                else:
                    frac = algorithmic_bytes(info, n, leaves, s) / (ms * 1e-3) / HBM_PEAK
                print(json.dumps({"workload": cfg, "name": name, "rows": n,
                                  "strategy": s, "auto": s == auto, "leaf_ids": leaves,
                                  "ms": round(ms, 4), "rows_per_s": n / (ms * 1e-3),
                                  "bound": "mfma" if s == "gemm" else "hbm", "frac": frac,
                                  "kernel": kernel_label(h, s, n)}), flush=True)
        del X, scores, ids
        h.close()
        torch.cuda.empty_cache()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=2, help="workload 1..5 (default 2, the headline)")
    ap.add_argument("--rows", type=int, default=None)
    ap.add_argument("--strategy", default="auto", choices=["auto", "ptt", "tt", "gemm"])
    ap.add_argument("--no-leaves", action="store_true", help="scores only")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--only-main", action="store_true", help="skip the other strategies")
    ap.add_argument("--no-e2e", action="store_true", help="skip the end-to-end timing with host copies")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a 1 GiB device copy (to scale HBM byte counters)")
    ap.add_argument("--sweep", action="store_true",
                    help="strategy crossover sweep (depth 3/7/12, batch 1..1M) instead of the bench line")
    ap.add_argument("--latency", action="store_true",
                    help="small-batch latency (eager and graph-replayed) instead of the bench line")
    ap.add_argument("--batches", default="",
                    help="comma-separated batch sizes for --latency")
    ap.add_argument("--pruning", action="store_true",
                    help="wide inputs whose trees test few columns, instead of the bench line")
    ap.add_argument("--configs", action="store_true",
                    help="every workload and strategy against its roofline, instead of the bench line")
    ap.add_argument("--lds-probe", action="store_true",
                    help="LDS read rates of the traversal walks' read shapes (probe library)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": f"--gpus {args.gpus}: this benchmark runs on one GPU only. Rows are "
                                   "independent, so N GPUs would each score n/N rows with a "
                                   "replica of the compiled tables and no exchange step."}))
        sys.exit(2)

    if args.sweep:
        return run_sweep()
    if args.latency:
        if args.batches:
            return run_latency(args.config, tuple(int(b) for b in args.batches.split(",")))
        return run_latency(args.config)
    if args.pruning:
        return run_pruning()
    if args.configs:
        return run_configs()
    if args.lds_probe:
        return run_lds_probe()

    import torch

    import paper_2010_04804_amd as hb
    from paper_2010_04804_amd import synth

    cfg = args.config
    n = args.rows or synth.CONFIGS[cfg]["n_rows"]
    model = synth.make_model(cfg)
    X = synth.make_rows(cfg, n)
    dev = torch.device("cuda:0")
    h = hb.compile(model, device=0)
    info = h.info()
    strategy = h.select(n) if args.strategy == "auto" else args.strategy
    leaves = not args.no_leaves
    Xd = torch.from_numpy(X).to(dev)
    scores = torch.empty((n, info["n_outputs"]), dtype=torch.float32, device=dev)
    ids = torch.empty((n, info["n_trees"]), dtype=torch.int32, device=dev) if leaves else None
    stream = torch.cuda.current_stream(dev)

    # each strategy gets the workspace the library asks for at this batch
    # size (hb_workspace_bytes: the inputs' ranks for large PTT batches, a
    # tree split for small ones), allocated once, outside the timed calls
    ws = {}
    for s in ("ptt", "tt", "gemm"):
        if info["feasible"][s]:
            nws = hb.workspace_bytes(h, n, s)
            ws[s] = (torch.empty(nws, dtype=torch.uint8, device=dev), nws) if nws else (None, 0)

    def step(strat):
        buf, nws = ws[strat]
        hb.predict_ptr(h, Xd.data_ptr(), n, scores.data_ptr(),
                       ids.data_ptr() if ids is not None else None, strat, stream.cuda_stream,
                       buf.data_ptr() if buf is not None else None, nws)

    per_call = {}

    def timed(strat, steps, warmup):
        """Average launch time in ms, HIP events recorded on the launch stream
        around the K back-to-back calls; an event between every two calls
        also gives the per-call median and minimum (per_call[strat])."""
        for _ in range(warmup):
            step(strat)
        torch.cuda.synchronize()
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
        evs[0].record(stream)
        for i in range(steps):
            step(strat)
            evs[i + 1].record(stream)
        torch.cuda.synchronize()
        calls = sorted(evs[i].elapsed_time(evs[i + 1]) for i in range(steps))
        per_call[strat] = {"median_ms": calls[len(calls) // 2] if steps % 2 else 0.5 * (calls[steps // 2 - 1] + calls[steps // 2]),
                           "min_ms": calls[0]}
        return evs[0].elapsed_time(evs[-1]) / steps

    mfma_measured = mfma_peak_measured()

    def roofline(strat, ms):
        if strat == "gemm":
            ops = gemm_ops(model, n)
            achieved = ops / (ms * 1e-3)
            r = {"bound": "mfma", "achieved": achieved / 1e12, "peak": INT8_PEAK / 1e12,
                 "unit": "TOP/s", "frac": achieved / INT8_PEAK, "traffic": None,
                 "kernel": kernel_label(h, strat, n, ws[strat][1]), "avg_launch_ms": ms, "ops_per_launch": ops}
            if mfma_measured:
                r["peak_measured"] = mfma_measured / 1e12
                r["frac_of_measured"] = achieved / mfma_measured
            return r
        b = algorithmic_bytes(info, n, leaves, strat)
        achieved = b / (ms * 1e-3)
        return {"bound": "hbm", "achieved": achieved / 1e9, "peak": HBM_PEAK / 1e9, "unit": "GB/s",
                "frac": achieved / HBM_PEAK, "traffic": recorded_traffic(cfg, strat, n, leaves),
                "kernel": kernel_label(h, strat, n, ws[strat][1]), "avg_launch_ms": ms, "bytes_per_launch": b}

    print(f"[bench] config {cfg}: {n} rows, strategy {strategy}, leaf ids {leaves}", flush=True)
    t_wall = time.perf_counter()
    ms = timed(strategy, args.steps, args.warmup)
    t_wall = time.perf_counter() - t_wall
    print(f"[bench] {strategy}: {ms:.4f} ms per step", flush=True)
    stats = synth.model_stats(model)
    out = {
        "metric": METRIC, "value": n / (ms * 1e-3), "unit": "rows/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic: seeded random trees and rows of the workload's shape",
        "config": {"workload": synth.CONFIGS[cfg]["name"], "rows": n, "trees": info["n_trees"],
                   "max_depth": stats["max_depth"], "features": info["n_features"],
                   "outputs": info["n_outputs"], "strategy": strategy, "leaf_ids": leaves},
        "roofline": roofline(strategy, ms),
        "per_call_ms": per_call[strategy],
        "timed_wall_s": t_wall,
    }
    if not args.only_main:
        others = {}
        for s in ("ptt", "tt", "gemm"):
            if s == strategy or not info["feasible"][s]:
                continue
            k = args.steps if s != "gemm" else max(2, args.steps // 5)
            mss = timed(s, k, 1)
            print(f"[bench] {s}: {mss:.4f} ms per step", flush=True)
            r = roofline(s, mss)
            others[s] = {"rows_per_s": n / (mss * 1e-3), "ms": mss, "per_call_ms": per_call[s], "bound": r["bound"],
                         "achieved": r["achieved"], "unit": r["unit"], "frac": r["frac"]}
            if "frac_of_measured" in r:
                others[s]["peak_measured"] = r["peak_measured"]
                others[s]["frac_of_measured"] = r["frac_of_measured"]
        out["other_strategies"] = others
    if strategy != "gemm" and not args.copy_calibration:
        # HBM fraction also against what a plain 1 GiB device copy reaches here
        src = torch.empty(1 << 28, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        copy_ms = _event_ms(stream, lambda: dst.copy_(src), 5)
        copy_gbs = 2.0 * (1 << 30) / (copy_ms * 1e-3) / 1e9
        out["roofline"]["copy_GBps_measured"] = copy_gbs
        out["roofline"]["frac_of_copy"] = out["roofline"]["achieved"] / copy_gbs
        del src, dst
    if args.copy_calibration:
        # a plain device copy of exactly 1 GiB, to scale FETCH_SIZE / WRITE_SIZE
        src = torch.empty(1 << 28, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        out["copy_calibration_bytes"] = 1 << 30
    if not args.no_e2e:
        out["end_to_end"] = end_to_end(hb, h, X, n, info, leaves, strategy, dev)
    if not args.no_cpu:
        print("[bench] timing the CPU oracle", flush=True)
        out["cpu_baseline"] = cpu_baseline(model, cfg)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
