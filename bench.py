#!/usr/bin/env python3
"""Benchmark of the sparse-binary BMU search on one MI355X.

One step = one pass of the whole hot path over one synthetic batch: the fp64
codebook norms, then the search (tile plan, fused sweep, finalize) over all N
rows -- the BMU phase of one training epoch. Inputs are resident in HBM
before timing starts. Prints one JSON line.

  python bench.py [--steps K] [--warmup W] [--config 1024|512|256|64|tiny]

The default workload is the 1024x1024 map (M = 1,048,576 neurons, a 125.8 GB
fp32 codebook resident in one GPU's HBM, 500,000 rows): the largest map that
fits one GPU.

Codebook byte counts per step, all counted exactly on the host from the CSR:
  effective (algorithmic)  4*M bytes for every distinct feature of every tile
                           of 16 consecutive rows -- the codebook rows the
                           paper's tiled kernel reads (SpMM-tile kernel
                           section, TA = 16);
  gather                   4*M bytes per id (no reuse inside a tile);
  compulsory               4*M bytes per distinct feature of the batch.
The effective rate exceeds the HBM peak because the sweep serves most of its
rows from L2 and the Infinity Cache. The roofline object therefore divides
the bytes the sweep actually moves past L2 -- the rocprofv3 FETCH_SIZE and
WRITE_SIZE counters of the same workload, calibrated on a plain copy and
committed under profiles/ -- by the sweep's HIP-event time, and compares
that with the 8 TB/s HBM peak (null when no counter record matches the
current kernel source).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
ALG_TILE = 16  # tile size that defines the algorithmic bytes
METRIC = "BMU-search samples/sec + effective codebook HBM GB/s (% of peak) per map size"
# the sources the sweep kernel is compiled from: a counter record is used only while they are unchanged
SWEEP_SRC = [os.path.join(ROOT, "paper_2608_24067_amd", "csrc", f)
             for f in ("som_sweep.hip", "som_device.h", "som_tree16.h", "som_tree8.h")]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def log(msg: str):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for path in SWEEP_SRC:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def counter_record(workload: str):
    """The committed rocprofv3 counter record of the sweep on this workload (fp32 codebook, binary rows, best
    unit, default tile), or None if there is none or the kernel source has changed since it was taken."""
    try:
        with open(TRAFFIC_FILE) as f:
            table = json.load(f)
    except (OSError, ValueError):
        return None
    rec = table.get(workload)
    if not rec or rec.get("kernel_sha256_16") != kernel_source_hash():
        return None
    return rec


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


# oracle rows per workload: about 1.3e11 dense element updates each (5e9 for the tiny map)
CPU_ROWS = {"tiny": 10_000, "64": 1_000, "256": 64, "512": 16, "1024": 4}


def cpu_baseline(cfg, row_ptr, col_idx, W_host, rows: int):
    """The oracle as it stands on the first `rows` rows of the batch over the whole map.

    The headline figure runs the single-threaded oracle with the calling thread
    pinned to one core. The informational all-core figure splits each neuron
    block into one range per host thread and runs the same oracle on each
    (merged by the same rule; the two answers must agree). The codebook is drawn
    block by block (excluded from both timings).
    """
    from concurrent.futures import ThreadPoolExecutor

    import oracle
    import synth

    M, V = cfg.M, cfg.V
    rows = int(max(1, min(rows, cfg.N)))
    rp = np.ascontiguousarray(row_ptr[: rows + 1])
    ci = np.ascontiguousarray(col_idx[: int(rp[-1])])
    block = M if W_host is not None else max(1, min(M, (8 << 30) // (4 * V)))
    threads = synth.default_threads()
    allowed = os.sched_getaffinity(0)
    core = min(allowed)
    t_one = t_all = 0.0
    parts_one, parts_all = [], []
    for i0 in range(0, M, block):
        i1 = min(M, i0 + block)
        blk = W_host if W_host is not None else synth.codebook(cfg.seed, cfg.kind, V, M, i0=i0, i1=i1)
        os.sched_setaffinity(0, {core})  # this thread only: the oracle runs on it
        try:
            t0 = time.perf_counter()
            parts_one.append(oracle.bmu(blk, rp, ci, i0=i0))
            t_one += time.perf_counter() - t0
        finally:
            os.sched_setaffinity(0, allowed)
        width = -(-(i1 - i0) // threads)
        starts = list(range(0, i1 - i0, width))
        with ThreadPoolExecutor(max_workers=len(starts)) as ex:
            t0 = time.perf_counter()
            parts_all.extend(ex.map(lambda k: oracle.bmu(blk[:, k:min(i1 - i0, k + width)], rp, ci, i0=i0 + k),
                                    starts))
            t_all += time.perf_counter() - t0
        log(f"oracle: neurons [{i0}, {i1}) done, {t_one:.1f} s on one core, {t_all:.1f} s on {len(starts)} threads")
        del blk
    one = oracle.merge_blocks(parts_one)
    every = oracle.merge_blocks(parts_all)
    if not all(np.array_equal(x, y) for x, y in zip(one, every)):
        raise RuntimeError("the oracle's one-thread and all-thread answers differ")
    return {
        "value": rows / t_one,
        "unit": "samples/s",
        "cores": 1,
        "kind": "oracle",
        "sample": (f"first {rows} rows of the batch over the whole map (dense fp64 over all V={V} features x "
                   f"M={M} neurons), {t_one:.1f} s on one thread pinned to core {core} of {cpu_model()} "
                   f"({len(allowed)} cores available)"),
        "projected_full_batch_s": cfg.N * t_one / rows,
        "all_cores": {"value": rows / t_all, "unit": "samples/s", "threads": threads,
                      "note": "informational: the same oracle on one neuron range per thread, merged"},
    }


def batch_sha256(row_ptr, col_idx) -> str:
    h = hashlib.sha256()
    h.update(np.ascontiguousarray(row_ptr).view(np.uint8))
    h.update(np.ascontiguousarray(col_idx).view(np.uint8))
    return h.hexdigest()


def versions() -> dict:
    import torch

    out = {"torch": torch.__version__, "hip": getattr(torch.version, "hip", None), "python": platform.python_version()}
    try:
        with open("/opt/rocm/.info/version") as f:
            out["rocm"] = f.read().strip()
    except OSError:
        pass
    return out


def device_facts(dev) -> dict:
    """What the runtime reports about the GPU the bench ran on."""
    import torch

    p = torch.cuda.get_device_properties(dev)
    out = {"name": p.name, "arch": getattr(p, "gcnArchName", ""), "compute_units": p.multi_processor_count,
           "hbm_GB": round(p.total_memory / 1e9, 1)}
    l2 = getattr(p, "L2_cache_size", None)
    if l2:
        out["l2_MB_per_xcd"] = round(l2 / 2**20, 1)
    return out


def sustained_read(dev, reps: int = 5) -> float:
    """HBM read bandwidth a plain stream reaches on this GPU: GB/s of the read-stream probe
    (16-byte loads, eight in flight per thread) over a 4 GiB buffer, far beyond the 256 MB
    MALL; the best of `reps` runs at each of 4, 8, 16 and 32 workgroups per CU. The measured
    denominator beside the published 8 TB/s."""
    import ctypes

    import torch

    from paper_2608_24067_amd import build as pkg_build

    if not os.path.exists(pkg_build.PROBE_LIB):
        raise RuntimeError(f"{pkg_build.PROBE_LIB} is missing: run __graft_entry__.build() first")
    lib = ctypes.CDLL(pkg_build.PROBE_LIB)
    lib.somprobe_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p]
    lib.somprobe_read.restype = ctypes.c_int
    nbytes = 4 << 30
    x = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
    sink = torch.zeros(1, dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream(dev)

    def run(per_cu):
        rc = lib.somprobe_read(x.data_ptr(), nbytes, sink.data_ptr(), per_cu, ctypes.c_void_p(stream.cuda_stream))
        if rc != 0:
            raise RuntimeError(f"somprobe_read failed ({rc})")

    best = float("inf")
    for per_cu in (4, 8, 16, 32):
        run(per_cu)
        torch.cuda.synchronize()
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            run(per_cu)
            e1.record(stream)
            torch.cuda.synchronize()
            best = min(best, e0.elapsed_time(e1))
    del x, sink
    torch.cuda.empty_cache()
    return nbytes / (best / 1e3) / 1e9


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", default="1024",
                    help="tiny, 64, 256, 512 or 1024 (default 1024: the 1024x1024 map, the largest that fits one GPU)")
    ap.add_argument("--tile", type=int, default=0, help="tile_samples passed to the library (0 = default)")
    ap.add_argument("--cpu-rows", type=int, default=0,
                    help="oracle rows for cpu_baseline (0 = the workload's default: 4 rows at 1024x1024, 16 at 512x512, "
                         "64 at 256x256, 1,000 at 64x64, all 10,000 of the tiny map)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--dtype", choices=("f32", "f16"), default="f32",
                    help="codebook storage: fp32 (the workloads' own) or fp16 (rounded from it; fp32 accumulation)")
    ap.add_argument("--values", action="store_true",
                    help="sparse real-valued rows: a U(0,1] value with every id (the gather-multiply variant)")
    ap.add_argument("--epoch", action="store_true",
                    help="time one whole batch-SOM epoch: the two-best search plus the batch update (first-epoch radius)")
    ap.add_argument("--update-chunk-gb", type=float, default=16.0, help="workspace budget of the update, GB")
    ap.add_argument("--top2", action="store_true",
                    help="time the two-best search (som_bmu2_*) instead of the single-best one")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="first run one plain 1 GiB device-to-device copy, the reference for HBM byte counters")
    args = ap.parse_args()
    if args.epoch:
        args.top2 = True

    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only: sharding over samples or neuron ranges "
                                   "is designed but not built", "n_gpus": args.gpus}))
        sys.exit(2)

    import torch

    import paper_2608_24067_amd.som as som
    import synth

    cfg = synth.CONFIGS[args.config]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    M, V, N = cfg.M, cfg.V, cfg.N

    t0 = time.perf_counter()
    row_ptr, col_idx = synth.make_csr(cfg.seed, N, V, cfg.lam, cfg.zipf_s)
    nnz = int(row_ptr[-1])
    alg_rows = int(synth.tile_distinct(row_ptr, col_idx, ALG_TILE).astype(np.int64).sum())
    elem = 2 if args.dtype == "f16" else 4
    alg_bytes = float(elem) * M * alg_rows
    distinct_ids = int(np.count_nonzero(np.bincount(col_idx, minlength=V)))
    gather_bytes = float(elem) * M * nnz
    min_bytes = float(elem) * M * distinct_ids
    data_sha = batch_sha256(row_ptr, col_idx)
    log(f"csr: N={N} nnz={nnz} distinct rows per 16-row tile total={alg_rows}, distinct ids {distinct_ids} "
        f"({time.perf_counter() - t0:.1f} s)")

    t0 = time.perf_counter()
    keep_host = 4 * V * M <= (2 << 30)
    if keep_host:
        W_host = synth.codebook(cfg.seed, cfg.kind, V, M)
        if args.dtype == "f16":
            W_host = W_host.astype(np.float16)
            W = torch.from_numpy(W_host).to(dev)
            W_host = W_host.astype(np.float32)  # the values the oracle sees: exact widening
        else:
            W = torch.from_numpy(W_host).to(dev)
    else:
        W_host = None
        W = synth.codebook_to_device(cfg.seed, cfg.kind, V, M, dev,
                                     dtype=torch.float16 if args.dtype == "f16" else torch.float32)
    rp = torch.from_numpy(row_ptr).to(dev)
    ci = torch.from_numpy(col_idx).to(dev)
    norms = torch.empty(M, dtype=torch.float64, device=dev)
    bmu = torch.empty(N, dtype=torch.int32, device=dev)
    dist = torch.empty(N, dtype=torch.float64, device=dev)
    if args.values:
        vals_d = torch.from_numpy(synth.values(cfg.seed, nnz)).to(dev)
        alloc = som.alloc_workspace_sf
    else:
        alloc = som.alloc_workspace2 if args.top2 else som.alloc_workspace
    ws = alloc(N, M, V, nnz, dev, tile_samples=args.tile)
    if args.top2:
        out2 = (bmu, dist, torch.empty(N, dtype=torch.int32, device=dev), torch.empty(N, dtype=torch.float64, device=dev))
    torch.cuda.synchronize()
    log(f"inputs resident: codebook {elem * V * M / 1e9:.2f} GB, workspace {ws.numel() / 1e9:.2f} GB "
        f"({time.perf_counter() - t0:.1f} s)")

    if args.calibrate_copy:
        src = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        log("calibration copy: 1073741824 bytes read, 1073741824 bytes written")

    sustained = sustained_read(dev)
    log(f"sustained HBM read (read-stream probe over 4 GiB): {sustained:.0f} GB/s")

    if args.epoch:
        r_epoch = som.radius(som.sigma(1, 0.5 * cfg.edge, 0.5))
        chunk = int(max(1, min(V, args.update_chunk_gb * 1e9 / (12.0 * M))))
        uws = torch.empty(som.update_workspace_bytes(V, cfg.edge, N, chunk), dtype=torch.uint8, device=dev)
        log(f"update: radius {r_epoch}, {chunk} features per chunk, workspace {uws.numel() / 1e9:.2f} GB")
    phases = ("norms", "plan", "sweep", "finalize") + (("update",) if args.epoch else ())

    def step(ev=None):
        if ev is not None:
            ev[0].record()
        som.codebook_norms(W, V, M, out=norms)
        if ev is not None:
            ev[1].record()
        if args.values:
            som.bmu_sf_plan(rp, ci, vals_d, V, M, nnz, ws, tile_samples=args.tile)
        else:
            som.bmu_plan(rp, ci, V, M, nnz, ws, tile_samples=args.tile)
        if ev is not None:
            ev[2].record()
        if args.values:
            som.bmu_sf_sweep(W, norms, V, M, N, nnz, ws, two_best=args.top2, tile_samples=args.tile)
        elif args.top2:
            som.bmu2_sweep(W, norms, V, M, N, nnz, ws, tile_samples=args.tile)
        else:
            som.bmu_sweep(W, norms, V, M, N, nnz, ws, tile_samples=args.tile)
        if ev is not None:
            ev[3].record()
        if args.values:
            som.bmu_sf_finalize(norms, rp, V, M, nnz, out2 if args.top2 else (bmu, dist), ws, tile_samples=args.tile)
        elif args.top2:
            som.bmu2_finalize(norms, rp, V, M, nnz, out2, ws, tile_samples=args.tile)
        else:
            som.bmu_finalize(norms, rp, V, M, nnz, bmu, dist, ws, tile_samples=args.tile)
        if ev is not None:
            ev[4].record()
        if args.epoch:
            som.update(W, rp, ci, bmu, V, cfg.edge, r_epoch, nnz=nnz, chunk_features=chunk, workspace=uws)
            if ev is not None:
                ev[5].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    events = [[torch.cuda.Event(enable_timing=True) for _ in range(len(phases) + 1)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for k in range(args.steps):
        step(events[k])
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    log(f"timed {args.steps} steps in {elapsed:.3f} s")
    if som.input_flags(ws, N, M, V, nnz, tile_samples=args.tile) != 0:
        raise RuntimeError("the device flagged the generated CSR as invalid")

    phase_ms = {p: float(np.mean([e[i].elapsed_time(e[i + 1]) for e in events])) for i, p in enumerate(phases)}
    step_ms = float(np.mean([e[0].elapsed_time(e[len(phases)]) for e in events]))
    ms_per_step = 1e3 * elapsed / args.steps
    value = N / (ms_per_step / 1e3)
    eff_gbps = alg_bytes / (ms_per_step / 1e3) / 1e9
    sweep_s = phase_ms["sweep"] / 1e3
    alg_rate = alg_bytes / sweep_s / 1e9
    workload = cfg.describe()
    # the committed counter runs are of the default variant: fp32, binary rows, best unit, default tile
    default_variant = not (args.top2 or args.values or args.epoch or args.dtype != "f32"
                           or args.tile not in (0, som.DEFAULT_TILE_SAMPLES))
    rec = counter_record(args.config) if default_variant else None
    traffic = rec.get("hbm_bytes_per_launch") if rec else None
    achieved = traffic / sweep_s / 1e9 if traffic else None
    l2_hit = rec.get("l2_hit_rate") if rec else None

    out = {
        "metric": METRIC,
        "value": value,
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": ("f16 codebook, " if args.dtype == "f16" else "") + "f32 sums, f64 norms and distances",
        "data": "synthetic (seeded stand-in for the MEDLINE/MeSH corpus)",
        "config": {"workload": workload, "map": f"{cfg.edge}x{cfg.edge}", "M": M, "V": V, "N": N, "nnz": nnz,
                   "tile_samples": args.tile or som.DEFAULT_TILE_SAMPLES,
                   "keep_order": False, "alg_tile_samples": ALG_TILE, "parallelism": "single GPU",
                   "search": ("two best units + batch update (one epoch)" if args.epoch else
                              "two best units" if args.top2 else "best unit"), "codebook": args.dtype,
                   "rows": "real-valued" if args.values else "binary"},
        # the metric's second half: effective (algorithmic) codebook bytes over the whole step; they are mostly
        # served from L2 and the Infinity Cache, so this rate is not a fraction of what HBM delivers
        "effective_codebook_GBps": eff_gbps,
        "effective_vs_hbm_peak": eff_gbps / HBM_PEAK_GBPS,
        "codebook_bytes_per_step": {"effective_alg": alg_bytes, "gather": gather_bytes, "compulsory": min_bytes,
                                    "distinct_ids": distinct_ids},
        "sweep_rates_GBps": {"effective_alg": alg_rate, "gather": gather_bytes / sweep_s / 1e9,
                             "compulsory": min_bytes / sweep_s / 1e9},
        "hbm_read_sustained_GBps": sustained,
        "sweep_alg_vs_sustained": alg_rate / sustained,
        "sweep_l2_hit_rate": l2_hit,
        "device": device_facts(dev),
        "versions": versions(),
        "data_sha256": data_sha,
        "event_ms_per_step": step_ms,
        "phase_ms": phase_ms,
        "roofline": {"bound": "hbm", "kernel": "k_sweep" + (" (real values)" if args.values else "")
                     + (" (two-best)" if args.top2 else ""),
                     "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS if achieved else None,
                     "traffic": traffic,
                     "basis": ("bytes past L2 per sweep launch (rocprofv3 FETCH_SIZE and WRITE_SIZE, calibrated on a "
                               "plain copy; served by the Infinity Cache or HBM) / HIP-event sweep time"),
                     "algorithmic_bytes": alg_bytes, "algorithmic_GBps": alg_rate},
    }
    if not args.no_cpu_baseline:
        log("timing the oracle (cpu_baseline)")
        out["cpu_baseline"] = cpu_baseline(cfg, row_ptr, col_idx, W_host, args.cpu_rows or CPU_ROWS[args.config])
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
