"""Throughput of the SCRAM hot path on one MI355X.

A step is one pass of the whole path over one batch of resident synthetic
input: PatchMatch (random init + T Jacobi sweeps, one library call) then the
sparse window attention (one call), on the 256x256, d=64, bf16, 4-slice
workload by default.  ``--kappa K`` runs K constrained PatchMatch runs (run c
given the maps of runs 0..c-1, separation ``--sep``) and attends over the
union of their windows; ``--causal`` masks keys after each query;
``--snis T`` replaces the window softmax by the importance-sampling estimate
with T samples per query (``--alpha``, ``--radius``); ``--backward`` adds the
gradients of the window attention to every step.  Two timed regions: A runs the steps as a caller would
(throughput: ``value``, ``ms_per_step``); B runs the same steps with every
kernel dispatch stamping caller-created HIP start/stop events on the launch
stream (per-kernel durations for ``kernels_ms`` and ``roofline``; the stamps
add small gaps between kernels, which is why A is timed separately).

Prints one JSON line.  ``--gpus N`` with N > 1 exits: this path runs on one
GPU (independent slices would shard across GPUs with no communication).
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import re
import statistics
import sys
import time
import warnings

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "queries/sec (PatchMatch argmax + sparse attend), 256×256 grid d=64; HBM GB/s"
HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E, public spec
BF16_MFMA_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix peak, public spec
CSRC = os.path.join(ROOT, "paper_1905_10308_amd", "csrc")
# the sources of each timed kernel: its traffic record holds only while they are unchanged
KERNEL_SRCS = {
    "pm_iter": ("scram_device.h", "scram_pm.hip"),
    "attend": ("scram_device.h", "scram_tile.h", "scram_attend.hip"),
}
# how each timed kernel appears in a rocprofv3 trace (its function name)
KERNEL_NAMES = {
    "pm_iter": re.compile(r"::pm_iter_kernel<"),
    "attend": re.compile(r"::attend(_window|_tile)?_kernel<"),
}
COPY_NAME = re.compile(r"neg_kernel")  # the known-size reference kernel of --copy-calibration (torch.neg)
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def pm_bytes_per_query_sweep(cfg, n_prev: int = 0) -> int:
    """Algorithmic bytes of one query in one sweep: its q row, C candidate key
    rows, 4 B each for the previous index and score read and the new index
    and score written, and 4 B per previous run's match."""
    row = cfg.d * cfg.elem_bytes
    return row * (1 + cfg.candidates) + 16 + 4 * n_prev


def attend_bytes_per_query(cfg, kappa: int = 1) -> int:
    """q row, kappa windows of w^2 key rows and w^2 value rows (every window
    read in full), kappa 4 B indices, the output row."""
    row = cfg.d * cfg.elem_bytes
    return row * (2 + 2 * kappa * cfg.window ** 2) + 4 * kappa


def snis_bytes_per_query(cfg, samples: int, kappa: int = 1) -> int:
    """q row, T key rows and T value rows, kappa 4 B modes, the output row."""
    row = cfg.d * cfg.elem_bytes
    return row * (2 + 2 * samples) + 4 * kappa


def kernel_source_hash(kernel: str = "pm_iter") -> str:
    h = hashlib.sha256()
    for name in KERNEL_SRCS[kernel]:
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def load_traffic(cfg, kernel: str = "pm_iter"):
    """The measured traffic record of ``kernel`` on this workload -- bytes past L2 per launch from
    copy-calibrated FETCH_SIZE + WRITE_SIZE -- if it was taken on the kernel's current source; else None."""
    try:
        with open(TRAFFIC_FILE) as f:
            records = json.load(f)["records"]
    except (OSError, ValueError, KeyError):
        return None
    for r in records:
        if r.get("workload") == cfg.name and r.get("kernel") == kernel and \
                r.get("kernel_source_sha256_16") == kernel_source_hash(kernel):
            return r
    return None


def _per_dispatch(path, counter):
    """{dispatch id: (kernel name, summed counter value)} from a rocprofv3 counter-collection CSV."""
    out = {}
    with open(path, newline="") as f:
        for row in csv.DictReader(f):
            if row["Counter_Name"] != counter:
                continue
            d = row["Dispatch_Id"]
            name, v = out.get(d, (row["Kernel_Name"], 0.0))
            out[d] = (name, v + float(row["Counter_Value"]))
    return out


def record_traffic(cfg, fetch_csv: str, write_csv: str, stats_csv: str | None, copy_mib: int) -> list:
    """Turn two rocprofv3 --pmc runs of this bench (FETCH_SIZE, then WRITE_SIZE; KiB per dispatch) into
    traffic records of the timed kernels, written to ``profiles/traffic.json``.

    Each counter is scaled by what it reads for the --copy-calibration kernel, which reads and writes
    exactly ``copy_mib`` MiB; a kernel's bytes per launch are the mean over its dispatches.  With the
    --kernel-trace --stats CSV of the same command, the rocprof mean duration is kept beside them."""
    fetch, write = _per_dispatch(fetch_csv, "FETCH_SIZE"), _per_dispatch(write_csv, "WRITE_SIZE")

    def mean_of(table, pattern):
        vals = [v for name, v in table.values() if pattern.search(name)]
        if not vals:
            raise ValueError(f"no dispatch of {pattern.pattern} in the counter file")
        return sum(vals) / len(vals), len(vals)

    (cf, _), (cw, _) = mean_of(fetch, COPY_NAME), mean_of(write, COPY_NAME)
    fs, ws = copy_mib * 1024 / cf, copy_mib * 1024 / cw
    stats = {}
    if stats_csv:
        with open(stats_csv, newline="") as f:
            for row in csv.DictReader(f):
                for k, pat in KERNEL_NAMES.items():
                    if pat.search(row["Name"]):
                        calls, tot = stats.get(k, (0, 0.0))
                        stats[k] = (calls + int(row["Calls"]), tot + float(row["TotalDurationNs"]))
    new = []
    for k, pat in KERNEL_NAMES.items():
        try:
            (f_kib, nf), (w_kib, nw) = mean_of(fetch, pat), mean_of(write, pat)
        except ValueError:
            continue
        rec = {"workload": cfg.name, "kernel": k, "kernel_source_sha256_16": kernel_source_hash(k),
               "bytes_per_launch": (f_kib * fs + w_kib * ws) * 1024, "read_bytes_per_launch": f_kib * fs * 1024,
               "write_bytes_per_launch": w_kib * ws * 1024, "dispatches": [nf, nw], "fetch_scale": fs,
               "write_scale": ws}
        if k in stats:
            rec["rocprof_avg_ns"] = stats[k][1] / stats[k][0]
        new.append(rec)
    try:
        with open(TRAFFIC_FILE) as f:
            records = json.load(f)["records"]
    except (OSError, ValueError, KeyError):
        records = []
    keep = [r for r in records if (r.get("workload"), r.get("kernel")) not in {(n["workload"], n["kernel"]) for n in new}]
    with open(TRAFFIC_FILE, "w") as f:
        json.dump({"note": "bytes past L2 per launch: FETCH_SIZE and WRITE_SIZE (KiB per dispatch) scaled by "
                           "their reading for a copy of known size; written by bench.py --record-traffic",
                   "records": keep + new}, f, indent=1)
        f.write("\n")
    return new


def roofline_entry(cfg, kernel: str, launch_ms: float, requested_bytes: float, with_traffic: bool) -> dict:
    """The HBM roofline of one kernel: measured bytes past L2 per launch (its traffic record) over the
    live mean launch time, against the 8 TB/s peak.  The bytes past L2 include Infinity-Cache hits, so
    actual HBM bytes are at most these and the fraction cannot exceed 1 by more than counter noise.  The
    requested bytes (every row the algorithm names, the nominal count) are reported beside them: they
    are mostly served by the L1 and L2 caches, so their rate is a cache-level figure, not an HBM one."""
    rec = load_traffic(cfg, kernel) if with_traffic else None
    measured = None if rec is None else rec["bytes_per_launch"]
    achieved = None if measured is None else measured / (launch_ms * 1e-3) / 1e9
    return {
        "bound": "hbm",
        "kernel": kernel,
        "achieved": achieved,
        "peak": HBM_PEAK_GBPS,
        "unit": "GB/s",
        "frac": None if achieved is None else achieved / HBM_PEAK_GBPS,
        "traffic": achieved,
        "traffic_bytes_per_launch": measured,
        "launch_ms": launch_ms,
        "rocprof_launch_ms": None if rec is None or "rocprof_avg_ns" not in rec else rec["rocprof_avg_ns"] * 1e-6,
        "requested_bytes_per_launch": requested_bytes,
        "requested_GBps": requested_bytes / (launch_ms * 1e-3) / 1e9,
        "basis": "achieved = bytes past L2 per launch (copy-calibrated FETCH_SIZE + WRITE_SIZE, "
                 "profiles/traffic.json, tied to the kernel's source hash) / live mean launch time",
    }


def map_quality(cfg, Q, K, J, per_slice: int = 4096, seed: int = 3):
    """Quality of a final map, outside the timed regions: recall against the exact argmax over all keys
    (fp64 products on the GPU, the first index among equal maxima) and the mean ratio of the map's
    score to the exact maximum, on ``per_slice`` sampled queries of each slice.  A comparator, like the
    dense attention timing; the paper prints no quality figure for these workloads."""
    import torch

    gen = torch.Generator(device="cpu").manual_seed(seed)
    plane, nk = cfg.Hq * cfg.Wq, cfg.Hk * cfg.Wk
    hits = total = 0
    ratios = []
    for s in range(cfg.S):
        ids = torch.randperm(plane, generator=gen)[:per_slice].to(Q.device)
        q = Q[s].reshape(plane, cfg.d)[ids].double()
        kt = K[s].reshape(nk, cfg.d).double().t().contiguous()
        jm = J[s].reshape(plane)[ids].long()
        step = max(1, min(1024, (1 << 27) // nk))  # score rows per product: at most 1 GiB of fp64 scores
        for c0 in range(0, ids.numel(), step):
            sc = q[c0:c0 + step] @ kt
            best, arg = sc.max(dim=1)
            mine = sc.gather(1, jm[c0:c0 + step, None]).squeeze(1)
            hits += int((arg == jm[c0:c0 + step]).sum())
            total += arg.numel()
            pos = best > 0
            ratios.append(mine[pos] / best[pos])
    return {"recall_vs_exact_argmax": hits / total, "mean_score_ratio": float(torch.cat(ratios).mean()),
            "sample": f"{min(per_slice, plane)} queries per slice ({total} in all), exact argmax from fp64 "
                      "products on the GPU"}


EXTRA_PM_SEEDS = (1, 2, 3)


def quality_over_seeds(cfg, Q, K, iters, first, workspace, seeds=EXTRA_PM_SEEDS):
    """Spread of the final map's quality over PatchMatch seeds: extra runs with ``seeds`` (outside the
    timed regions), each scored on the same sampled queries as ``first`` (the run with the workload's
    own seed)."""
    import paper_1905_10308_amd as scram
    import torch

    runs = [(cfg.pm_seed, first)]
    for sd in seeds:
        Jx = torch.empty((cfg.S, cfg.Hq, cfg.Wq), dtype=torch.int32, device=Q.device)
        scram.patchmatch(Q, K, iters, sd, out=Jx, workspace=workspace)
        runs.append((sd, map_quality(cfg, Q, K, Jx)))
    rec = [q["recall_vs_exact_argmax"] for _, q in runs]
    rat = [q["mean_score_ratio"] for _, q in runs]
    return {"seeds": [sd for sd, _ in runs], "recall": rec, "recall_mean": statistics.fmean(rec),
            "recall_std": statistics.stdev(rec), "mean_score_ratio": rat,
            "mean_score_ratio_mean": statistics.fmean(rat), "mean_score_ratio_std": statistics.stdev(rat)}


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(cfg, arrays, min_s: float, kappa: int = 1, sep: int = 1, causal: bool = False, snis=None,
                 threads: int | None = None):
    """The fp64 oracle on the host cores, on whole slices of the same workload.

    Slices are run in turn (wrapping around) until at least ``min_s`` seconds
    of oracle work have been timed, so the rate is stable but the run bounded.
    ``threads`` sets the oracle's OpenMP thread count for this run (default:
    what the runtime gives it, i.e. OMP_NUM_THREADS or every core).
    """
    import numpy as np

    import oracle

    before = oracle.num_threads()
    if threads is not None:
        oracle.set_num_threads(threads)
    used = oracle.num_threads()
    flags = oracle.CAUSAL if causal else 0
    Q, K, V = (arrays[k].astype(np.float64) for k in ("Q", "K", "V"))
    done_q, elapsed, runs, scored = 0, 0.0, 0, 0
    per_slice = cfg.Hq * cfg.Wq
    try:
        while elapsed < min_s and runs < 64 * cfg.S:
            s = runs % cfg.S
            t0 = time.perf_counter()
            maps = []  # kappa constrained runs; the oracle counts the valid candidates it scores
            for _ in range(kappa):
                J1, _, _, ncand = oracle.patchmatch(Q[s:s + 1], K[s:s + 1], cfg.iters, cfg.pm_seed, flags=flags,
                                                    prev=np.stack(maps) if maps else None, sep=sep)
                maps.append(J1)
                scored += ncand
            J = np.stack(maps)
            if snis:
                T, alpha, radius = snis
                oracle.snis(Q[s:s + 1], K[s:s + 1], V[s:s + 1], J, T, alpha, radius, cfg.scale, cfg.pm_seed,
                            flags=flags)
            else:
                oracle.sparse_attend(Q[s:s + 1], K[s:s + 1], V[s:s + 1], J, cfg.window, cfg.scale, flags=flags)
            elapsed += time.perf_counter() - t0
            done_q += per_slice
            runs += 1
    finally:
        oracle.set_num_threads(before)
    return {
        "value": done_q / elapsed,
        "unit": "queries/s",
        "cores": used,
        "kind": "oracle",
        "candidates_per_query_sweep": scored / (done_q * kappa * cfg.iters),
        "sample": f"{runs} slice passes over the {cfg.S}-slice workload ({done_q} queries; {kappa} x {cfg.iters} "
                  f"sweeps + " + (f"{snis[0]}-sample SNIS" if snis else f"{cfg.window}x{cfg.window} attend")
                  + f" each), fp64, {used} thread{'s' if used > 1 else ''}, {elapsed:.1f} s",
    }


def copy_bandwidth(device, mib: int = 1024, reps: int = 10) -> float:
    """Achievable HBM bandwidth on this device: a plain device-to-device copy of ``mib`` MiB (read + write
    bytes / time), for context beside the published peak."""
    import torch

    src = torch.empty(mib << 20, dtype=torch.uint8, device=device)
    dst = torch.empty_like(src)
    dst.copy_(src)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        dst.copy_(src)
    b.record()
    b.synchronize()
    gbps = 2 * src.numel() * reps / (a.elapsed_time(b) * 1e-3) / 1e9
    del src, dst
    return gbps


def dense_attention(cfg, Q, K, V, reps: int | None = None):
    """Dense exact softmax attention over the same slices, for scale: torch's
    scaled-dot-product attention restricted in turn to each of its fused
    kernels (flash, memory efficient), so no n x n matrix is formed.  Each
    backend that runs is timed; the fastest is the comparator.  Its matrix
    work is 4 * S * nq * nk * d flops (QK^T and PV), reported against the
    bf16 matrix-core peak.  None if no backend runs."""
    import torch
    from torch.nn.attention import SDPBackend, sdpa_kernel

    S, n = cfg.S, cfg.Hq * cfg.Wq
    q = Q.reshape(S, 1, n, cfg.d).contiguous()
    k = K.reshape(S, 1, cfg.Hk * cfg.Wk, cfg.d).contiguous()
    v = V.reshape(S, 1, cfg.Hk * cfg.Wk, cfg.dv).contiguous()
    flops = 4.0 * S * n * cfg.Hk * cfg.Wk * cfg.d
    if reps is None:
        reps = 1 if flops > 1e15 else 3  # seconds per call on the largest grids
    timed = {}
    for backend in (SDPBackend.FLASH_ATTENTION, SDPBackend.EFFICIENT_ATTENTION):
        try:
            # a backend that cannot take these shapes says why in a warning, then raises: it is skipped
            with warnings.catch_warnings(), sdpa_kernel([backend]):
                warnings.simplefilter("ignore", UserWarning)
                torch.nn.functional.scaled_dot_product_attention(q, k, v, scale=cfg.scale)
                torch.cuda.synchronize()
                start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                start.record()
                for _ in range(reps):
                    torch.nn.functional.scaled_dot_product_attention(q, k, v, scale=cfg.scale)
                stop.record()
                torch.cuda.synchronize()
        except RuntimeError:
            continue
        ms = start.elapsed_time(stop) / reps
        tflops = flops / (ms * 1e-3) / 1e12
        timed[backend.name.lower()] = {"ms": ms, "TFLOPs": tflops,
                                       "frac_of_bf16_mfma_peak": tflops / BF16_MFMA_PEAK_TFLOPS}
    if not timed:
        return None
    best = min(timed, key=lambda b: timed[b]["ms"])
    return {"ms": timed[best]["ms"], "backend": f"torch SDPA {best}", "dtype": str(q.dtype).replace("torch.", ""),
            "flops": flops, "backends": timed}


def progress(msg: str) -> None:
    """A progress line on stderr (stdout carries only the JSON line)."""
    print(f"bench.py: {msg}", file=sys.stderr, flush=True)


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default=None,
                    help="workload index or name (default: the 256x256 bf16 one; large2048_bf16: one 2048x2048 "
                         "slice whose working set exceeds the Infinity Cache)")
    ap.add_argument("--kappa", type=int, default=1, help="matches per query (constrained PatchMatch runs)")
    ap.add_argument("--sep", type=int, default=1, help="separation between the runs' matches (Chebyshev)")
    ap.add_argument("--causal", action="store_true", help="mask keys after each query (raster order)")
    ap.add_argument("--snis", type=int, default=0, metavar="T",
                    help="estimate with T importance samples per query instead of the window softmax")
    ap.add_argument("--backward", action="store_true", help="add the attend backward (maps held fixed) to each step")
    ap.add_argument("--graph", action="store_true",
                    help="capture one step in a HIP graph and time its replays (region A)")
    ap.add_argument("--alpha", type=float, default=0.9, help="SNIS mixture weight of the local densities")
    ap.add_argument("--radius", type=int, default=4, help="SNIS binomial radius m (variance m/2)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="seconds of oracle work for the CPU baseline")
    ap.add_argument("--cpu-seconds-1t", type=float, default=3.0,
                    help="seconds of single-thread oracle work for the CPU baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="before timing, run one plain device copy of this many MiB (a known-size "
                         "reference kernel for hardware byte counters)")
    ap.add_argument("--record-traffic", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="no benchmark: write the traffic records of the workload's timed kernels from the "
                         "counter CSVs of two rocprofv3 --pmc runs of this bench (FETCH_SIZE, then WRITE_SIZE, "
                         "both with --copy-calibration MIB) into profiles/traffic.json")
    ap.add_argument("--stats-csv", default=None,
                    help="with --record-traffic: the kernel_stats CSV of a --kernel-trace --stats run of the "
                         "same command, whose mean kernel durations are kept in the record")
    args = ap.parse_args(argv)

    if args.record_traffic:
        import scram_inputs as si

        if args.copy_calibration <= 0:
            print("bench.py: --record-traffic needs the --copy-calibration MIB of the profiled runs", file=sys.stderr)
            return 2
        cfg = si.get(si.HEADLINE if args.config is None else args.config)
        for r in record_traffic(cfg, *args.record_traffic, args.stats_csv, args.copy_calibration):
            print(json.dumps(r), flush=True)
        return 0
    if args.gpus != 1:
        print(f"bench.py: this path runs on one GPU; --gpus {args.gpus} is not supported "
              "(slices are independent and would shard across GPUs without communication)", file=sys.stderr)
        return 2
    if int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py: launched with WORLD_SIZE > 1; this path runs on one GPU", file=sys.stderr)
        return 2

    import torch

    import paper_1905_10308_amd as scram
    import scram_inputs as si

    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        return 1
    scram.lib()
    if args.copy_calibration > 0:
        # an elementwise kernel that reads and writes exactly MIB MiB each (a
        # same-dtype copy_ would go to the runtime's blit path instead)
        src = torch.ones(args.copy_calibration << 18, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        torch.neg(src, out=dst)
        torch.cuda.synchronize()
        del src, dst
    cfg = si.get(si.HEADLINE if args.config is None else args.config)
    progress(f"generating {cfg.describe()}")
    data = si.make(cfg, device="cuda")
    progress("inputs resident; timing")
    Q, K, V = data["Q"], data["K"], data["V"]
    S, Hq, Wq = cfg.S, cfg.Hq, cfg.Wq
    dev = Q.device
    stream = torch.cuda.current_stream(dev)

    kappa, sep, causal = args.kappa, args.sep, args.causal
    J = torch.empty((kappa, S, Hq, Wq), dtype=torch.int32, device=dev)
    ws = torch.empty(scram.patchmatch_workspace_bytes(S, Hq, Wq), dtype=torch.uint8, device=dev)
    out = torch.empty((S, Hq, Wq, cfg.dv), dtype=Q.dtype, device=dev)
    T = cfg.iters
    per_run = 2 * (T + 1)  # events of one PatchMatch call: init, T sweeps
    n_bwd_ev = 6 if args.backward else 0
    if args.backward and args.snis:
        print("bench.py: --backward applies to the window attention, not to --snis", file=sys.stderr)
        return 2
    dO = torch.randn((S, Hq, Wq, cfg.dv), generator=torch.Generator(device=dev).manual_seed(7), device=dev,
                     dtype=torch.float32).to(Q.dtype) if args.backward else None
    bwd_ws = torch.empty(scram.sparse_attend_backward_workspace_bytes(S, Hq, Wq, cfg.Hk, cfg.Wk, kappa, d=cfg.d,
                                                                      dtype=Q.dtype),
                         dtype=torch.uint8, device=dev) if args.backward else None

    def new_events():
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(kappa * per_run + 2 + n_bwd_ev)]
        for e in evs:  # create the underlying HIP events before handing them to the library
            e.record(stream)
        return evs

    def step(ev=None):
        # the dispatches stamp start/stop events: per run init and T sweeps, then attend
        for c in range(kappa):
            scram.patchmatch(Q, K, T, cfg.pm_seed, prev=J[:c] if c else None, sep=sep, causal=causal, out=J[c],
                             workspace=ws, events=None if ev is None else ev[c * per_run:(c + 1) * per_run])
        maps = J if kappa > 1 else J[0]
        a0 = kappa * per_run  # the attend step's events
        if args.snis:
            scram.snis_attend(Q, K, V, maps, args.snis, alpha=args.alpha, radius=args.radius, scale=cfg.scale,
                              seed=cfg.pm_seed, causal=causal, out=out, events=None if ev is None else ev[a0:a0 + 2])
        else:
            scram.sparse_attend(Q, K, V, maps, cfg.window, cfg.scale, causal=causal, out=out,
                                events=None if ev is None else ev[a0:a0 + 2])
        if args.backward:
            scram.sparse_attend_backward(Q, K, V, maps, dO, cfg.window, cfg.scale, causal=causal,
                                         workspace=bwd_ws, events=None if ev is None else ev[a0 + 2:a0 + 8])

    # comparators first (the final map's quality, dense attention for scale): their GPU work also brings
    # the clock to its working level before the timed regions
    progress("comparators")
    comparators = {}
    if kappa == 1 and not causal:
        Jq = torch.empty((S, Hq, Wq), dtype=torch.int32, device=dev)
        scram.patchmatch(Q, K, T, cfg.pm_seed, out=Jq, workspace=ws)  # the map every timed step computes
        comparators["map_quality"] = map_quality(cfg, Q, K, Jq)
        comparators["map_quality_over_seeds"] = quality_over_seeds(cfg, Q, K, T, comparators["map_quality"], ws)
    dense = dense_attention(cfg, Q, K, V) if not (kappa > 1 or causal or args.snis) else None
    progress("timing")
    for _ in range(args.warmup):
        step()
    run = step
    if args.graph:
        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            step()
        stream.wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        run = graph.replay
        for _ in range(args.warmup):
            run()
    # timed region A: the path as a caller runs it (throughput)
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    start.record(stream)
    for _ in range(args.steps):
        run()
    stop.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    # timed region B: the same steps with every dispatch stamping start/stop
    # events (per-kernel durations; the stamps add gaps between kernels, so
    # region B is not used for the throughput)
    events = [new_events() for _ in range(args.steps)]
    torch.cuda.synchronize()
    for k in range(args.steps):
        step(events[k])
    torch.cuda.synchronize()

    def dur(ev, k):
        return ev[2 * k].elapsed_time(ev[2 * k + 1])

    ms_step = start.elapsed_time(stop) / args.steps
    # a fresh run has no init launch: its first sweep recomputes the random
    # initial field, and the init's event pair brackets no work

    iter_by_run = [sum(dur(ev, c * (T + 1) + t) for ev in events for t in range(1, T + 1)) / (args.steps * T)
                   for c in range(kappa)]
    iter_ms = sum(iter_by_run) / kappa
    att_ms = sum(dur(ev, kappa * (T + 1)) for ev in events) / args.steps
    # per-step durations for the median and minimum over the timed steps (a sweep's: the mean of its run's T)
    per_step = {"pm_iter": [sum(dur(ev, c * (T + 1) + t) for c in range(kappa) for t in range(1, T + 1)) / (kappa * T)
                            for ev in events],
                "attend": [dur(ev, kappa * (T + 1)) for ev in events]}
    bwd = {}
    if args.backward:
        for i, name in enumerate(("backward_scan_fill", "backward_query", "backward_key_side")):
            bwd[name] = sum(dur(ev, kappa * (T + 1) + 1 + i) for ev in events) / args.steps
            per_step[name] = [dur(ev, kappa * (T + 1) + 1 + i) for ev in events]

    nq = cfg.nq
    # the dominant kernel: the sweep, averaged over the runs (run c reads c previous maps)
    pm_launch_bytes = nq * sum(pm_bytes_per_query_sweep(cfg, c) for c in range(kappa)) / kappa
    att_bytes = nq * (snis_bytes_per_query(cfg, args.snis, kappa) if args.snis else attend_bytes_per_query(cfg, kappa))
    default_path = kappa == 1 and not causal and not args.snis
    roof = roofline_entry(cfg, "pm_iter", iter_ms, pm_launch_bytes, default_path)
    att_roof = roofline_entry(cfg, "attend", att_ms, att_bytes, default_path)

    res = {
        "metric": METRIC,
        "value": nq / (ms_step * 1e-3),
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "accumulate": "f32",
        "data": "synthetic",
        "config": {
            "workload": cfg.name,
            "grid": f"{Hq}x{Wq}" + ("" if (Hq, Wq) == (cfg.Hk, cfg.Wk) else f"->{cfg.Hk}x{cfg.Wk}"),
            "slices": S,
            "batch": cfg.batch,
            "heads": cfg.heads,
            "d": cfg.d,
            "storage": cfg.dtype,
            "iters": T,
            "window": cfg.window,
            "kappa": kappa,
            "separation": sep,
            "causal": causal,
            "estimator": f"snis T={args.snis} alpha={args.alpha} m={args.radius}" if args.snis else "window",
            "backward": args.backward,
            "launch": "hip graph replay" if args.graph else "eager",
            "queries_per_step": nq,
        },
        "roofline": roof,
        "attend_roofline": att_roof,
        "kernels_ms": {"pm_iter": iter_ms, "attend": att_ms, **bwd},
        "pm_init": "fused into the first sweep",
        "pm_iter_ms_by_run": iter_by_run,
        "kernels_ms_source": "dispatch-stamped HIP events, timed region B",
        "kernels_ms_stats": {k: {"median": statistics.median(v), "min": min(v), "reps": len(v)}
                             for k, v in per_step.items()},
        "candidate_evals_per_s_nominal": kappa * nq * T * cfg.candidates / (ms_step * 1e-3),
        "step_requested_GBps": (T * kappa * pm_launch_bytes + att_bytes) / (ms_step * 1e-3) / 1e9,
        "hbm_copy_GBps": copy_bandwidth(dev),
        "wall_ms_per_step": wall * 1e3 / args.steps,
        "device": torch.cuda.get_device_name(dev),
    }
    progress("timed regions done")
    if kappa == 1 and not causal:
        if not torch.equal(Jq, J[0]):  # a run is deterministic: the timed steps' map is the one scored
            raise RuntimeError("the timed steps' final map differs from the comparator's run")
        res.update(comparators)
    if dense is not None:
        dense["step_speedup"] = dense["ms"] / ms_step
        res["dense_exact_attention"] = dense
    if not args.no_cpu_baseline and cfg.Hq * cfg.Wq > (1 << 18):
        # one slice pass of the oracle would take minutes on one thread
        res["cpu_baseline"] = None
        res["cpu_baseline_skipped"] = f"{cfg.Hq}x{cfg.Wq} slices: one oracle pass exceeds the bounded sample"
    elif not args.no_cpu_baseline:
        progress("oracle on the host cores")
        snis_opt = (args.snis, args.alpha, args.radius) if args.snis else None
        base = cpu_baseline(cfg, data["np"], args.cpu_seconds, kappa, sep, causal, snis_opt)
        one = cpu_baseline(cfg, data["np"], args.cpu_seconds_1t, kappa, sep, causal, snis_opt, threads=1)
        # valid candidates per query-sweep as the oracle counts them on its sample (duplicates included)
        per_sweep = base.pop("candidates_per_query_sweep")
        one.pop("candidates_per_query_sweep")
        res["candidate_evals_per_s"] = kappa * nq * T * per_sweep / (ms_step * 1e-3)
        res["candidates_per_query_sweep"] = per_sweep
        base["cpu_model"] = cpu_model()
        base["single_thread"] = one
        res["cpu_baseline"] = base
    print(json.dumps(res), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
