"""Benchmark of the fused multi-table embedding lookup on one MI355X.

A step is one pass of the whole hot path over one batch: dpi_plan (bag scan,
wave partition) then dpi_lookup (fused gather-pool into the [B, sum dim]
block), on resident inputs, rotating over R independently drawn batches.
Prints one JSON line.

  python bench.py [--config 4] [--steps K] [--warmup W] [--gpus 1]

Roofline: the lookup kernel is bound by HBM bandwidth.  Its algorithmic bytes
per batch are the distinct table rows the batch touches times their row
bytes, plus 4 bytes per id, 4 bytes per offset and the output block; the
achieved rate divides them by the lookup kernel's mean duration measured with
HIP events on the stream it runs on.  HBM traffic measured by rocprofv3
counters (FETCH_SIZE, WRITE_SIZE) is read from profiles/ when it was taken on
the current kernel source, else reported as null.
"""
from __future__ import annotations

import argparse
import gc
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
WORKLOAD_TEXT = {
    1: "tiny one-hot: 8 tables x 1000 rows, D=16 fp32, B=256, uniform ids, sum",
    2: "CTR one-hot: 26 tables, rows logU[10,1e6], D=16 fp32, B=4096, Zipf(1.05) ids, sum",
    3: "multi-hot: 26 tables, rows logU[1e3,5e6], D=64 fp16 -> fp16, B=16384, bags Poisson(10) clip [1,64], "
       "Zipf(1.05) ids, sum",
    4: "large: 100 tables, rows logU[1e5,1e7] (59.3 GB fp16), D=128 fp16 -> fp16, B=65536, bags "
       "floor(LogNormal(ln 20, 0.8)) clip [0,256], Zipf(1.1) ids, even fields sum / odd fields mean",
    5: "heterogeneous: 39 fields, D in {8,16,32,64} fp32, 13 one-hot + 26 multi-hot, rows logU[10,1e7], "
       "Zipf(1.2) ids, sum",
    6: "allocation comparison: 26 one-hot fields x 500000 rows, D=60 fp32, B=65536, Zipf(1.05) ids, sum",
}


def kernel_source_hash() -> str:
    """Hash of the lookup and plan kernel sources, comments and whitespace
    removed (a comment edit does not make a profile stale)."""
    h = hashlib.sha256()
    for name in ("lookup.hip", "small.hip", "gather.h", "plan.hip", "dpi_internal.h"):
        with open(os.path.join(ROOT, "paper_2606_21101_amd", "csrc", name)) as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        text = re.sub(r"//[^\n]*", "", text)
        h.update("".join(text.split()).encode())
    return h.hexdigest()[:16]


def read_profile(config_key: int) -> dict:
    """Counter-measured figures of the lookup kernel from profiles/, if they
    were taken from the current kernel sources: HBM bytes per launch and the
    L2 hit rate (None where absent or stale)."""
    path = os.path.join(ROOT, "profiles", f"lookup_traffic_config{config_key}.txt")
    res = {"traffic": None, "l2_hit_rate": None}
    if not os.path.exists(path):
        return res
    vals = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                vals[k.strip()] = v.strip()
    if vals.get("kernel_source_hash") != kernel_source_hash():
        return res
    for key, name in (("traffic", "hbm_bytes_per_launch"), ("l2_hit_rate", "l2_hit_rate")):
        try:
            res[key] = float(vals[name])
        except (KeyError, ValueError):
            pass
    return res


def _counter_per_dispatch(csv_path: str, counter: str, kernel_regex: str) -> float:
    """Mean over dispatches of a rocprofv3 counter (summed over its instances)."""
    import csv
    import re
    per = {}
    with open(csv_path) as f:
        for r in csv.DictReader(f):
            if r["Counter_Name"] == counter and re.search(kernel_regex, r["Kernel_Name"]):
                per[r["Dispatch_Id"]] = per.get(r["Dispatch_Id"], 0.0) + float(r["Counter_Value"])
    if not per:
        raise SystemExit(f"no {counter} rows for /{kernel_regex}/ in {csv_path}")
    return sum(per.values()) / len(per)


def write_traffic_profile(config_key: int, fetch_csv: str, write_csv: str, copy_fetch_csv: str,
                          copy_write_csv: str, copy_gib: float, commands: str, out_dir: str,
                          l2_csv: str = None):
    """HBM bytes per lookup launch from FETCH_SIZE / WRITE_SIZE passes, each scaled by
    what the same counter reads for a plain device copy of known size; optionally
    the L2 hit rate from a TCC_HIT_sum / TCC_MISS_sum pass."""
    fetch = _counter_per_dispatch(fetch_csv, "FETCH_SIZE", "lookup_")
    write = _counter_per_dispatch(write_csv, "WRITE_SIZE", "lookup_")
    copy_bytes = copy_gib * (1 << 30)
    cf = _counter_per_dispatch(copy_fetch_csv, "FETCH_SIZE", "copy|Copy")
    cw = _counter_per_dispatch(copy_write_csv, "WRITE_SIZE", "copy|Copy")
    f_scale = copy_bytes / (cf * 1024.0)
    w_scale = copy_bytes / (cw * 1024.0)
    hbm = fetch * 1024.0 * f_scale + write * 1024.0 * w_scale
    path = os.path.join(out_dir, f"lookup_traffic_config{config_key}.txt")
    with open(path, "w") as f:
        f.write(f"# HBM traffic of the fused lookup kernel, workload config {config_key}\n")
        f.write(f"# {WORKLOAD_TEXT[config_key]}\n")
        f.write("# commands (run from /tmp, repository at $R, profiler output under $OUT):\n")
        for line in commands.strip().splitlines():
            f.write(f"#   {_portable(line)}\n")
        f.write("# FETCH_SIZE / WRITE_SIZE are KiB per dispatch; each is scaled by the ratio of the\n")
        f.write("# known bytes of a plain device copy to what the same counter reads for it.\n")
        f.write(f"kernel_source_hash: {kernel_source_hash()}\n")
        f.write(f"fetch_kib_per_dispatch: {fetch:.1f}\n")
        f.write(f"write_kib_per_dispatch: {write:.1f}\n")
        f.write(f"copy_probe_bytes: {copy_bytes:.0f}\n")
        f.write(f"copy_fetch_kib_per_dispatch: {cf:.1f}\n")
        f.write(f"copy_write_kib_per_dispatch: {cw:.1f}\n")
        f.write(f"fetch_scale: {f_scale:.4f}\n")
        f.write(f"write_scale: {w_scale:.4f}\n")
        f.write(f"hbm_read_bytes_per_launch: {fetch * 1024.0 * f_scale:.0f}\n")
        f.write(f"hbm_write_bytes_per_launch: {write * 1024.0 * w_scale:.0f}\n")
        f.write(f"hbm_bytes_per_launch: {hbm:.0f}\n")
        if l2_csv:
            hit = _counter_per_dispatch(l2_csv, "TCC_HIT_sum", "lookup_")
            miss = _counter_per_dispatch(l2_csv, "TCC_MISS_sum", "lookup_")
            f.write(f"tcc_hit_per_dispatch: {hit:.0f}\n")
            f.write(f"tcc_miss_per_dispatch: {miss:.0f}\n")
            f.write(f"l2_hit_rate: {hit / (hit + miss):.4f}\n")
    print(path)


def _portable(command: str) -> str:
    """A recorded command with the profiler's output directory written as $OUT
    and this checkout's absolute path as $R."""
    root = os.path.dirname(os.path.abspath(__file__))
    out = re.sub(re.escape(root) + r"/[A-Za-z0-9_]+/prof[0-9]+", "$OUT", command.strip())
    return out.replace(root, "$R")


def summarize_kernel_stats(stats_csv: str, out_path: str, commands: str):
    """Condense a rocprofv3 --stats kernel_stats.csv to the library's kernels."""
    import csv
    rows = list(csv.DictReader(open(stats_csv)))
    keep = [r for r in rows if any(k in r["Name"] for k in ("lookup_", "plan_"))]
    with open(out_path, "w") as f:
        f.write("# rocprofv3 kernel statistics of the library's kernels (durations in ns)\n")
        f.write("# commands (run from /tmp, repository at $R, profiler output under $OUT):\n")
        for line in commands.strip().splitlines():
            f.write(f"#   {_portable(line)}\n")
        f.write(f"# kernel_source_hash: {kernel_source_hash()}\n")
        cols = [c for c in ("Calls", "TotalDurationNs", "AverageNs", "MinNs", "MaxNs", "Percentage") if c in rows[0]]
        f.write("name | " + " | ".join(cols) + "\n")
        for r in keep:
            f.write(r["Name"][:90] + " | " + " | ".join(r[c] for c in cols) + "\n")
    print(out_path)


def cpu_baseline(cfg, samples: int, threads: int = 0):
    """Time the CPU oracle on samples [0, samples) of rotation 0, all fields
    (on `threads` threads; 0: every host core available)."""
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import oracle
    from cases import sub_problem
    cores = len(os.sched_getaffinity(0))
    if os.environ.get("OMP_NUM_THREADS", "").isdigit():
        cores = min(cores, int(os.environ["OMP_NUM_THREADS"]))
    if threads > 0:
        cores = min(cores, threads)
    samples = min(samples, cfg.batch)
    p = sub_problem(cfg, ranges=[(0, samples)])
    nnz = int(len(p["ids"]))
    t0 = time.perf_counter()
    oracle.lookup(p["dims"], p["tables"], p["ids"], p["offsets"], p["pooling"], p["B"], with_mag=False,
                  nthreads=cores)
    dt = time.perf_counter() - t0
    return {"value": nnz / dt, "unit": "rows/s", "cores": cores, "kind": "oracle",
            "sample": f"samples [0, {samples}) of batch rotation 0, all {cfg.num_tables} fields: {nnz} pooled ids "
                      f"in {dt:.3f} s ({dt * cores:.1f} thread-seconds), fp64 sequential per bag"}


def stage_sweep(args, dev) -> dict:
    """Host-to-device staging of one-hot features, per batch size of the
    heterogeneous workload, over its one-hot fields.  'per_field': one pinned
    float column per field, each copied and converted to int64 on its own
    (the unconsolidated pipeline of the paper's breakdown), then narrowed to
    int32 and concatenated field-major for the lookup; 'consolidated': one
    pinned sample-major float matrix, dpi_stage_onehot (one copy, one
    kernel).  Host wall time to ids ready on the device (synchronized), p50."""
    import numpy as np
    import torch

    from paper_2606_21101_amd import dpi
    from synth import configs, generate as G

    from paper_2606_21101_amd.lookup import FusedLookup

    base = configs.get(5)
    T = base.onehot_fields
    reps, warm = 200, 20
    rows = []
    tables = [G.make_table(base, t, dev) for t in range(base.num_tables)]
    for B in base.batches:
        cfg = base.with_batch(B)
        batch = G.make_batch(cfg, device="cpu")
        ids_np = batch.ids[: T * B].numpy().reshape(T, B)          # field-major one-hot ids
        x = torch.empty((B, T), dtype=torch.float32, pin_memory=True)
        x.copy_(torch.from_numpy(ids_np.T.astype(np.float32)))
        cols = [torch.empty(B, dtype=torch.float32, pin_memory=True) for _ in range(T)]
        for t in range(T):
            cols[t].copy_(torch.from_numpy(ids_np[t].astype(np.float32)))
        staging = torch.empty(B * T * 4, dtype=torch.uint8, device=dev)
        ids = torch.empty(T * B, dtype=torch.int32, device=dev)

        def per_field():
            longs = [c.to(dev, non_blocking=True).long() for c in cols]
            out = torch.cat([v.int() for v in longs])
            torch.cuda.synchronize()
            return out

        def consolidated():
            dpi.dpi_stage_onehot(x, dpi.DPI_X_F32, B, T, T, staging, ids)
            torch.cuda.synchronize()
            return ids

        if not torch.equal(per_field(), consolidated()):
            raise SystemExit("staged ids differ")
        res = {"batch": B, "fields": T}
        for name, fn in (("per_field", per_field), ("consolidated", consolidated)):
            for _ in range(warm):
                fn()
            ts = []
            for _ in range(reps):
                t0 = time.perf_counter()
                fn()
                ts.append(time.perf_counter() - t0)
            res[name + "_us"] = float(np.median(ts) * 1e6)
        res["speedup"] = res["per_field_us"] / res["consolidated_us"]

        # all 39 fields as CSR (int64 offsets and ids, as a loader holds them):
        # per field two copies and two conversions, against one packed copy and
        # one kernel (dpi_stage_csr)
        T_all = cfg.num_tables
        offs64 = batch.offsets_host.astype(np.int64)
        ids64 = batch.ids.numpy().astype(np.int64)
        id_start = np.concatenate([[0], np.cumsum(offs64[:, -1])])
        f_ids = [torch.empty(int(offs64[t, -1]), dtype=torch.int64, pin_memory=True) for t in range(T_all)]
        f_off = [torch.empty(B + 1, dtype=torch.int64, pin_memory=True) for t in range(T_all)]
        for t in range(T_all):
            f_ids[t].copy_(torch.from_numpy(ids64[id_start[t]:id_start[t + 1]]))
            f_off[t].copy_(torch.from_numpy(offs64[t]))
        packed = torch.empty(T_all * (B + 1) + len(ids64), dtype=torch.int64, pin_memory=True)
        packed.copy_(torch.from_numpy(np.concatenate([offs64.reshape(-1), ids64])))
        st2 = torch.empty(packed.numel() * 8, dtype=torch.uint8, device=dev)
        o32 = torch.empty((T_all, B + 1), dtype=torch.int32, device=dev)
        i32 = torch.empty(max(1, len(ids64)), dtype=torch.int32, device=dev)

        def csr_per_field():
            oi = [f_off[t].to(dev, non_blocking=True).int() for t in range(T_all)]
            ii = [f_ids[t].to(dev, non_blocking=True).int() for t in range(T_all)]
            o, i = torch.stack(oi), torch.cat(ii)
            torch.cuda.synchronize()
            return o, i

        def csr_consolidated():
            dpi.dpi_stage_csr(packed, dpi.DPI_X_I64, T_all, B, len(ids64), st2, o32, i32)
            torch.cuda.synchronize()
            return o32, i32[: len(ids64)]

        a, b = csr_per_field(), csr_consolidated()
        if not (torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])):
            raise SystemExit("staged CSR differs")
        for name, fn in (("csr_per_field", csr_per_field), ("csr_consolidated", csr_consolidated)):
            for _ in range(warm):
                fn()
            ts = []
            for _ in range(reps):
                t0 = time.perf_counter()
                fn()
                ts.append(time.perf_counter() - t0)
            res[name + "_us"] = float(np.median(ts) * 1e6)
        res["csr_fields"] = T_all
        res["csr_speedup"] = res["csr_per_field_us"] / res["csr_consolidated_us"]

        # the whole step from the host CSR to the pooled block: dpi_stage_csr,
        # then dpi_plan and dpi_lookup; against dpi_plan and dpi_lookup_csr
        # (one copy and one kernel when the lookup is the batch's only launch)
        fl = FusedLookup(tables, None, torch.float32, num_rows=G.table_sizes(cfg))
        out = torch.empty((B, fl.total_dim), dtype=torch.float32, device=dev)
        n_ids = len(ids64)

        def step_staged():
            dpi.dpi_stage_csr(packed, dpi.DPI_X_I64, T_all, B, n_ids, st2, o32, i32)
            p = fl.plan(o32, B, n_ids)
            fl.lookup(p, i32, o32, out)
            torch.cuda.synchronize()
            return out.clone()

        def step_fused():
            p = fl.plan(o32, B, n_ids)
            dpi.dpi_lookup_csr(p, packed, dpi.DPI_X_I64, st2, fl._table_ptrs, None, o32, i32, out)
            torch.cuda.synchronize()
            return out.clone()

        fused_ok = True
        try:
            a_out = step_staged()
            b_out = step_fused()
        except dpi.DpiError:
            fused_ok = False          # a batch planned by its own launch: no fused path
        if fused_ok:
            if not torch.equal(a_out.view(torch.int32), b_out.view(torch.int32)):
                raise SystemExit("dpi_lookup_csr output differs from staging then lookup")
            for name, fn in (("step_staged", step_staged), ("step_fused", step_fused)):
                for _ in range(warm):
                    fn()
                ts = []
                for _ in range(reps):
                    t0 = time.perf_counter()
                    fn()
                    ts.append(time.perf_counter() - t0)
                res[name + "_us"] = float(np.median(ts) * 1e6)
            res["step_fused_speedup"] = res["step_staged_us"] / res["step_fused_us"]
        rows.append(res)
    return {"metric": "input staging latency", "unit": "us", "reps": reps, "higher_is_better": False,
            "data": "synthetic (heterogeneous workload: its one-hot fields as a float matrix, all fields as "
                    "int64 CSR)", "results": rows}


def sched_sweep(args, dev) -> dict:
    """The interaction modules after the lookup (a cross network of 3 layers and
    an MLP of 1024-512-256 over the CTR one-hot workload's pooled block,
    B = 4096 and B = 16384, d = 26 * 16) under the three launch orders.
    Reported per order: p50 of the whole forward (HIP events on the stream the
    modules join), and p50 of the gap between the starts of the two modules'
    first operators (device wall clock), the measurement of §V for
    Algorithm 2."""
    import numpy as np
    import torch

    from paper_2606_21101_amd import dpi

    khz = dpi.dpi_wall_clock_khz()
    rng = np.random.default_rng(2606)
    d, n_cross, mlp = 26 * 16, 3, [1024, 512, 256]
    cw = [torch.from_numpy((rng.standard_normal((d, d)) / np.sqrt(d)).astype(np.float32)).to(dev) for _ in range(n_cross)]
    cb = [torch.zeros(d, device=dev) for _ in range(n_cross)]
    mw, mb, prev = [], [], d
    for h in mlp:
        mw.append(torch.from_numpy((rng.standard_normal((h, prev)) / np.sqrt(prev)).astype(np.float32)).to(dev))
        mb.append(torch.zeros(h, device=dev))
        prev = h
    names = {dpi.DPI_SCHED_BREADTH_FIRST: "breadth_first", dpi.DPI_SCHED_DEPTH_FIRST: "depth_first",
             dpi.DPI_SCHED_ONE_STREAM: "one_stream"}
    se, si = torch.cuda.Stream(), torch.cuda.Stream()
    after = torch.cuda.current_stream()
    results = []
    for B in (4096, 16384):
        head = dpi.DcnHead(B, d, cw, cb, mw, mb)
        x0 = torch.from_numpy(rng.standard_normal((B, d)).astype(np.float32)).to(dev)
        oc = torch.empty((B, d), device=dev)
        om = torch.empty((B, mlp[-1]), device=dev)
        marks = torch.zeros((args.steps + args.warmup, 2), dtype=torch.int64, device=dev)
        row = {"batch": B}
        for mode, name in names.items():
            evs = timing_events(args.steps + args.warmup, 2, after)
            for i in range(args.steps + args.warmup):
                evs[i][0].record(after)
                head.forward(x0, oc, om, mode, se, si, after, marks[i])
                evs[i][1].record(after)
                torch.cuda.synchronize()
            ms = [e[0].elapsed_time(e[1]) for e in evs[args.warmup:]]
            m = marks[args.warmup:].cpu().numpy().astype(np.float64)
            gap_us = np.abs(m[:, 1] - m[:, 0]) / khz * 1e3
            row[name] = {"p50_forward_ms": float(np.median(ms)), "p50_start_gap_us": float(np.median(gap_us))}
        results.append(row)
        del head
    return {"metric": "interaction modules: forward time and start gap of the two modules", "unit": "ms / us",
            "wall_clock_khz": khz, "cross_layers": n_cross, "mlp": mlp, "dim": d, "results": results}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--warm-seconds", type=float, default=0.3,
                    help="untimed steps for this long before the warm-up steps (clock ramp)")
    ap.add_argument("--config", type=int, default=4)
    ap.add_argument("--batch", type=int, default=None, help="override the batch size (heterogeneous sweep)")
    ap.add_argument("--rotations", type=int, default=4)
    ap.add_argument("--out-dtype", choices=["f16", "f32"], default=None)
    ap.add_argument("--dim", type=int, default=None, help="override the embedding dim (allocation comparison)")
    ap.add_argument("--mapping", choices=["literal", "scattered"], default="literal")
    ap.add_argument("--flags", type=int, default=0)
    ap.add_argument("--num-waves", type=int, default=0)
    ap.add_argument("--cpu-samples", type=int, default=6144)
    ap.add_argument("--cpu-threads", type=int, default=0, help="oracle threads for cpu_baseline (0: all cores)")
    ap.add_argument("--cpu-samples-1t", type=int, default=1024,
                    help="samples of the single-thread oracle leg of cpu_baseline")
    ap.add_argument("--second-config", type=int, default=None,
                    help="also measure this workload in the same run (default: the multi-hot workload when the "
                         "large one is the headline); 0: none")
    ap.add_argument("--graph-steps", type=int, default=16,
                    help="steps captured in one HIP graph for the device-side series; 0: none")
    ap.add_argument("--graph-replays", type=int, default=50)
    ap.add_argument("--cold-steps", type=int, default=10,
                    help="extra steps, each after overwriting a buffer larger than the caches (0: none)")
    ap.add_argument("--flush-mib", type=int, default=1024)
    ap.add_argument("--stage-sweep", action="store_true",
                    help="only measure one-hot input staging latency (per-field copies and conversions "
                         "against dpi_stage_onehot) over the heterogeneous workload's batch sizes")
    ap.add_argument("--inflight", type=int, default=1,
                    help="also time a series with this many batches in flight (each with its own stream, "
                         "workspace and output, so one batch's plan overlaps another's lookup, as in a "
                         "serving loop); 1: no such series.  value stays the one-batch-at-a-time series")
    ap.add_argument("--sched-sweep", action="store_true",
                    help="only measure the interaction modules under the three launch orders (Algorithm 2)")
    ap.add_argument("--fm", action="store_true",
                    help="also time the second-order FM term over the lookup output (fields of one dim)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe-gib", type=float, default=0.0,
                    help="only run a plain device copy of this size (counter calibration)")
    ap.add_argument("--write-traffic-profile", nargs=4, metavar=("FETCH_CSV", "WRITE_CSV", "COPY_FETCH_CSV",
                                                                  "COPY_WRITE_CSV"),
                    help="write profiles/lookup_traffic_config<N>.txt from rocprofv3 counter CSVs")
    ap.add_argument("--l2-csv", default=None, help="rocprofv3 TCC_HIT_sum/TCC_MISS_sum CSV for the traffic profile")
    ap.add_argument("--summarize-kernel-stats", nargs=2, metavar=("STATS_CSV", "OUT"))
    ap.add_argument("--commands", default="", help="command lines recorded in a written profile")
    ap.add_argument("--profile-dir", default=os.path.join(ROOT, "profiles"))
    args = ap.parse_args()

    if args.write_traffic_profile:
        write_traffic_profile(args.config, *args.write_traffic_profile, copy_gib=args.copy_probe_gib or 1.0,
                              commands=args.commands, out_dir=args.profile_dir, l2_csv=args.l2_csv)
        return
    if args.summarize_kernel_stats:
        summarize_kernel_stats(*args.summarize_kernel_stats, commands=args.commands)
        return

    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}); the lookup is a single-GPU "
              "path here. Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2606_21101_amd import dpi
    from paper_2606_21101_amd.lookup import FusedLookup
    from synth import configs, generate as G

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    if args.stage_sweep:
        print(json.dumps(stage_sweep(args, dev)), flush=True)
        return
    if args.sched_sweep:
        print(json.dumps(sched_sweep(args, dev)), flush=True)
        return

    if args.copy_probe_gib > 0:
        n = int(args.copy_probe_gib * (1 << 30)) // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes_read": n * 4, "copy_probe_bytes_written": n * 4, "launches": 3}))
        return

    if args.second_config is None:
        args.second_config = 3 if args.config == 4 else 0
    cfg = configs.get(args.config, batch=args.batch, out_dtype=args.out_dtype, dim=args.dim)
    m = measure(cfg, args, dev, steps=args.steps, warmup=args.warmup, fm=args.fm, inflight=args.inflight)
    roof = roofline(m["alg_mean"], m["look_mean_ms"], read_profile(cfg.key)["traffic"])
    roof_cold = None if m["cold"] is None else roofline(m["alg_mean"], m["cold"]["mean_lookup_ms"], None)
    prof = read_profile(cfg.key)
    hdr = m["header"]

    line = {
        "metric": "pooled embedding rows/s",
        "value": m["value"],
        "unit": "rows/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup, "warm_seconds": args.warm_seconds,
        "ms_per_step": m["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded generator; stands in for Criteo-scale CTR fields)",
        "config": {
            "workload": f"config {cfg.key} " + WORKLOAD_TEXT[cfg.key]
                        + (f" [B={cfg.batch}]" if args.batch else "") + (f" [D={args.dim}]" if args.dim else ""),
            "global_batch": cfg.batch,
            "fields": cfg.num_tables,
            "table_dtype": cfg.dtype,
            "out_dtype": cfg.out_dtype,
            "id_mapping": args.mapping,
            "plan_flags": args.flags,
            "allocation": "input-first" if args.flags & 8 else "output-first",
            "rotating_batches": m["rotations"],
            "waves": int(hdr[3]),
            "items": int(hdr[9]),
            "split_bags": int(hdr[12]),
            "parallelism": "single GPU",
        },
        "p50_lookup_ms": m["p50_lookup_ms"],
        "p90_lookup_ms": m["p90_lookup_ms"],
        "p50_plan_ms": m["p50_plan_ms"],
        "p50_step_ms": m["p50_step_ms"],
        "wall_ms_per_step": m["wall_ms_per_step"],
        "max_gap_ms": m["max_gap_ms"],
        "pooled_ids_per_batch": m["nnz_mean"],
        "algorithmic_bytes_per_batch": m["alg_mean"],
        "gathered_bytes_per_batch": m["gathered_mean"],
        "hbm_gbs": roof["achieved"],
        "hbm_frac": roof["frac"],
        "gathered_gbs": m["gathered_mean"] / (m["look_mean_ms"] / 1e3) / 1e9,
        "roofline": roof,
        "roofline_cold": roof_cold,
        "l2_hit_rate": prof["l2_hit_rate"],
        "cold": m["cold"],
        "fm_second_order": m["fm"],
        "inflight": m["inflight"],
        "device_series": m["device_series"],
        "setup_s": m["setup_s"],
        "kernel_source_hash": kernel_source_hash(),
    }
    if args.second_config and not args.batch and not args.dim and not args.flags and not args.num_waves:
        # the other workload of the bandwidth target, measured in the same run
        cfg2 = configs.get(args.second_config, out_dtype=args.out_dtype)
        del m
        torch.cuda.empty_cache()
        m2 = measure(cfg2, args, dev, steps=max(args.steps, 50), warmup=args.warmup)
        prof2 = read_profile(cfg2.key)
        line[f"config{cfg2.key}"] = {
            "workload": f"config {cfg2.key} " + WORKLOAD_TEXT[cfg2.key],
            "steps": max(args.steps, 50),
            "value": m2["value"], "unit": "rows/s", "ms_per_step": m2["ms_per_step"],
            "p50_lookup_ms": m2["p50_lookup_ms"], "p90_lookup_ms": m2["p90_lookup_ms"],
            "p50_plan_ms": m2["p50_plan_ms"], "p50_step_ms": m2["p50_step_ms"],
            "device_series": m2["device_series"],
            "cold": m2["cold"],
            "pooled_ids_per_batch": m2["nnz_mean"],
            "algorithmic_bytes_per_batch": m2["alg_mean"],
            "waves": int(m2["header"][3]), "split_bags": int(m2["header"][12]),
            "roofline": roofline(m2["alg_mean"], m2["look_mean_ms"], prof2["traffic"]),
            "roofline_cold": None if m2["cold"] is None else
            roofline(m2["alg_mean"], m2["cold"]["mean_lookup_ms"], None),
            "l2_hit_rate": prof2["l2_hit_rate"],
        }
    if not args.no_cpu_baseline:
        cb = cpu_baseline(cfg, args.cpu_samples, args.cpu_threads)
        one = cpu_baseline(cfg, args.cpu_samples_1t, 1)
        cb["single_thread"] = {"value": one["value"], "unit": one["unit"], "cores": 1, "sample": one["sample"]}
        line["cpu_baseline"] = cb
    print(json.dumps(line), flush=True)


def roofline(alg_bytes: float, mean_ms: float, traffic) -> dict:
    """HBM roofline of the lookup kernel: algorithmic bytes per launch over its
    mean duration, against the 8 TB/s peak."""
    achieved = alg_bytes / (mean_ms / 1e3) / 1e9
    return {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS, "traffic": traffic, "mean_lookup_ms": mean_ms}


def timing_events(n: int, k: int, stream):
    """n lists of k timing events, each recorded once already: torch creates an
    event's device object on its first record, which costs tens of
    microseconds of host time, far more than a small batch's step."""
    import torch
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(k)] for _ in range(n)]
    for row in evs:
        for e in row:
            e.record(stream)
    torch.cuda.synchronize()
    return evs


def measure(cfg, args, dev, steps: int, warmup: int, fm: bool = False, inflight: int = 1) -> dict:
    """Tables and R rotating batches of one workload resident on the device, then
    untimed clock-ramp steps, warm-up steps, the timed warm series (HIP events on
    the launch stream around each dpi_plan and dpi_lookup), optional series (FM
    epilogue, batches in flight) and the cold series."""
    import numpy as np
    import torch

    from paper_2606_21101_amd import dpi
    from paper_2606_21101_amd.lookup import FusedLookup
    from synth import configs, generate as G

    t_setup = time.perf_counter()
    tables = [G.make_table(cfg, t, dev) for t in range(cfg.num_tables)]
    batches = G.make_batches(cfg, range(args.rotations), dev, mapping=args.mapping)
    out_dt = torch.float16 if cfg.out_dtype == configs.F16 else torch.float32
    pool = [1 if p == configs.MEAN else 0 for p in G.table_pooling(cfg)]
    fl = FusedLookup(tables, pool, out_dt, num_rows=G.table_sizes(cfg), flags=args.flags)
    osize = 2 if out_dt == torch.float16 else 4
    esize = 2 if cfg.dtype == configs.F16 else 4
    total_d = fl.total_dim

    # algorithmic bytes of each batch: distinct rows + ids + offsets + output
    alg_bytes, nnz_list = [], []
    for bt in batches:
        base = bt.id_base
        uniq_bytes = 0
        for t in range(cfg.num_tables):
            seg = bt.ids[int(base[t]):int(base[t + 1])]
            if seg.numel():
                uniq_bytes += int(torch.unique(seg).numel()) * cfg.dim(t) * esize
        offs_bytes = 4 * cfg.num_tables * (cfg.batch + 1) if bt.offsets is not None else 0
        alg_bytes.append(uniq_bytes + 4 * bt.total_ids + offs_bytes + cfg.batch * total_d * osize)
        nnz_list.append(bt.total_ids)
    gathered = [4 * n + (4 * cfg.num_tables * (cfg.batch + 1)) + cfg.batch * total_d * osize
                + int(sum(int(bt.nnz[t]) * cfg.dim(t) * esize for t in range(cfg.num_tables)))
                for n, bt in zip(nnz_list, batches)]

    stream = torch.cuda.current_stream()
    out = torch.empty((cfg.batch, total_d), dtype=out_dt, device=dev)
    max_total = max(nnz_list)
    opts = fl.opts(args.num_waves)
    ws_bytes = dpi.dpi_plan_workspace_bytes(cfg.num_tables, cfg.batch, max_total, max(fl.dims), opts)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    setup_s = time.perf_counter() - t_setup

    table_ptrs = dpi.table_array(tables)
    pool_arr = None if pool is None else dpi.pooling_array(pool)

    def step(i, ev=None, s=None):
        s = stream if s is None else s
        bt = batches[i % len(batches)]
        if ev is not None:
            ev[0].record(s)
        plan = dpi.dpi_plan(fl.meta, bt.offsets, cfg.batch, bt.total_ids, opts, ws, ws_bytes, stream=s)
        if ev is not None:
            ev[1].record(s)
        dpi.dpi_lookup(plan, table_ptrs, bt.ids, bt.offsets, pool_arr, out, stream=s)
        if ev is not None:
            ev[2].record(s)
        return plan

    # untimed steps until the clocks have ramped (short steps would otherwise be
    # timed partly at idle clocks), then the W warm-up steps
    t_warm, i = time.perf_counter(), 0
    while time.perf_counter() - t_warm < args.warm_seconds:
        step(i)
        i += 1
        if i % 8 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    plans = []
    evs = timing_events(steps, 3, stream)
    # no garbage collection inside the timed loop (a collection pass stalls the
    # host for milliseconds, and small steps wait on the host)
    gc.collect()
    gc.disable()
    t0 = time.perf_counter()
    for i in range(steps):
        plans.append(step(warmup + i, evs[i]))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gc.enable()
    status = dpi.dpi_plan_sync_status(plans[-1])
    if status != dpi.DPI_OK:
        raise SystemExit(f"device reported {dpi.dpi_status_str(status)}")
    hdr = dpi.dpi_plan_export(plans[-1])["header"]   # before later steps plan into the same workspace
    # device-side series: K consecutive steps captured in one HIP graph and
    # replayed, so the GPU runs them back to back instead of waiting for the
    # host.  For small batches the host's enqueue (Python, ctypes, events)
    # takes longer than a step, so the timed series above measures the host;
    # a replay's time over K is the device's own time per step (launch gaps
    # between the step's kernels included).  The replayed output is checked
    # against the same step run eagerly.
    graph_res = None
    if args.graph_steps > 0:
        K, R = args.graph_steps, args.graph_replays
        gs = torch.cuda.Stream()
        gs.wait_stream(stream)
        g = torch.cuda.CUDAGraph()
        gplans = []
        with torch.cuda.graph(g, stream=gs):
            for i in range(K):
                gplans.append(step(i, s=gs))
        torch.cuda.synchronize()
        rev = timing_events(R, 2, stream)
        for r in range(R):
            rev[r][0].record(stream)
            g.replay()
            rev[r][1].record(stream)
        torch.cuda.synchronize()
        replayed = out.clone()
        step(K - 1)
        torch.cuda.synchronize()
        if not torch.equal(replayed.view(torch.uint8), out.view(torch.uint8)):
            raise SystemExit("graph replay output differs from the eager step")
        per_step = np.array([e[0].elapsed_time(e[1]) for e in rev]) / K
        graph_res = {"steps_per_graph": K, "replays": R, "p50_step_ms": float(np.median(per_step)),
                     "min_step_ms": float(per_step.min()), "mean_step_ms": float(per_step.mean())}
        del g, gplans
    inflight_res = None
    if inflight > 1:
        # steps dealt round-robin to `inflight` streams, each with its own
        # workspace and output; one batch's plan overlaps another's lookup
        n = inflight
        streams = [torch.cuda.Stream() for _ in range(n)]
        wss = [torch.empty(ws_bytes, dtype=torch.uint8, device=dev) for _ in range(n)]
        outs = [torch.empty_like(out) for _ in range(n)]
        keep = []

        def step_on(i, k):
            bt = batches[i % len(batches)]
            p = dpi.dpi_plan(fl.meta, bt.offsets, cfg.batch, bt.total_ids, opts, wss[k], ws_bytes, stream=streams[k])
            dpi.dpi_lookup(p, table_ptrs, bt.ids, bt.offsets, pool_arr, outs[k], stream=streams[k])
            keep.append(p)

        for i in range(warmup):
            step_on(i, i % n)
        torch.cuda.synchronize()
        (e0, e1), = timing_events(1, 2, stream)
        e0.record(stream)
        for st in streams:
            st.wait_stream(stream)
        for i in range(steps):
            step_on(warmup + i, i % n)
        for st in streams:
            stream.wait_stream(st)
        e1.record(stream)
        torch.cuda.synchronize()
        span = e0.elapsed_time(e1)
        for p in keep[-n:]:
            if dpi.dpi_plan_sync_status(p) != dpi.DPI_OK:
                raise SystemExit("device reported an error in the in-flight series")
        inflight_res = {"batches_in_flight": n, "ms_per_step": span / steps,
                        "value": sum(nnz_list[(warmup + i) % len(batches)] for i in range(steps)) / (span / 1e3)}
        del keep
    fm_res = None
    if fm:
        dims = {cfg.dim(t) for t in range(cfg.num_tables)}
        if len(dims) != 1:
            raise SystemExit("--fm needs fields of one dim")
        D = dims.pop()
        y = torch.empty(cfg.batch, dtype=torch.float32, device=dev)
        odt = dpi.DPI_F16 if out_dt == torch.float16 else dpi.DPI_F32
        fev = timing_events(steps + warmup, 2, stream)
        for i in range(steps + warmup):
            fev[i][0].record(stream)
            dpi.dpi_fm_second_order(out, odt, cfg.batch, cfg.num_tables, D, total_d, y, stream=stream)
            fev[i][1].record(stream)
        torch.cuda.synchronize()
        fm_ms = np.array([e[0].elapsed_time(e[1]) for e in fev[warmup:]])
        fm_bytes = cfg.batch * total_d * osize + 4 * cfg.batch
        fm_gbs = fm_bytes / (float(fm_ms.mean()) / 1e3) / 1e9
        fm_res = {"kernel": "fm_kernel", "p50_ms": float(np.median(fm_ms)), "bytes_per_launch": fm_bytes,
                  "roofline": {"bound": "hbm", "achieved": fm_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                               "frac": fm_gbs / HBM_PEAK_GBS}}
    cold = None
    if args.cold_steps > 0:
        # cold series: the L2s and the 256 MB Infinity Cache are overwritten
        # before each step, outside the timed events
        flush = torch.empty(args.flush_mib << 20, dtype=torch.uint8, device=dev)
        cev = timing_events(args.cold_steps, 3, stream)
        for i in range(args.cold_steps):
            flush.fill_(i & 0xFF)
            step(warmup + steps + i, cev[i])
        torch.cuda.synchronize()
        del flush
        c_look = np.array([e[1].elapsed_time(e[2]) for e in cev])
        c_alg = float(np.mean([alg_bytes[(warmup + steps + i) % len(batches)] for i in range(args.cold_steps)]))
        cold = {"steps": args.cold_steps, "flush_bytes": args.flush_mib << 20,
                "p50_lookup_ms": float(np.median(c_look)), "mean_lookup_ms": float(c_look.mean()),
                "p50_plan_ms": float(np.median([e[0].elapsed_time(e[1]) for e in cev])),
                "algorithmic_bytes_per_batch": c_alg}
    plan_ms = np.array([evs[i][0].elapsed_time(evs[i][1]) for i in range(steps)])
    look_ms = np.array([evs[i][1].elapsed_time(evs[i][2]) for i in range(steps)])
    span_ms = evs[0][0].elapsed_time(evs[-1][2])
    rot = [(warmup + i) % len(batches) for i in range(steps)]
    steps_nnz = sum(nnz_list[r] for r in rot)
    steps_alg = np.array([alg_bytes[r] for r in rot], dtype=np.float64)
    steps_gath = np.array([gathered[r] for r in rot], dtype=np.float64)
    res = {
        "value": steps_nnz / (span_ms / 1e3),
        "ms_per_step": span_ms / steps,
        "p50_lookup_ms": float(np.median(look_ms)),
        "p90_lookup_ms": float(np.percentile(look_ms, 90)),
        "look_mean_ms": float(look_ms.mean()),
        "p50_plan_ms": float(np.median(plan_ms)),
        "p50_step_ms": float(np.median(plan_ms + look_ms)),
        "wall_ms_per_step": wall * 1e3 / steps,
        "max_gap_ms": float(max([evs[i][2].elapsed_time(evs[i + 1][0]) for i in range(steps - 1)], default=0.0)),
        "nnz_mean": float(np.mean(nnz_list)),
        "alg_mean": float(steps_alg.mean()),
        "gathered_mean": float(steps_gath.mean()),
        "rotations": len(batches),
        "header": hdr,
        "cold": cold,
        "fm": fm_res,
        "inflight": inflight_res,
        "device_series": graph_res,
        "setup_s": setup_s,
    }
    del plans, tables, batches, out, ws
    return res


if __name__ == "__main__":
    main()
