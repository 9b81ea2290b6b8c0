"""Throughput of memoized mutation testing on one MI355X.

One step = the whole hot path over one batch of inputs: load the model (a1),
apply the mutants (a2: clusters, copy-on-write layers), run the original once
over the batch and fill the prefix cache (a3), run every mutant's suffix over
the batch (a4 delta at the first mutated layer, a5 layers after it) and
reduce to kill bits and the mutation score (a6).  The workload's inputs are
resident in device memory before the timed region; consecutive steps take
consecutive batches of them (resnet18w: batches of 1,000 of its 5,000
inputs, so five steps cover the test set; the other workloads: the whole set
per step).

value = (mutants x inputs per step) / step time: (mutant, input)
evaluations per second of the whole job.  The line also carries the
suffix-only rate (run_mutants alone), the dominant kernel's achieved rate
against its roofline (per-launch HIP events on the library's stream), and the
CPU oracle timed on a bounded sample.

    python bench.py [--steps K] [--warmup W] [--config resnet18w] [--gpus 1]
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

import workloads as W  # noqa: E402

PEAK_TFLOPS = {"f32": 157.3, "bf16": 2500.0}    # MI355X dense MFMA
KERNELS = ["dense_kernel (DENSE layers, MFMA GEMM)",
           "conv_valu_kernel (CONV2D with few output channels, vector ALU)",
           "conv_lds_kernel (CONV2D, LDS-resident images, MFMA)",
           "conv_mfma_kernel (CONV2D, im2col implicit GEMM with scalar gathers, MFMA)",
           "conv_big_kernel (bf16 CONV2D, tiled implicit GEMM, MFMA)",
           "dw_col_kernel (depthwise CONV2D, vector ALU; dw_full_kernel for filters other than 3x3)",
           "embed_kernel (token embedding gather)",
           "lstm_kernel (LSTM recursion, MFMA per step)",
           "conv_halo_kernel (bf16 3x3 CONV2D, A operand from LDS halo tiles, MFMA)"]
KERNEL_NAMES = ["dense_kernel", "conv_valu_kernel", "conv_lds_kernel", "conv_mfma_kernel",
                "conv_big_kernel", "dw_col_kernel", "embed_kernel", "lstm_kernel", "conv_halo_kernel"]
VALU_FAMILIES = (1, 5)                           # fused multiply-add chains on the vector ALU
PEAK_VALU_TFLOPS = 78.6                          # fp32 FMA without packed-fp32 instructions
PEAK_HBM_GBS = 8000.0
PROFILES = os.path.join(ROOT, "profiles")
ORACLE_SAMPLE = {"mlp": (100, 500), "lenet5": (24, 6000), "vgg": (3, 64), "resnet20": (8, 256),
                 "resnet18w": (6, 64), "mobilenetv2": (8, 256), "lstm": (8, 500), "rnn_imdb": (8, 500)}
INPUTS_PER_STEP = {"resnet18w": 1000}             # others: the whole input set per step


def cpu_baseline(wl, n_mut: int, n_in: int):
    """The oracle (vanilla: every mutant from the raw input), as it stands,
    on a bounded sample of the workload, timed on this host's cores."""
    import oracle as O
    try:
        from threadpoolctl import threadpool_info
        threads = max(int(p.get("num_threads", 1)) for p in threadpool_info()) if threadpool_info() else 1
    except Exception:
        threads = os.cpu_count() or 1
    sub = W.Workload(wl.name, wl.model, wl.inputs[:n_in], wl.mutants.subset(n_mut))
    om = O.OracleModel(wl.model)
    t = time.perf_counter()
    O.run_vanilla(om, sub.inputs, sub.mutants, chunk=256)
    dt = time.perf_counter() - t
    return {"value": n_mut * n_in / dt, "unit": "evals/s", "cores": threads, "kind": "oracle",
            "sample": f"first {n_mut} mutants x first {n_in} inputs of {wl.name} "
                      f"(vanilla, float64 accumulation), {dt:.1f} s"}


def library_source_hash() -> str:
    """Hash of the library's sources: HBM counters taken on other sources no
    longer describe the kernels."""
    import hashlib
    h = hashlib.sha256()
    d = os.path.join(ROOT, "paper_2607_18582_amd", "csrc")
    for f in sorted(os.listdir(d)):
        if f.endswith((".hip", ".hpp", ".cpp")):
            h.update(f.encode())
            with open(os.path.join(d, f), "rb") as fh:
                h.update(fh.read())
    with open(os.path.join(ROOT, "include", "mure.h"), "rb") as fh:
        h.update(fh.read())
    return h.hexdigest()[:16]


def traffic_path(kernel: str, config: str) -> str:
    return os.path.join(PROFILES, f"{kernel}_{config}_hbm_traffic.md")


def read_traffic(kernel: str, config: str, n_inputs: int, n_mutants: int):
    """HBM bytes per run_mutants launch of ``kernel`` from its committed
    counter summary, or None when there is none for this workload or the
    library changed since the counters were taken."""
    try:
        with open(traffic_path(kernel, config)) as f:
            for ln in f:
                if ln.startswith('{"traffic_bytes_per_launch"'):
                    d = json.loads(ln)
                    if (d["source_hash"] == library_source_hash() and d["n_inputs"] == n_inputs
                            and d["n_mutants"] == n_mutants):
                        return d
    except OSError:
        pass
    return None


def counters_path(kernel: str, config: str) -> str:
    return os.path.join(PROFILES, f"{kernel}_{config}_mfma_counters.md")


def read_counters(kernel: str, config: str, n_inputs: int, n_mutants: int):
    """MFMA busy share and clock of ``kernel`` from its committed counter
    summary, or None (no summary for this workload, or the library changed
    since the counters were taken)."""
    try:
        with open(counters_path(kernel, config)) as f:
            for ln in f:
                if ln.startswith('{"kernel"'):
                    d = json.loads(ln)
                    if (d["source_hash"] == library_source_hash() and d["n_inputs"] == n_inputs
                            and d["n_mutants"] == n_mutants):
                        return d
    except OSError:
        pass
    return None


# kernels of one family (the library times a family's launches together)
FAMILY_KERNELS = {"lstm_kernel": ("lstm_kernel", "lstm_wide_kernel"),
                  "dw_col_kernel": ("dw_col_kernel", "dw_full_kernel", "dw_list_kernel")}


def _in_family(kernel: str, name: str) -> bool:
    return any(k in name for k in FAMILY_KERNELS.get(kernel, (kernel,)))


def _run_mutants_windows(rows):
    """Dispatch ids bracketing each run_mutants call: after run_original's
    label kernel, up to and including the score kernel."""
    wins, start = [], None
    for r in rows:
        name = r["Kernel_Name"]
        if "labels_kernel" in name:
            start = int(r["Dispatch_Id"])
        elif "score_kernel" in name and start is not None:
            wins.append((start, int(r["Dispatch_Id"])))
            start = None
    return wins


def summarize_pmc(fetch_csv: str, write_csv: str, kernel: str, args) -> str:
    """Markdown summary of two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE)
    of ``bench.py --steps 1 --warmup 0 --gain 0 --copy-calibration-mib M``:
    the copy of M MiB calibrates each counter (bytes it should see / bytes
    it reports); the kernel's run_mutants dispatches give the scaled HBM
    bytes per launch."""
    import csv
    per = {}
    calib = {}
    nbytes = args.copy_calibration_mib << 20
    for ctr, path in (("FETCH_SIZE", fetch_csv), ("WRITE_SIZE", write_csv)):
        rows = sorted(csv.DictReader(open(path)), key=lambda r: int(r["Dispatch_Id"]))
        rows = [r for r in rows if r["Counter_Name"] == ctr]
        copies = [r for r in rows if "copyBuffer" in r["Kernel_Name"]]
        big = max(copies, key=lambda r: float(r["Counter_Value"]))
        calib[ctr] = nbytes / (float(big["Counter_Value"]) * 1024.0)
        wins = _run_mutants_windows(rows)
        for r in rows:
            d = int(r["Dispatch_Id"])
            if _in_family(kernel, r["Kernel_Name"]) and any(a < d < b for a, b in wins):
                per.setdefault(d, {})[ctr] = float(r["Counter_Value"]) * 1024.0 * calib[ctr]
    ids = sorted(per)
    fetch = sum(per[d].get("FETCH_SIZE", 0.0) for d in ids)
    write = sum(per[d].get("WRITE_SIZE", 0.0) for d in ids)
    n = max(len(ids), 1)
    cmd = ("cd /tmp && export TMPDIR=/tmp && timeout -s KILL 240 rocprofv3 --pmc {C} --output-format csv "
           "-d <dir> -o pmc -- python3 bench.py --config %s --steps 1 --warmup 0 --no-cpu-baseline --gain 0 "
           "--copy-calibration-mib %d" % (args.config, args.copy_calibration_mib))
    out = [f"# HBM traffic of {kernel}, {args.config} ({args.inputs or 'default'} inputs, "
           f"{args.mutants or 'default'} mutants)", "",
           "Commands (one run per counter, C = FETCH_SIZE, then WRITE_SIZE), from the repository root:", "",
           "```", cmd, "python3 bench.py --summarize-pmc <fetch csv> <write csv> --kernel %s --config %s "
           "--copy-calibration-mib %d" % (kernel, args.config, args.copy_calibration_mib), "```", "",
           f"Calibration: a {args.copy_calibration_mib} MiB device-to-device copy (`__amd_rocclr_copyBuffer`) "
           f"moves {nbytes} bytes each way; bytes per reported byte: FETCH_SIZE x{calib['FETCH_SIZE']:.3f}, "
           f"WRITE_SIZE x{calib['WRITE_SIZE']:.3f}.", "",
           "| run_mutants dispatch | FETCH bytes (scaled) | WRITE bytes (scaled) |", "|---|---|---|"]
    for d in ids:
        out.append(f"| {d} | {per[d].get('FETCH_SIZE', 0):.4g} | {per[d].get('WRITE_SIZE', 0):.4g} |")
    rec = {"traffic_bytes_per_launch": (fetch + write) / n, "fetch_bytes_per_launch": fetch / n,
           "write_bytes_per_launch": write / n, "launches": len(ids), "kernel": kernel,
           "config": args.config, "n_inputs": args.n_inputs_resolved, "n_mutants": args.n_mutants_resolved,
           "calibration": calib, "source_hash": library_source_hash()}
    out += ["", "Per launch (machine-read by bench.py while the library sources hash to `source_hash`):",
            "", "```json", json.dumps(rec), "```", ""]
    return "\n".join(out)


def summarize_counters(csv_path: str, kernel: str, args) -> str:
    """Markdown summary of one rocprofv3 --pmc run of the MFMA counters
    (SQ_INSTS_VALU_MFMA_MOPS_<dtype>, SQ_VALU_MFMA_BUSY_CYCLES, GRBM_GUI_ACTIVE)
    over ``bench.py --steps 1 --warmup 0``: per launch of ``kernel`` inside
    run_mutants, the MFMA flops the hardware executed (512 per MOP), the core
    clock (GRBM_GUI_ACTIVE is summed over the XCDs: per XCD it counts the
    cycles of the dispatch), and the share of SIMD cycles with the matrix core
    busy (busy cycles summed over the SIMDs / (cycles x SIMDs))."""
    import csv
    rows = sorted(csv.DictReader(open(csv_path)), key=lambda r: int(r["Dispatch_Id"]))
    wins = _run_mutants_windows(rows)
    per, dur = {}, {}
    for r in rows:
        d = int(r["Dispatch_Id"])
        if _in_family(kernel, r["Kernel_Name"]) and any(a < d < b for a, b in wins):
            per.setdefault(d, {})
            per[d][r["Counter_Name"]] = per[d].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
            dur[d] = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9
    ids = sorted(per)
    names = sorted({c for d in ids for c in per[d]})
    mops = [c for c in names if c.startswith("SQ_INSTS_VALU_MFMA_MOPS_")]
    simds, xcds = args.simds, args.xcds
    cmd = ("cd /tmp && export TMPDIR=/tmp && timeout -s KILL 240 rocprofv3 --pmc %s --output-format csv "
           "-d <dir> -o pmc -- python3 bench.py --config %s --steps 1 --warmup 0 --no-cpu-baseline --gain 0 "
           "--no-measured-peaks" % (" ".join(names), args.config))
    out = [f"# MFMA counters of {kernel}, {args.config}", "",
           "Commands, from the repository root:", "", "```", cmd,
           "python3 bench.py --summarize-counters <counter_collection.csv> --kernel %s --config %s"
           % (kernel, args.config), "```", "",
           f"Per run_mutants launch of `{kernel}` ({len(ids)} launches; times are those of the counter "
           "run, whose dispatches are serialized and slower than in the kernel trace). Executed MFMA flops "
           f"= 512 x the MOPS counter; cycles = GRBM_GUI_ACTIVE / {xcds} XCDs; clock = cycles / "
           f"duration; MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (cycles x {simds} SIMDs).", "",
           "| dispatch | " + " | ".join(names) + " | ms | clock GHz | MFMA flops | MFMA busy |",
           "|---" * (len(names) + 5) + "|"]
    tot = {c: 0.0 for c in names}
    for d in ids:
        v = per[d]
        for c in names:
            tot[c] += v.get(c, 0.0)
        fl = 512.0 * sum(v.get(c, 0.0) for c in mops)
        cyc = v.get("GRBM_GUI_ACTIVE", 0.0) / xcds
        busy = v.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) / (cyc * simds) if cyc else 0.0
        ghz = cyc / dur[d] / 1e9 if dur[d] > 0 else 0.0
        out.append(f"| {d} | " + " | ".join(f"{v.get(c, 0.0):.4g}" for c in names) +
                   f" | {dur[d] * 1e3:.3f} | {ghz:.2f} | {fl:.4g} | {busy:.3f} |")
    n = max(len(ids), 1)
    fl = 512.0 * sum(tot[c] for c in mops) / n
    cyc = tot.get("GRBM_GUI_ACTIVE", 0.0) / xcds
    secs = sum(dur.values())
    rec = {"kernel": kernel, "config": args.config, "n_inputs": args.n_inputs_resolved,
           "n_mutants": args.n_mutants_resolved, "launches": len(ids), "mfma_flops_per_launch": fl,
           "mfma_busy": tot.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) / (cyc * simds) if cyc else 0.0,
           "cycles_per_launch": cyc / n, "mean_clock_ghz": cyc / secs / 1e9 if secs > 0 else 0.0,
           "ms_per_launch_counter_run": secs * 1e3 / n, "source_hash": library_source_hash()}
    out += ["", "All launches together:", "", "```json", json.dumps(rec), "```", ""]
    return "\n".join(out)


def summarize_trace(trace_csv: str, stats_csv: str, kernel: str, args) -> str:
    """Markdown summary of ``rocprofv3 --kernel-trace --stats`` over a default
    bench run: per-kernel totals, and the average duration of ``kernel``'s
    launches inside the timed memoized run_mutants calls (the figure bench.py
    measures with HIP events)."""
    import csv
    stats = list(csv.DictReader(open(stats_csv)))
    trace = sorted(csv.DictReader(open(trace_csv)), key=lambda r: int(r["Dispatch_Id"]))
    wins = _run_mutants_windows(trace)[args.warmup:args.warmup + args.steps]
    durs = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e6 for r in trace
            if _in_family(kernel, r["Kernel_Name"]) and any(a < int(r["Dispatch_Id"]) < b for a, b in wins)]
    cmd = ("cd /tmp && export TMPDIR=/tmp && rocprofv3 --kernel-trace --stats --output-format csv "
           "-d <dir> -o kt -- python3 bench.py --config %s --steps %d --warmup %d"
           % (args.config, args.steps, args.warmup))
    out = [f"# Kernel trace, {args.config} bench run", "", "Command, from the repository root:", "",
           "```", cmd, "python3 bench.py --summarize-trace <kernel_trace.csv> <kernel_stats.csv> --kernel %s "
           "--config %s --steps %d --warmup %d" % (kernel, args.config, args.steps, args.warmup), "```", "",
           f"`{kernel}` inside the {len(wins)} timed memoized run_mutants calls: {len(durs)} launches, "
           f"average {np.mean(durs) if durs else 0:.4f} ms, total {np.sum(durs):.3f} ms.", "",
           "All dispatches of the run (warm-up, timed, vanilla-mode gain steps, run_original):", "",
           "| kernel | calls | total ms | average us | % |", "|---|---|---|---|---|"]
    for r in sorted(stats, key=lambda r: -float(r["TotalDurationNs"]))[:20]:
        out.append(f"| `{r['Name'][:80]}` | {r['Calls']} | {float(r['TotalDurationNs']) / 1e6:.3f} | "
                   f"{float(r['AverageNs']) / 1e3:.1f} | {float(r['Percentage']):.1f} |")
    return "\n".join(out) + "\n"


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", default="resnet18w")
    ap.add_argument("--ratio-index", type=int, default=1)
    ap.add_argument("--inputs", type=int, default=None)
    ap.add_argument("--inputs-per-step", type=int, default=None,
                    help="inputs of one step's batch (default: 1,000 for resnet18w, else all)")
    ap.add_argument("--mutants", type=int, default=None)
    ap.add_argument("--oracle-mutants", type=int, default=None)
    ap.add_argument("--oracle-inputs", type=int, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--fused", type=int, default=1)
    ap.add_argument("--conv-tile", type=int, default=0)
    ap.add_argument("--workspace-mb", type=int, default=0,
                    help="cap the per-chunk activation workspace (0: the library default)")
    ap.add_argument("--set", action="append", metavar="NAME=VALUE",
                    help="a library option (mure_set_option), e.g. group_reads=0; repeatable")
    ap.add_argument("--gain", type=int, default=None,
                    help="also time vanilla mutation testing (every mutant from the raw "
                         "input) and report the paper's gain (t_v - t) / t_v (default: on "
                         "for mlp/lenet5)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="first copy a buffer of this many MiB device to device (a plain copy "
                         "kernel of known size, to scale the HBM byte counters of a profile)")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="print the HBM traffic summary of two rocprofv3 --pmc runs and exit")
    ap.add_argument("--summarize-trace", nargs=2, metavar=("TRACE_CSV", "STATS_CSV"),
                    help="print the kernel-trace summary of a rocprofv3 run and exit")
    ap.add_argument("--summarize-counters", metavar="COUNTER_CSV",
                    help="print the MFMA counter summary of a rocprofv3 --pmc run and exit")
    ap.add_argument("--simds", type=int, default=1024, help="SIMDs of the GPU (counter summaries)")
    ap.add_argument("--xcds", type=int, default=8, help="XCDs of the GPU (counter summaries)")
    ap.add_argument("--kernel", default="conv_lds_kernel", help="kernel the summaries follow")
    ap.add_argument("--no-measured-peaks", action="store_true",
                    help="skip the STREAM copy and MFMA-loop ceilings measured after the timed steps")
    args = ap.parse_args()
    cfgd = W.CONFIGS[args.config]
    n_all = args.inputs or cfgd["n_inputs"]
    ips = min(args.inputs_per_step or INPUTS_PER_STEP.get(args.config, n_all), n_all)
    if args.summarize_pmc or args.summarize_trace or args.summarize_counters:
        args.n_inputs_resolved = ips
        args.n_mutants_resolved = args.mutants or cfgd["n_mutants"]
        if args.summarize_pmc:
            print(summarize_pmc(*args.summarize_pmc, args.kernel, args), end="")
        elif args.summarize_counters:
            print(summarize_counters(args.summarize_counters, args.kernel, args), end="")
        else:
            print(summarize_trace(*args.summarize_trace, args.kernel, args), end="")
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: this build has no multi-GPU path "
              "(the inputs would shard across GPUs with one small all-gather of the "
              "per-mutant label masks at the end)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2607_18582_amd import Mure

    if args.copy_calibration_mib:
        nbytes = args.copy_calibration_mib << 20
        a = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda:0")
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": nbytes}), file=sys.stderr, flush=True)
        del a, b
    wl = W.make_workload(args.config, n_inputs=args.inputs, n_mutants=args.mutants,
                         ratio_index=args.ratio_index)
    md = wl.model
    M, N_all = wl.mutants.n_mutants, wl.n_inputs
    N = ips                                            # inputs per step
    n_batches = N_all // N
    dev = torch.device("cuda:0")
    x = wl.inputs
    xt = torch.from_numpy(x.view(np.int16).copy() if x.dtype == np.uint16 else x).to(dev)
    kill = torch.empty((M, (N + 63) // 64), dtype=torch.int64, device=dev)
    batch = [0]
    m = Mure(device=0)
    m.set_option("kernel_timing", 1)
    m.set_option("fused_paths", args.fused)
    m.set_option("conv_tile", args.conv_tile)
    if args.workspace_mb:
        m.set_option("max_workspace_mb", args.workspace_mb)
    for kv in args.set or []:
        k, v = kv.split("=", 1)
        m.set_option(k, int(v))

    walls = []                                         # host wall time of each call, per step

    def step():
        b0 = (batch[0] % n_batches) * N                # the next batch of the input set
        batch[0] += 1
        t = [time.perf_counter()]
        m.load_model(md.nodes, md.in_hwc, md.dtype, md.weights, md.biases)
        t.append(time.perf_counter())
        m.apply(wl.mutants)
        t.append(time.perf_counter())
        m.run_original(xt[b0:b0 + N])
        t.append(time.perf_counter())
        r = m.run_mutants(kill)
        t.append(time.perf_counter())
        walls.append(np.diff(t) * 1e3)
        return r

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    stats = []
    for _ in range(args.steps):
        _, kills, score = step()
        stats.append(m.stats())
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / args.steps

    ms_mut = float(np.median([s["ms_run_mutants"] for s in stats]))
    st = stats[-1]
    peak = PEAK_TFLOPS[md.dtype]
    kernel_peak = lambda f: PEAK_VALU_TFLOPS if f in VALU_FAMILIES else peak
    kernel_ms = np.mean([s["kernel_ms"] for s in stats], axis=0)

    def family_roof(f):
        """Roofline of kernel family f over run_mutants: HBM-bound when its
        algorithmic FLOP per byte sits below the ridge point of its compute
        peak, else bound by that peak."""
        ms = float(kernel_ms[f])
        flops = 2.0 * st["kernel_macs_algorithmic"][f]
        nbytes = float(st["kernel_bytes_algorithmic"][f])
        intensity = flops / nbytes if nbytes > 0 else float("inf")
        ridge = kernel_peak(f) * 1e12 / (PEAK_HBM_GBS * 1e9)
        if intensity < ridge:
            r = {"bound": "hbm", "achieved": nbytes / (ms * 1e-3) / 1e9 if ms > 0 else 0.0,
                 "peak": PEAK_HBM_GBS, "unit": "GB/s"}
        else:
            r = {"bound": "alu" if f in VALU_FAMILIES else "mfma",
                 "achieved": flops / (ms * 1e-3) / 1e12 if ms > 0 else 0.0,
                 "peak": kernel_peak(f), "unit": "TFLOP/s"}
        r["frac"] = r["achieved"] / r["peak"]
        return r, ms, flops, nbytes, intensity, ridge

    # the dominant kernel of run_mutants (largest summed launch time)
    fam = int(np.argmax(kernel_ms))
    roof, ms_k, alg_flops, alg_bytes, intensity, ridge = family_roof(fam)
    launches = st["kernel_launches"][fam]
    ms_gemm = float(np.mean([s["ms_gemm"] for s in stats]))
    all_flops = 2.0 * st["gemm_macs_algorithmic"]
    all_achieved = all_flops / (ms_gemm * 1e-3) / 1e12 if ms_gemm > 0 else 0.0
    tr = read_traffic(KERNEL_NAMES[fam], args.config, N, M)
    mc = read_counters(KERNEL_NAMES[fam], args.config, N, M)
    # every kernel family that ran: time, launches and its own roofline
    families = {}
    for f in range(len(KERNEL_NAMES)):
        if st["kernel_launches"][f] > 0:
            r = family_roof(f)[0]
            families[KERNEL_NAMES[f]] = {"ms": round(float(kernel_ms[f]), 4),
                                         "launches": int(st["kernel_launches"][f]),
                                         "bound": r["bound"], "frac": round(r["frac"], 4)}
    line = {
        "metric": "mutant-input suffix evals/sec + MFMA/HBM roofline fraction, 1 MI355X",
        "value": M * N / dt,
        "unit": "evals/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": dt * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": md.dtype,
        "data": "synthetic",
        "config": {"workload": f"{wl.name}: {wl.description}", "n_inputs": N_all, "n_mutants": M,
                   "inputs_per_step": N, "parallelism": "single GPU"},
        "suffix_evals_per_s": M * N / (ms_mut * 1e-3),
        "ms_run_mutants": ms_mut,
        "ms_run_original": float(np.median([s["ms_run_original"] for s in stats])),
        "ms_apply": float(np.median([s["ms_apply"] for s in stats])),
        # where a step's device time goes: a2 apply, a3 the original forward,
        # a4 the first mutated nodes, a5 + a6 the suffix layers and the kill /
        # score reduction (run_mutants minus a4)
        "time_split_ms": {"a2_apply": float(np.median([s["ms_apply"] for s in stats])),
                          "a3_run_original": float(np.median([s["ms_run_original"] for s in stats])),
                          "a4_first_mutated": float(np.median([s["ms_mmi"] for s in stats])),
                          "a5_a6_suffix_and_kill": ms_mut - float(np.median([s["ms_mmi"] for s in stats]))},
        # the same step by host wall time around each call (each returns once
        # its device work is done): a2 includes marshalling the records and
        # staging their noise, which the device time above does not see
        "wall_split_ms": dict(zip(("a1_load_model", "a2_apply_mutants", "a3_run_original", "a4_a6_run_mutants"),
                                  np.median(walls[args.warmup:args.warmup + args.steps], axis=0).round(2).tolist())),
        "mutation_score": [score["ms_num"], score["ms_den"]],
        "roofline": {**roof, "kernel": KERNELS[fam],
                     "traffic": tr["traffic_bytes_per_launch"] if tr else None,
                     "traffic_source": os.path.relpath(traffic_path(KERNEL_NAMES[fam], args.config), ROOT)
                     if tr else None,
                     # the hardware's view from the committed MFMA counter run: the
                     # share of SIMD cycles with the matrix core busy, at the clock
                     # the card ran (the vendor peak assumes 2.4 GHz)
                     "mfma_counters": {"busy": mc["mfma_busy"], "clock_ghz": mc["mean_clock_ghz"],
                                       "executed_flops_per_launch": mc["mfma_flops_per_launch"],
                                       "source": os.path.relpath(counters_path(KERNEL_NAMES[fam], args.config), ROOT)}
                     if mc else None,
                     "launches": launches, "avg_launch_ms": ms_k / max(launches, 1),
                     "alg_flops_per_launch": alg_flops / max(launches, 1),
                     "alg_bytes_per_launch": alg_bytes / max(launches, 1),
                     "flop_per_byte": intensity, "ridge_flop_per_byte": ridge,
                     "compute_frac": alg_flops / (ms_k * 1e-3) / 1e12 / kernel_peak(fam) if ms_k > 0 else 0.0,
                     "share_of_run_mutants": ms_k / ms_mut if ms_mut else None,
                     "all_weighted_layers": {"achieved": all_achieved, "frac": all_achieved / peak,
                                             "ms": ms_gemm, "launches": st["gemm_launches"]},
                     "families": families},
        "work": {"macs_algorithmic": st["macs_algorithmic"], "macs_executed": st["macs_executed"],
                 "macs_vanilla": st["macs_vanilla"], "macs_memoized": st["macs_memoized"],
                 "groups": st["n_groups"], "cache_bytes": st["cache_bytes"],
                 "launches_run_mutants": st["launches"]},
    }
    if args.gain if args.gain is not None else args.config in ("mlp", "lenet5"):
        # the paper's measure (Section 5.2): gain = (t_v - t) / t_v with every
        # overhead in both times; vanilla = the same library with memoization off
        m.set_option("vanilla", 1)
        batch[0] = 0                                     # the memoized steps' batches again
        for _ in range(args.warmup):
            step()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        vstats = []
        for _ in range(args.steps):
            _, vk, vscore = step()
            vstats.append(m.stats())
        torch.cuda.synchronize()
        dtv = (time.perf_counter() - t0) / args.steps
        m.set_option("vanilla", 0)
        line["paper_gain"] = {"gain": (dtv - dt) / dtv, "ms_per_step_memoized": dt * 1e3,
                              "ms_per_step_vanilla": dtv * 1e3,
                              "ms_run_mutants_vanilla": float(np.median([s["ms_run_mutants"] for s in vstats])),
                              "same_score": [vscore["ms_num"], vscore["ms_den"]] == [score["ms_num"], score["ms_den"]],
                              "macs_vanilla": vstats[-1]["macs_executed"]}
    if not args.no_measured_peaks:
        # the ceilings this card sustains (a STREAM copy, a register-only MFMA
        # loop), measured after the timed steps; the fractions above are
        # against the vendor's figures, these against the measured ones
        # (a failure here is reported in the line, which is printed regardless)
        try:
            from paper_2607_18582_amd.peaks import measure_peaks
            mp = measure_peaks(0)
            line["measured_peaks"] = {k: round(v, 2) for k, v in mp.items()}
            meas = {"hbm": mp["hbm_copy_gbs"],
                    "mfma": mp["mfma_bf16_tflops"] if md.dtype == "bf16" else mp["mfma_f32_tflops"]}
            mpk = meas.get(roof["bound"])
            line["roofline"]["measured_peak"] = mpk
            line["roofline"]["frac_of_measured"] = roof["achieved"] / mpk if mpk else None
        except Exception as e:  # noqa: BLE001
            line["measured_peaks"] = {"error": f"{type(e).__name__}: {e}"}
    if not args.no_cpu_baseline:
        # about 10 s of oracle work on the host cores
        om, oi = ORACLE_SAMPLE[args.config]
        om = args.oracle_mutants or om
        oi = args.oracle_inputs or oi
        line["cpu_baseline"] = cpu_baseline(wl, min(om, M), min(oi, N_all))
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
