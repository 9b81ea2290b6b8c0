"""The bench's profile summarizers on synthetic rocprofv3 CSVs (host only):
the kernel's launches inside run_mutants are the only ones counted."""
import argparse
import csv
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def _write(path, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value",
                                          "Start_Timestamp", "End_Timestamp"])
        w.writeheader()
        for r in rows:
            w.writerow(dict(zip(w.fieldnames, r)))


def test_summarize_counters_counts_only_run_mutants_launches(tmp_path):
    ctr = ("SQ_INSTS_VALU_MFMA_MOPS_BF16", "SQ_VALU_MFMA_BUSY_CYCLES", "GRBM_GUI_ACTIVE")
    rows = []
    # run_original's conv launch (outside any window), then one run_mutants
    # window: labels_kernel ... two conv launches ... score_kernel
    # (GRBM_GUI_ACTIVE summed over 8 XCDs; durations in ns)
    for d, name, vals, ns in [(1, "conv_halo_kernel<64,2,0>", (1e9, 1e9, 1e9), 10),
                              (2, "labels_kernel", (0, 0, 8), 10),
                              (3, "conv_halo_kernel<64,2,0>", (1000.0, 512000.0, 8000.0), 500),
                              (4, "conv_big_kernel<128>", (7.0, 7.0, 7.0), 10),
                              (5, "conv_halo_kernel<32,2,1>", (3000.0, 1536000.0, 24000.0), 1500),
                              (6, "score_kernel", (0, 0, 8), 10)]:
        for c, v in zip(ctr, vals):
            rows.append((d, name, c, v, 1000 * d, 1000 * d + ns))
    p = tmp_path / "pmc.csv"
    _write(p, rows)
    args = argparse.Namespace(config="resnet18w", simds=1024, xcds=8, n_inputs_resolved=1000,
                              n_mutants_resolved=500)
    md = bench.summarize_counters(str(p), "conv_halo_kernel", args)
    rec = json.loads(md.split("```json")[1].split("```")[0])
    assert rec["launches"] == 2
    assert rec["mfma_flops_per_launch"] == 512.0 * (1000.0 + 3000.0) / 2
    # cycles per XCD: 1,000 and 3,000; busy = SIMD-cycles busy / (cycles x SIMDs)
    assert abs(rec["mfma_busy"] - (512000.0 + 1536000.0) / ((1000.0 + 3000.0) * 1024)) < 1e-12
    assert rec["cycles_per_launch"] == 2000.0
    # 4,000 cycles in 2,000 ns: 2 GHz
    assert abs(rec["mean_clock_ghz"] - 2.0) < 1e-12
