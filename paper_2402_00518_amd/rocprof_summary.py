"""Summaries of rocprofv3 runs of bench.py, for profiles/.

    python -m paper_2402_00518_amd.rocprof_summary trace --workload W \\
        --stats DIR/run_kernel_stats.csv --command "..." --bench-line BENCH.json --out profiles/step_kernels_W.md

writes a markdown table of the kernel-trace statistics and records each
step kernel's mean duration in profiles/kernel_times.json (tied to a digest
of the kernel sources; bench.py quotes it beside its own event timing while
the sources are unchanged).

    python -m paper_2402_00518_amd.rocprof_summary pmc --workload W \\
        --counters DIR/run_counter_collection.csv --command "..." --out profiles/mfma_W.md

summarises a counter run with SQ_VALU_MFMA_BUSY_CYCLES, SQ_BUSY_CYCLES and
GRBM_GUI_ACTIVE: per GEMM of the step, the mean duration under counter
collection, the shader clock per XCD (GRBM_GUI_ACTIVE is summed over the 8
XCDs), the MFMA-busy counter as a fraction of the SIMD cycles of the
dispatch (256 CUs x 4 SIMDs x active cycles per XCD), and the executed bf16
MFMA rate against the peak at 2.4 GHz and at the measured clock.
"""

from __future__ import annotations

import argparse
import csv
import json
import os
from collections import defaultdict

from .traffic import LABEL_KERNELS, ROOT, source_digest

TIMES_FILE = os.path.join(ROOT, "profiles", "kernel_times.json")
N_XCD, N_CU, SIMDS = 8, 256, 4
PEAK_BF16_TFLOPS = 2500.0
PEAK_CLOCK_GHZ = 2.4


def label_of(name: str):
    for label, pat in LABEL_KERNELS.items():
        pats = pat if isinstance(pat, tuple) else (pat,)
        if any(q in name for q in pats):
            return label
    return None


def short(name: str) -> str:
    s = name.replace("void ", "").replace("(anonymous namespace)::", "").split("(")[0]
    return s.replace("unsigned short", "bf16")


def gemm_flops(workload: str, label: str):
    import workloads as W
    w = W.WORKLOADS[workload]
    N, h, V, I = w.n_tokens, w.hidden, w.vocab, w.intermediate
    return {
        "logits + softmax partials": 2 * N * h * V,
        "output-matrix gradient": 2 * N * h * V,
        "dZ": 2 * N * h * V,
        "gate and up projections + swiglu": 4 * N * h * I,
        "down projection + residual": 2 * N * h * I,
        "dA + swiglu backward, down gradient": 4 * N * h * I,
        "gate and up gradients": 4 * N * h * I,
    }.get(label)


def cmd_trace(args):
    rows = list(csv.DictReader(open(args.stats)))
    total = sum(float(r["TotalDurationNs"]) for r in rows)
    digest = source_digest()
    rel = os.path.relpath(args.out, ROOT)
    try:
        data = json.load(open(TIMES_FILE))
    except (OSError, ValueError):
        data = {}
    rec = {}
    lines = [f"# Kernel durations of the exit-head step, {args.workload}", "",
             "Command (run from /tmp with `export TMPDIR=/tmp`; R = repository root):", "", "```",
             args.command, "```", ""]
    if args.bench_line:
        b = json.load(open(args.bench_line))
        r = b.get("roofline", {})
        lines += [f"The bench line of the same command: {b['ms_per_step']:.4f} ms/step, "
                  f"{b['value'] / 1e6:.3f} M tokens/s, {100 * b['mfma_peak_frac']:.1f}% of the 2.5 PF bf16 "
                  f"MFMA peak; dominant kernel {r.get('kernel')} at {r.get('avg_ms', float('nan')):.4f} ms mean by "
                  f"HIP events on the launch stream ({r.get('achieved', float('nan')):.0f} TFLOP/s, "
                  f"frac {r.get('frac', float('nan')):.3f}).", ""]
    lines += ["All kernels of the command: the step's (warmup, timed and event-timed steps), then the",
              "Adam update and the decode-time exit decision legs of bench.py.", "",
              "| kernel | calls | avg µs | min µs | max µs | % time |", "|---|---|---|---|---|---|"]
    for r in rows:
        lines.append(f"| `{short(r['Name'])}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                     f"{float(r['MinNs']) / 1e3:.1f} | {float(r['MaxNs']) / 1e3:.1f} | "
                     f"{100 * float(r['TotalDurationNs']) / total:.2f} |")
        lab = label_of(r["Name"])
        if lab is not None and lab not in rec:
            rec[lab] = {"avg_us": float(r["AverageNs"]) / 1e3, "calls": int(r["Calls"]), "source_digest": digest,
                        "file": rel, "command": args.command}
    lines.append("")
    for lab, v in rec.items():
        f = gemm_flops(args.workload, lab)
        if f is not None:
            tf = f / (v["avg_us"] / 1e6) / 1e12
            lines.append(f"- {lab}: {v['avg_us']:.1f} µs mean = {tf:.0f} TFLOP/s, "
                         f"{100 * tf / PEAK_BF16_TFLOPS:.1f}% of the bf16 peak")
    data[args.workload] = rec
    with open(TIMES_FILE, "w") as fh:
        json.dump(data, fh, indent=1, sort_keys=True)
        fh.write("\n")
    with open(args.out, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def cmd_pmc(args):
    disp = defaultdict(dict)
    for r in csv.DictReader(open(args.counters)):
        d = disp[int(r["Dispatch_Id"])]
        d["name"] = r["Kernel_Name"]
        d[r["Counter_Name"]] = float(r["Counter_Value"])
        d["ns"] = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
    acc = defaultdict(list)
    for d in disp.values():
        lab = label_of(d["name"])
        if lab is not None and gemm_flops(args.workload, lab) is not None:
            acc[lab].append(d)
    lines = [f"# MFMA utilisation and shader clock of the step's GEMMs, {args.workload}", "",
             "Command (run from /tmp with `export TMPDIR=/tmp`; R = repository root):", "", "```",
             args.command, "```", "",
             "Per GEMM, means over its dispatches (durations are under counter collection, which",
             "serialises dispatches).  clock = GRBM_GUI_ACTIVE / 8 XCDs / duration.  MFMA busy =",
             "SQ_VALU_MFMA_BUSY_CYCLES / (256 CUs x 4 SIMDs x GRBM_GUI_ACTIVE / 8).  SQ busy =",
             "SQ_BUSY_CYCLES / (GRBM_GUI_ACTIVE / 8), the raw ratio (summed over the SQs that report).",
             "Executed TF/s = the GEMM's 2MNK flops / duration; % of peak against 2.5 PF (2.4 GHz)",
             "and against the same MFMA rate at the measured clock.", "",
             "| GEMM | dispatches | avg µs | clock GHz | MFMA busy | SQ busy ratio | TFLOP/s | % 2.5 PF | % peak at clock |",
             "|---|---|---|---|---|---|---|---|---|"]
    for lab, ds in acc.items():
        n = len(ds)
        us = sum(d["ns"] for d in ds) / n / 1e3
        grbm = sum(d.get("GRBM_GUI_ACTIVE", 0.0) for d in ds) / n
        mfma = sum(d.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) for d in ds) / n
        sqb = sum(d.get("SQ_BUSY_CYCLES", 0.0) for d in ds) / n
        cyc = grbm / N_XCD
        clk = cyc / (us * 1e3)
        f = gemm_flops(args.workload, lab)
        tf = f / (us / 1e6) / 1e12
        lines.append(f"| {lab} | {n} | {us:.1f} | {clk:.2f} | {100 * mfma / (N_CU * SIMDS * cyc):.1f}% | "
                     f"{sqb / cyc:.2f} | {tf:.0f} | {100 * tf / PEAK_BF16_TFLOPS:.1f}% | "
                     f"{100 * tf / (PEAK_BF16_TFLOPS * clk / PEAK_CLOCK_GHZ):.1f}% |")
    with open(args.out, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    sub = ap.add_subparsers(dest="cmd", required=True)
    t = sub.add_parser("trace")
    t.add_argument("--workload", required=True)
    t.add_argument("--stats", required=True)
    t.add_argument("--command", required=True)
    t.add_argument("--bench-line", default="")
    t.add_argument("--out", required=True)
    p = sub.add_parser("pmc")
    p.add_argument("--workload", required=True)
    p.add_argument("--counters", required=True)
    p.add_argument("--command", required=True)
    p.add_argument("--out", required=True)
    args = ap.parse_args()
    cmd_trace(args) if args.cmd == "trace" else cmd_pmc(args)


if __name__ == "__main__":
    main()
