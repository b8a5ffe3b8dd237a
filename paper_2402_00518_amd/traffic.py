"""HBM traffic per kernel launch from rocprofv3 counter runs.

Two counter runs of the same bench command give, per dispatch, FETCH_SIZE
(KiB read past L2) and WRITE_SIZE (KiB written past L2).  The bench command
also copies a buffer of known size a few times (``bench.py
--copy-calibration-mib M``); what the counters read for that plain copy
calibrates them: scaled bytes = counter bytes * known bytes / copy's counter
bytes, separately for reads and writes.

    python -m paper_2402_00518_amd.traffic --workload llama7b_norm \\
        --fetch DIR_A/run_counter_collection.csv --write DIR_B/run_counter_collection.csv \\
        --copy-bytes 1073741824 --command "..."

updates ``profiles/traffic.json``.  The figures are tied to a digest of the
kernel sources; bench.py reports them only while the sources are unchanged.
"""

from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
from collections import defaultdict

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")

# Profiling label -> substring(s) of the demangled kernel name (one launch
# per exit and step each; a tuple lists the alternatives, e.g. with and
# without a split-K tail).
LABEL_KERNELS = {
    "logits + softmax partials": "gemm_kernel<unsigned short, true, true, ee::EpiLogits<",
    "output-matrix gradient": ("gemm_kernel<unsigned short, true, true, ee::EpiWeightGrad<",
                               "gemm_persistent_kernel<unsigned short, true, true, ee::EpiWeightGrad<"),
    "dZ": ("gemm_kernel<unsigned short, false, false, ee::EpiStoreF32<",
           "gemm_pair_kernel<unsigned short, false, false, ee::EpiStoreF32<"),
    "gate and up gradients": ("gemm_pair_kernel<unsigned short, true, true, ee::EpiWeightGrad<",
                              "gemm_pair_persistent_kernel<unsigned short, true, true, ee::EpiWeightGrad<"),
    "gate and up projections + swiglu": "ee::EpiGateUp<",
    "down projection + residual": "ee::EpiResidual<",
    "dA + swiglu backward, down gradient": "ee::EpiSwiGLUBwd<",
    "logit seed": "seed_kernel",
    "operand scale (or seed, if out of range) and loss": "seed_or_scale_kernel",
    "cross-entropy reduce": "ce_reduce_kernel",
    # normalisation passes: the exit norm (and the MLP pre-norm, whose input
    # is the bf16 hidden state as well) in one pass, or as statistics and
    # apply where a block's rows do not fit its LDS; the statistics that
    # first add the split down projection's slices, the apply of the MLP
    # exit norm to the fp32 residual stream, and the norm backward of the
    # MLP exit
    "norm (one pass)": "norm_rows_kernel<",
    "norm statistics": "row_rms_kernel<",
    "norm statistics (split sum)": "row_rms_split_kernel<",
    "norm apply": "norm_apply_kernel<unsigned short, unsigned short>",
    "norm apply (fp32 input)": "norm_apply_kernel<float, unsigned short>",
    "exit norm backward": "norm_bwd_kernel<",
    "gain reduce": "gain_reduce_kernel",
    "adam update": "adam_kernel",
}
COPY_KERNEL = "__amd_rocclr_copyBuffer"


def source_digest() -> str:
    """Digest of the HIP/C++ sources of the library (kernels and ABI)."""
    d = hashlib.sha256()
    csrc = os.path.join(PKG, "csrc")
    for f in sorted(os.listdir(csrc)):
        if f.endswith((".h", ".hip", ".cpp")):
            d.update(open(os.path.join(csrc, f), "rb").read())
    return d.hexdigest()[:16]


def read_counter(path: str, counter: str):
    """[(dispatch id, kernel name, value in KiB)] for one counter, in dispatch order."""
    rows = []
    with open(path, newline="") as f:
        for r in csv.DictReader(f):
            if r["Counter_Name"] == counter:
                rows.append((int(r["Dispatch_Id"]), r["Kernel_Name"], float(r["Counter_Value"])))
    rows.sort()
    return rows


def copy_factor(rows, copy_bytes: int, copies: int) -> tuple[float, float]:
    """Known bytes / counter bytes of the calibration copies (the `copies`
    largest copy dispatches), and their mean counter KiB."""
    vals = sorted((v for _, name, v in rows if COPY_KERNEL in name), reverse=True)[:copies]
    if len(vals) < copies:
        raise SystemExit(f"found {len(vals)} copy dispatches, expected {copies}")
    kib = sum(vals) / len(vals)
    return copy_bytes / (kib * 1024.0), kib


def per_label(rows):
    """Mean counter KiB per dispatch for every label of LABEL_KERNELS."""
    acc = defaultdict(list)
    for _, name, v in rows:
        for label, pat in LABEL_KERNELS.items():
            pats = pat if isinstance(pat, tuple) else (pat,)
            if any(q in name for q in pats):
                acc[label].append(v)
    return {k: (sum(v) / len(v), len(v)) for k, v in acc.items()}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--workload", required=True)
    ap.add_argument("--fetch", required=True, help="counter_collection.csv of the FETCH_SIZE run")
    ap.add_argument("--write", required=True, help="counter_collection.csv of the WRITE_SIZE run")
    ap.add_argument("--copy-bytes", type=int, required=True)
    ap.add_argument("--copies", type=int, default=3)
    ap.add_argument("--command", default="", help="the rocprofv3 commands, recorded with the figures")
    ap.add_argument("--out", default=TRAFFIC_FILE)
    args = ap.parse_args()

    fr = read_counter(args.fetch, "FETCH_SIZE")
    wr = read_counter(args.write, "WRITE_SIZE")
    ff, fkib = copy_factor(fr, args.copy_bytes, args.copies)
    wf, wkib = copy_factor(wr, args.copy_bytes, args.copies)
    fl, wl = per_label(fr), per_label(wr)
    try:
        data = json.load(open(args.out))
    except (OSError, ValueError):
        data = {}
    digest = source_digest()
    data.setdefault("copy_calibration", {})[args.workload] = {
        "copy_bytes": args.copy_bytes, "fetch_kib": fkib, "write_kib": wkib,
        "fetch_factor": ff, "write_factor": wf}
    rec = data.setdefault(args.workload, {})
    for label in sorted(set(fl) & set(wl)):
        fb = fl[label][0] * 1024.0 * ff
        wb = wl[label][0] * 1024.0 * wf
        rec[label] = {"fetch_bytes_per_launch": fb, "write_bytes_per_launch": wb,
                      "bytes_per_launch": fb + wb, "dispatches": fl[label][1],
                      "source_digest": digest, "command": args.command}
        print(f"{label:28s} read {fb / 1e6:10.2f} MB  write {wb / 1e6:10.2f} MB  ({fl[label][1]} dispatches)")
    print(f"copy calibration: read factor {ff:.4f}, write factor {wf:.4f}")
    os.makedirs(os.path.dirname(args.out), exist_ok=True)
    with open(args.out, "w") as f:
        json.dump(data, f, indent=1, sort_keys=True)
        f.write("\n")


if __name__ == "__main__":
    main()
