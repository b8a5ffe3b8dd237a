"""Table of the GPU parity margins from EE_PARITY_LOG records.

    python tests/parity_table.py LOG.jsonl [LOG2.jsonl ...] --command "..." > profiles/parity_errors.md

One row per compared tensor (a later record of the same case and tensor
replaces an earlier one): the worst |gpu - oracle| over its bound
8 sigma (tests/error_model.py; at most 1 to pass) and the relative L2 error
(bar 2e-2, fp32 cases 1e-4).
"""

import argparse
import json


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("logs", nargs="+")
    ap.add_argument("--command", required=True)
    args = ap.parse_args()
    recs = {}
    for path in args.logs:
        for line in open(path):
            r = json.loads(line)
            recs[(r["case"], r["tensor"])] = r
    print("# GPU parity margins: every compared tensor of the `-m gpu` parity suite")
    print()
    print("Command (on one MI355X, from the repository root):")
    print()
    print("```")
    print(args.command)
    print("```")
    print()
    print("worst = max over the tensor's elements of |gpu - oracle| / (8 sigma), sigma from the")
    print("rounding-error model of tests/error_model.py (a tensor passes at worst <= 1); rel_l2 =")
    print("||gpu - oracle|| / ||oracle|| (bar 2e-2 for bf16, 1e-4 for fp32).  Row NLL: every row.")
    print()
    worst_all = max(r["worst_ratio"] for r in recs.values())
    print(f"{len(recs)} tensors; largest worst ratio {worst_all:.3f}.")
    print()
    print("| case | tensor | worst / 8σ | rel_l2 |")
    print("|---|---|---|---|")
    for (case, tensor), r in sorted(recs.items()):
        rel = "" if r["rel_l2"] is None else f"{r['rel_l2']:.2e}"
        print(f"| {case} | {tensor} | {r['worst_ratio']:.3f} | {rel} |")


if __name__ == "__main__":
    main()
