"""The committed rocprofv3 summaries label every GEMM of the step.

bench.py quotes the dominant kernel's mean from profiles/kernel_times.json
and its HBM bytes from profiles/traffic.json by label; a kernel whose name
no label matches (say, after a new launch form) would silently drop out of
both.  No GPU needed: these read committed text.
"""

import json
import os
import re

import pytest

from paper_2402_00518_amd.rocprof_summary import label_of

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PROFILES = os.path.join(ROOT, "profiles")

NORM_GEMMS = ["logits + softmax partials", "output-matrix gradient"]
STEP_GEMMS = {
    "llama7b_norm": NORM_GEMMS,
    "llama7b_norm_2exits": NORM_GEMMS,
    "llama70b_norm": NORM_GEMMS,
    "llama7b_layernorm": NORM_GEMMS,
    "llama13b_mlp": NORM_GEMMS + ["gate and up projections + swiglu", "down projection + residual", "dZ",
                                  "dA + swiglu backward, down gradient", "gate and up gradients"],
}


def test_kernel_times_hold_every_gemm_of_the_step():
    data = json.load(open(os.path.join(PROFILES, "kernel_times.json")))
    for workload, labels in STEP_GEMMS.items():
        missing = set(labels) - set(data.get(workload, {}))
        assert not missing, (workload, missing)


@pytest.mark.parametrize("workload", sorted(STEP_GEMMS))
def test_every_gemm_in_the_trace_has_a_label(workload):
    text = open(os.path.join(PROFILES, f"step_kernels_{workload}.md")).read()
    names = re.findall(r"^\| `([^`]*gemm[^`]*)` \|", text, flags=re.M)
    assert names
    for name in names:
        if "gated" in name:  # the shifted rerun, which returns at once unless a row is out of range
            continue
        raw = name.replace("bf16", "unsigned short")  # the summaries shorten the element type
        assert label_of(raw) is not None, name
