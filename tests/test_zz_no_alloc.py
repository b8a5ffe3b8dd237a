"""ee_exit_decide_static (the decode-time decision without a workspace
argument) against ee_exit_decide (the same decision with a caller
workspace), through the C ABI, on two calls in a row, the second with a
smaller input.  Both run the same kernels in the same order, so the token
ids, exit flags and confidences must agree bit for bit.
"""

import numpy as np
import pytest
import torch

import workloads as W
from paper_2402_00518_amd import binding as B
from paper_2402_00518_amd.session import to_device

pytestmark = pytest.mark.gpu


def say(msg):
    print(msg, flush=True)


def exit_on_device(kind, n, h, V, I, seed, norm="rms", bias=False):
    w = W.custom(kind, n, h, V, I, "bf16", (1.0,), row_scale=True, zipf=True, name=f"noalloc{seed}",
                 norm=norm, bias=bias)
    b = W.make_batch(w, seed, random_gamma=True)
    p = b.exits[0]
    d = {"w_out": p.w_out, "gamma": p.gamma, "gamma_mlp": p.gamma_mlp, "w_gate": p.w_gate,
         "w_up": p.w_up, "w_down": p.w_down, "beta": p.beta}
    t = {k: to_device(a, "cuda") for k, a in d.items() if a is not None}
    nrm = B.EE_NORM_LAYER if norm == "layer" else B.EE_NORM_RMS
    e = B.make_exit(kind, B.EE_BF16, h, V, I if kind == B.EE_EXIT_MLP else 0, 1e-5, norm=nrm, **t)
    return e, t, to_device(b.hidden[0], "cuda")


def decide_both(e, x, n, threshold):
    stream = torch.cuda.current_stream().cuda_stream
    outs = []
    for static in (False, True):
        token = torch.full((n,), -1, dtype=torch.int32, device="cuda")
        conf = torch.full((n,), -1.0, dtype=torch.float32, device="cuda")
        flag = torch.full((n,), -1, dtype=torch.int32, device="cuda")
        if static:
            B.ee_exit_decide_static(e, x, n, threshold, token, conf, flag, stream)
        else:
            ws_bytes = B.ee_decode_workspace_bytes(e, n)
            ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
            B.ee_exit_decide(e, x, n, threshold, token, conf, flag, ws, ws_bytes, stream)
        torch.cuda.synchronize()
        outs.append((token.cpu().numpy(), conf.cpu().numpy(), flag.cpu().numpy()))
    return outs


CASES = [
    ("norm", B.EE_EXIT_NORM, 4096, 32000, 0, "rms", False),
    ("mlp", B.EE_EXIT_MLP, 1024, 5000, 2048, "rms", False),
    ("layernorm_bias", B.EE_EXIT_NORM, 512, 3001, 0, "layer", True),
]


@pytest.mark.parametrize("name,kind,h,V,I,norm,bias", CASES, ids=[c[0] for c in CASES])
def test_static_workspace_matches_caller_workspace(name, kind, h, V, I, norm, bias):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()
    for call, (n, seed) in enumerate(((37, 1), (5, 2))):   # second call: fewer rows, other values
        say(f"case: no-alloc decide {name} call {call} rows {n} h {h} V {V} I {I}")
        e, params, x = exit_on_device(kind, n, h, V, I, seed, norm, bias)
        assert B.ee_decode_workspace_bytes(e, n) <= B.EE_STATIC_SCRATCH_BYTES
        (t0, c0, f0), (t1, c1, f1) = decide_both(e, x, n, 0.05)
        assert np.all((t0 >= 0) & (t0 < V)), t0
        assert np.all((f0 == 0) | (f0 == 1))
        np.testing.assert_array_equal(t1, t0)
        np.testing.assert_array_equal(f1, f0)
        np.testing.assert_array_equal(c1.view(np.uint32), c0.view(np.uint32))


def test_static_workspace_rejects_too_many_rows():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    e, params, x = exit_on_device(B.EE_EXIT_NORM, 8, 4096, 32000, 0, 3)
    n = 1
    while B.ee_decode_workspace_bytes(e, n) <= B.EE_STATIC_SCRATCH_BYTES:
        n *= 2
    out = torch.zeros(3 * n, dtype=torch.int32, device="cuda")
    s = B.ee_exit_decide_static(e, x, n, 0.5, out[:n], out[n:2 * n], out[2 * n:], None, check=False)
    assert s == B.EE_ERR_WORKSPACE, B.ee_last_error()
