"""Parity of the HIP path (through the C ABI) with the fp64 oracle.

Two bars, both per output tensor:
  * the stated tolerances (bf16 inputs, fp32 accumulation): loss relative
    error 1e-3, gradient relative L2 error 2e-2 (fp32 path 1e-5 / 1e-4);
  * element by element, |gpu - oracle| <= 8 sigma, with sigma the standard
    deviation of the rounding error that the mixed-precision convention
    puts into that element (tests/error_model.py: first-order propagation
    of every bf16 / fp32 rounding from the inputs to the output).  This is
    what catches a wrong element at a tile edge, which a norm over the
    tensor would let through.
Every row's NLL is compared the same way (the per-row loss of
ee_head_forward_loss).  Small shapes are compared in full and span several
tiles with ragged tails; the full-size workloads compare the loss, every
row's NLL, the gains' gradients in full, and weight-gradient rows at every
256-row tile boundary, across the whole last tile, at the most frequent
targets and at random.

Set EE_PARITY_LOG to a file path to append one JSON record per compared
tensor (worst error / bound ratio, relative L2 error).
"""

import json
import math
import os
import sys

import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
import error_model as EM

pytestmark = pytest.mark.gpu

LOSS_RTOL = 1e-3
GRAD_RTOL = 2e-2


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def record(case, tensor, worst, rel=None):
    path = os.environ.get("EE_PARITY_LOG")
    say(f"  {case} {tensor}: worst |err| / bound {worst:.3f}" + ("" if rel is None else f", rel_l2 {rel:.2e}"))
    if path:
        with open(path, "a") as f:
            f.write(json.dumps({"case": case, "tensor": tensor, "worst_ratio": worst, "rel_l2": rel}) + "\n")


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2402_00518_amd import binding
    binding.lib()          # fail loudly if the library is missing
    yield


def rel_l2(got, ref):
    ref = np.asarray(ref, dtype=np.float64)
    got = np.asarray(got, dtype=np.float64)
    den = np.linalg.norm(ref)
    if den < 1e-12:
        return float(np.max(np.abs(got))) if got.size else 0.0
    return float(np.linalg.norm(got - ref) / den)


def host(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def run(batch, flags=0, accumulate=0, steps=1):
    from paper_2402_00518_amd.session import Session
    s = Session.from_batch(batch)
    for _ in range(steps):
        s.step(flags=flags, accumulate=accumulate)
    torch.cuda.synchronize()
    s.check_device_error()
    return s


def gpu_row_losses(sess, flags=0):
    """Every row's NLL of every exit, from ee_head_forward_loss (run after the
    step; it leaves the gradients alone and rewrites the same losses)."""
    out = []
    for e in range(len(sess.c_exits)):
        sess.forward(e, flags=flags, row_loss=True)
        torch.cuda.synchronize()
        out.append(host(sess.row_loss))
    return out


def check_tensor(case, name, got, ref, sigma, rtol):
    err = rel_l2(got, ref)
    worst = EM.check_elementwise(f"{case} {name}", got, ref, sigma, floor=1e-30)
    record(case, name, worst, err)
    assert err <= rtol, (case, name, err)


def compare_full(sess, batch, loss_rtol=LOSS_RTOL, grad_rtol=GRAD_RTOL, dynamic=False, flags=0, case="case"):
    w = batch.workload
    exits = O.exits_from_batch(batch)
    xs = [W.decode(x) for x in batch.hidden]
    total, per = O.multi_exit_step(exits, xs, batch.targets, list(w.exit_weights), batch.token_weights, dynamic)
    got_total = float(sess.loss_total.item())
    assert abs(got_total - total) <= loss_rtol * abs(total), (got_total, total)
    rows = gpu_row_losses(sess, flags)
    for e, r in enumerate(per):
        got = float(sess.loss_per_exit[e].item())
        assert abs(got - r.loss) <= loss_rtol * abs(r.loss), (e, got, r.loss)
        sig = EM.step_sigma(exits[e], xs[e], batch.targets, w.exit_weights[e], w.dtype,
                            token_weights=batch.token_weights, dynamic_weights=dynamic)
        worst = EM.check_elementwise(f"{case} exit {e} row NLL", rows[e], r.row_loss, sig["row_loss"], floor=1e-30)
        record(case, f"exit {e} row NLL", worst)
        for name, ref in r.grads.items():
            check_tensor(case, f"exit {e} d_{name}", host(sess.grads[e]["d_" + name]), ref, sig[name], grad_rtol)
    return total, per


def small(kind, n, h, v, inter=0, dtype="bf16", weights=(1.0,), seed=0, random_gamma=True,
          token_weights=False, name="small", norm="rms", bias=False):
    w = W.custom(kind, n, h, v, inter, dtype, weights, row_scale=True, zipf=True, name=name,
                 norm=norm, bias=bias)
    return W.make_batch(w, seed, random_gamma=random_gamma, token_weights=token_weights)


# ------------------------------------------------------------------ small cases
def test_tiny_f32_workload_full_parity():
    """512 tokens, h 256, V 1024, fp32, single Norm exit (gain 1)."""
    say("case: tiny_norm_f32 seed 0")
    b = W.make_batch(W.WORKLOADS["tiny_norm_f32"], 0)
    s = run(b)
    compare_full(s, b, loss_rtol=1e-5, grad_rtol=1e-4, case="tiny_norm_f32")


SMALL_CASES = [
    ("norm_ragged", W.EXIT_NORM, 300, 192, 1000, 0, "bf16", False),
    ("norm_ragged_tokw", W.EXIT_NORM, 300, 192, 1000, 0, "bf16", True),
    ("embedding_ragged", W.EXIT_EMBEDDING, 200, 128, 777, 0, "bf16", False),
    ("mlp_ragged", W.EXIT_MLP, 260, 192, 900, 320, "bf16", False),
    ("mlp_ragged_tokw", W.EXIT_MLP, 130, 128, 513, 192, "bf16", True),
    ("norm_f32_ragged", W.EXIT_NORM, 70, 64, 333, 0, "f32", False),
    ("mlp_f32_ragged", W.EXIT_MLP, 150, 128, 300, 192, "f32", True),
    ("embedding_f32", W.EXIT_EMBEDDING, 129, 64, 129, 0, "f32", False),
    ("norm_one_token", W.EXIT_NORM, 1, 64, 50, 0, "bf16", False),
    ("norm_vocab_one", W.EXIT_NORM, 37, 64, 1, 0, "bf16", False),
    ("norm_multi_tile", W.EXIT_NORM, 1000, 512, 2000, 0, "bf16", False),
    # every MLP GEMM spans several 256-wide tiles with ragged M, N and K
    ("mlp_multi_tile", W.EXIT_MLP, 600, 320, 1100, 704, "bf16", False),
    # the widest rows the ABI accepts: hidden 32768 (K of the logits GEMM,
    # M of dW_out), and 8192 for an MLP exit (the norm backward's limit)
    ("norm_max_hidden", W.EXIT_NORM, 40, 32768, 200, 0, "bf16", False),
    ("mlp_max_hidden", W.EXIT_MLP, 96, 8192, 300, 256, "bf16", False),
    # the down projection and dZ with a split-K tail: 256 whole-K tiles
    # (tokens 0-2047) plus the last 152 tokens as four partial sums over I
    # (over V for dZ); then features 0-5375 whole and the last 64 features of
    # every token as four partial sums over a ragged I and V
    # (mlp_multi_tile: all outputs as two, and dZ as four)
    ("mlp_split_tokens", W.EXIT_MLP, 2200, 8192, 1024, 1024, "bf16", False),
    ("mlp_split_features", W.EXIT_MLP, 3000, 5440, 1088, 1088, "bf16", False),
    # the most tokens and the largest vocabulary the ABI accepts (2^20 each):
    # a dW_out product with K = 2^20 in one tile, and 16384 softmax slices
    ("norm_max_tokens", W.EXIT_NORM, 1 << 20, 64, 40, 0, "bf16", False),
    ("norm_max_vocab", W.EXIT_NORM, 64, 64, 1 << 20, 0, "bf16", False),
    # vocabulary-wide products of several rounds of 256-wide tiles with a
    # ragged last column of tiles (200 and 156 of 256 vocabulary ids), over
    # one and over four (ragged) rows of tiles
    ("norm_stagger_ragged_vocab", W.EXIT_NORM, 64, 64, 767 * 256 + 200, 0, "bf16", False),
    ("norm_stagger_ragged_rows", W.EXIT_NORM, 1000, 64, 199 * 256 + 156, 0, "bf16", True),
    # weight gradients launched as one block per CU looping over the tiles
    # (more than 512 tiles): dW_out over 3 x 201 tiles, ragged in both
    # dimensions; the gate and up gradients as one looping pair, 289 + 289
    # tiles ragged in both dimensions, with the pair's padding blocks between
    ("norm_loop_ragged", W.EXIT_NORM, 70, 576, 200 * 256 + 100, 0, "bf16", False),
    ("mlp_loop_ragged", W.EXIT_MLP, 96, 4160, 300, 4160, "bf16", False),
]


@pytest.mark.parametrize("name,kind,n,h,v,inter,dtype,tokw", SMALL_CASES, ids=[c[0] for c in SMALL_CASES])
def test_small_full_parity(name, kind, n, h, v, inter, dtype, tokw):
    say(f"case: {name} N={n} h={h} V={v} I={inter} {dtype}")
    b = small(kind, n, h, v, inter, dtype, seed=3, token_weights=tokw, name=name)
    s = run(b)
    tight = dtype == "f32"
    compare_full(s, b, loss_rtol=1e-5 if tight else LOSS_RTOL, grad_rtol=1e-4 if tight else GRAD_RTOL, case=name)


LAYERNORM_CASES = [
    ("layernorm_bias", 300, 192, 1000, "bf16", True, False),
    ("layernorm_no_bias", 300, 192, 1000, "bf16", False, False),
    ("layernorm_bias_tokw_multi_tile", 1000, 512, 2000, "bf16", True, True),
    ("layernorm_bias_f32", 70, 64, 333, "f32", True, False),
]


@pytest.mark.parametrize("name,n,h,v,dtype,bias,tokw", LAYERNORM_CASES, ids=[c[0] for c in LAYERNORM_CASES])
def test_layernorm_exit_parity(name, n, h, v, dtype, bias, tokw):
    # The LayerNorm flavour of the Norm exit (Sec. 2.1), with and without bias.
    say(f"case: {name} N={n} h={h} V={v} {dtype}")
    b = small(W.EXIT_NORM, n, h, v, 0, dtype, seed=4, token_weights=tokw, name=name, norm="layer", bias=bias)
    s = run(b)
    tight = dtype == "f32"
    _, per = compare_full(s, b, loss_rtol=1e-5 if tight else LOSS_RTOL, grad_rtol=1e-4 if tight else GRAD_RTOL,
                          case=name)
    assert ("beta" in per[0].grads) == bias


def test_row_losses_match():
    say("case: row losses norm_ragged")
    b = small(W.EXIT_NORM, 300, 192, 1000, seed=5, name="rows")
    from paper_2402_00518_amd.session import Session
    s = Session.from_batch(b)
    s.forward(0)
    torch.cuda.synchronize()
    ex, x = O.exits_from_batch(b)[0], W.decode(b.hidden[0])
    r = O.exit_step(ex, x, b.targets)
    sig = EM.step_sigma(ex, x, b.targets, 1.0, "bf16")
    worst = EM.check_elementwise("rows row NLL", host(s.row_loss), r.row_loss, sig["row_loss"], floor=1e-30)
    record("rows", "row NLL", worst)
    assert abs(float(s.loss_fwd[0, 0].item()) - r.loss) <= LOSS_RTOL * r.loss


def test_two_exits_mixed_kinds_weighted():
    say("case: two exits norm + mlp, weights 0.25 0.5")
    from paper_2402_00518_amd.session import Session
    bn = small(W.EXIT_NORM, 257, 128, 700, weights=(0.25,), seed=11, name="a")
    bm = small(W.EXIT_MLP, 257, 128, 700, 192, weights=(0.5,), seed=12, name="b")
    bm.targets = bn.targets
    exits = []
    for p in (bn.exits[0], bm.exits[0]):
        d = {"w_out": p.w_out, "gamma": p.gamma, "gamma_mlp": p.gamma_mlp, "w_gate": p.w_gate,
             "w_up": p.w_up, "w_down": p.w_down}
        exits.append({k: v for k, v in d.items() if v is not None})
    s = Session(W.EXIT_NORM, 1, 128, 700, 192, 1e-5, exits, [bn.hidden[0], bm.hidden[0]], bn.targets,
                None, (0.25, 0.5), kinds=[W.EXIT_NORM, W.EXIT_MLP])
    s.step()
    torch.cuda.synchronize()
    oe = O.exits_from_batch(bn) + O.exits_from_batch(bm)
    xs = [W.decode(bn.hidden[0]), W.decode(bm.hidden[0])]
    total, per = O.multi_exit_step(oe, xs, bn.targets, [0.25, 0.5])
    assert abs(s.loss_total.item() - total) <= LOSS_RTOL * total
    for e, wt in enumerate((0.25, 0.5)):
        sig = EM.step_sigma(oe[e], xs[e], bn.targets, wt, "bf16")
        for name, ref in per[e].grads.items():
            check_tensor("two_exits_mixed", f"exit {e} d_{name}", host(s.grads[e]["d_" + name]), ref, sig[name],
                         GRAD_RTOL)


def dynamic_batch(kind, n, h, v, inter, seed, tokw, name):
    b = small(kind, n, h, v, inter, seed=seed, token_weights=tokw, name=name)
    # larger output weights so that confidences vary between tokens
    b.exits[0].w_out = W.f32_to_bf16_bits(W.decode(b.exits[0].w_out).astype(np.float32) * 10)
    return b


DYNAMIC_CASES = [
    ("dyn_norm", W.EXIT_NORM, 300, 192, 500, 0, False),
    # Sec. 2.3 confidences times caller token weights, some of them zero
    ("dyn_norm_ragged_tokw", W.EXIT_NORM, 300, 192, 1000, 0, True),
    ("dyn_mlp_ragged_tokw", W.EXIT_MLP, 130, 128, 513, 192, True),
]


@pytest.mark.parametrize("name,kind,n,h,v,inter,tokw", DYNAMIC_CASES, ids=[c[0] for c in DYNAMIC_CASES])
def test_dynamic_token_weights(name, kind, n, h, v, inter, tokw):
    say(f"case: {name} dynamic token-wise weights N={n} h={h} V={v} I={inter} token weights {tokw}")
    from paper_2402_00518_amd.binding import EE_FLAG_DYNAMIC_TOKEN_WEIGHTS
    b = dynamic_batch(kind, n, h, v, inter, 21, tokw, name)
    if tokw:
        assert np.any(b.token_weights == 0) and np.any(b.token_weights != 1)
    s = run(b, flags=EE_FLAG_DYNAMIC_TOKEN_WEIGHTS)
    compare_full(s, b, dynamic=True, flags=EE_FLAG_DYNAMIC_TOKEN_WEIGHTS, case=name)


# -------------------------------------- the split entry points (Sec. 2.2)
SPLIT_CASES = [
    # name, kind, N, h, V, I, norm, bias, exit weight, dynamic
    ("split_norm", W.EXIT_NORM, 300, 192, 1000, 0, "rms", False, 0.35, False),
    ("split_mlp", W.EXIT_MLP, 260, 192, 900, 320, "rms", False, 0.6, False),
    ("split_layernorm_bias", W.EXIT_NORM, 300, 192, 1000, 0, "layer", True, 1.7, False),
    ("split_norm_dynamic_tokw", W.EXIT_NORM, 300, 192, 1000, 0, "rms", False, 0.5, True),
]


@pytest.mark.parametrize("name,kind,n,h,v,inter,norm,bias,wt,dyn", SPLIT_CASES, ids=[c[0] for c in SPLIT_CASES])
def test_split_forward_backward(name, kind, n, h, v, inter, norm, bias, wt, dyn):
    """ee_head_forward_loss then ee_head_backward (the per-exit forward and
    backward of Sec. 2.2): the loss and every row's NLL from the forward
    call, the gradients w_e dL_e/dtheta from the backward call, which reads
    the seed the forward call left in the workspace; a second pair with
    accumulate = 1 doubles the gradients."""
    say(f"case: {name} N={n} h={h} V={v} I={inter} {norm} bias {bias} w_e {wt} dynamic {dyn}")
    from paper_2402_00518_amd.binding import EE_FLAG_DYNAMIC_TOKEN_WEIGHTS
    from paper_2402_00518_amd.session import Session
    w = W.custom(kind, n, h, v, inter, "bf16", (wt,), row_scale=True, zipf=True, name=name, norm=norm, bias=bias)
    b = W.make_batch(w, 8, random_gamma=True, token_weights=dyn)
    flags = EE_FLAG_DYNAMIC_TOKEN_WEIGHTS if dyn else 0
    s = Session.from_batch(b)
    for g in s.grads[0].values():
        g.fill_(float("nan"))          # overwritten by accumulate = 0
    s.forward(0, flags=flags, row_loss=True)
    s.backward(0, accumulate=0)
    torch.cuda.synchronize()
    s.check_device_error()
    ex, x = O.exits_from_batch(b)[0], W.decode(b.hidden[0])
    r = O.exit_step(ex, x, b.targets, wt, b.token_weights, dyn)
    got = float(s.loss_fwd[0, 0].item())
    assert abs(got - r.loss) <= LOSS_RTOL * abs(r.loss), (got, r.loss)
    sig = EM.step_sigma(ex, x, b.targets, wt, "bf16", token_weights=b.token_weights, dynamic_weights=dyn)
    worst = EM.check_elementwise(f"{name} row NLL", host(s.row_loss), r.row_loss, sig["row_loss"], floor=1e-30)
    record(name, "row NLL", worst)
    first = {}
    for pname, ref in r.grads.items():
        g = s.grads[0]["d_" + pname]
        first[pname] = g.clone()
        check_tensor(name, f"d_{pname}", host(g), ref, sig[pname], GRAD_RTOL)
    assert set(first) == set(ex.param_names())
    s.forward(0, flags=flags, row_loss=False)
    s.backward(0, accumulate=1)
    torch.cuda.synchronize()
    for pname, g1 in first.items():
        # the same gradient again (deterministic), added in fp32: the sum of the
        # old value and this call's terms rounds once per addition (a bias adds
        # its term after the old value), so 2 g1 up to a few fp32 ulps of the terms
        g2 = s.grads[0]["d_" + pname]
        tol = 2.0 ** -21 * (2 * g1.abs() + g1.abs().max())
        assert torch.all((g2 - 2 * g1).abs() <= tol), pname


# ------------------------------------------------------------ properties
def test_zero_output_matrix_gives_ln_v():
    say("case: W_out = 0")
    b = small(W.EXIT_NORM, 200, 128, 1000, seed=31, name="zero")
    b.exits[0].w_out[:] = 0
    s = run(b)
    assert abs(s.loss_total.item() - math.log(1000)) < 1e-5 * math.log(1000)
    assert np.all(host(s.grads[0]["d_gamma"]) == 0.0)
    # Each seed row sums to zero up to bf16 rounding: sum_v |G[n, v]| <= 2 s_n and
    # bf16 keeps 8 significant bits, so |sum_v G[n, v]| <= 2^-7 s_n; the column
    # sums of dW_out = G^T Z are then bounded by 2^-7 sum_n s_n |Z[n, j]|.
    col = host(s.grads[0]["d_w_out"]).sum(axis=0)
    z = O.exit_forward(O.exits_from_batch(b)[0], W.decode(b.hidden[0]))["z"]
    bound = 2.0 ** -7 * np.sum(np.abs(z), axis=0) / 200 + 1e-6
    assert np.all(np.abs(col) <= bound)


def test_deterministic_and_accumulate():
    say("case: determinism + accumulate, mlp")
    b = small(W.EXIT_MLP, 200, 128, 600, 192, seed=41, name="det")
    s1, s2 = run(b), run(b)
    for k in s1.grads[0]:
        assert torch.equal(s1.grads[0][k], s2.grads[0][k]), k
    assert torch.equal(s1.loss_total, s2.loss_total)
    s3 = run(b, accumulate=1, steps=2)
    for k in s1.grads[0]:
        assert torch.allclose(s3.grads[0][k], 2 * s1.grads[0][k], rtol=1e-6, atol=0), k


def test_aliased_weights_give_identical_gradients():
    say("case: two exits aliasing one parameter set")
    from paper_2402_00518_amd import binding as B
    from paper_2402_00518_amd.session import Session
    b = small(W.EXIT_NORM, 150, 128, 400, seed=51, name="alias")
    p = b.exits[0]
    ex = {"w_out": p.w_out, "gamma": p.gamma}
    s = Session(W.EXIT_NORM, 1, 128, 400, 0, 1e-5, [ex, ex], [b.hidden[0], b.hidden[0]], b.targets,
                None, (1.0, 1.0))
    # point exit 1 at exit 0's parameter and hidden buffers (copy init shares weights)
    s.c_exits[1] = B.make_exit(W.EXIT_NORM, 1, 128, 400, 0, 1e-5, **s.params[0])
    s.x[1] = s.x[0]
    s.step()
    torch.cuda.synchronize()
    for k in s.grads[0]:
        assert torch.equal(s.grads[0][k], s.grads[1][k]), k


def test_mlp_gate_and_up_in_one_buffer():
    """The fused gate/up product reads W_up at a byte offset from W_gate (the
    interleaved B loader); an exit whose two projections are one buffer
    (offset 0) must match the oracle with W_up = W_gate, gradients included
    (d_w_gate and d_w_up stay separate outputs)."""
    say("case: MLP exit with W_up aliasing W_gate")
    from paper_2402_00518_amd import binding as B
    from paper_2402_00518_amd.session import Session
    b = small(W.EXIT_MLP, 260, 192, 900, 320, seed=61, name="gate_up_alias")
    b.exits[0].w_up = b.exits[0].w_gate.copy()
    s = Session.from_batch(b)
    prm = dict(s.params[0])
    prm["w_up"] = prm["w_gate"]
    s.c_exits[0] = B.make_exit(W.EXIT_MLP, s.dtype, 192, 900, 320, 1e-5, **prm)
    s.step()
    torch.cuda.synchronize()
    s.check_device_error()
    compare_full(s, b, case="gate_up_alias")


# Exits without a bias keep the logits unshifted (P = exp(S)) when every
# row's LSE is at most 50 and its largest logit at least -60; otherwise the
# step redoes the exit's logits, reduce and seed in the shifted form.  These
# cases force the second path: logits scaled up past the range (Norm, MLP,
# Embedding exits, and a ragged shape), and rows whose logits all lie far
# below zero.
FALLBACK_CASES = [
    ("range_large_norm", W.EXIT_NORM, 300, 256, 1000, 0, "bf16", "rms", False),
    ("range_large_norm_ragged", W.EXIT_NORM, 130, 192, 700, 0, "bf16", "rms", False),
    ("range_large_mlp", W.EXIT_MLP, 260, 192, 900, 320, "bf16", "rms", False),
    ("range_large_embedding", W.EXIT_EMBEDDING, 200, 128, 600, 0, "bf16", "rms", False),
    ("range_large_f32", W.EXIT_NORM, 150, 128, 300, 0, "f32", "rms", False),
    # a bias: the seed of the shifted rerun also sums G's rows
    ("range_large_layernorm_bias", W.EXIT_NORM, 300, 256, 1000, 0, "bf16", "layer", True),
]


@pytest.mark.parametrize("name,kind,n,h,v,inter,dtype,norm,bias", FALLBACK_CASES, ids=[c[0] for c in FALLBACK_CASES])
def test_logits_out_of_the_unshifted_range(name, kind, n, h, v, inter, dtype, norm, bias):
    say(f"case: {name} (logits scaled past the unshifted range)")
    b = small(kind, n, h, v, inter, dtype, seed=71, name=name, norm=norm, bias=bias)
    ex = b.exits[0]
    w = W.decode(ex.w_out)
    # rows of Z have norm about sqrt(h) (Embedding: the raw hidden rows);
    # aim the largest logits near 90
    scale = 90.0 / (3.0 * 0.02 * math.sqrt(h) * (3.0 if kind == W.EXIT_EMBEDDING else 1.0))
    ex.w_out = W._store((w * scale).astype(np.float32), dtype)
    s = run(b)
    _, per = compare_full(s, b, case=name,
                          loss_rtol=LOSS_RTOL if dtype == "bf16" else 1e-5,
                          grad_rtol=GRAD_RTOL if dtype == "bf16" else 1e-4)
    lse_max = max(float(np.max(r.row_loss)) for r in per)
    say(f"  {name}: largest row NLL {lse_max:.1f}")


def test_logits_all_far_below_zero():
    """Rows whose every logit is far below zero (their largest near -67):
    under -60, so the step takes the shifted form."""
    say("case: every logit near -80")
    n, h, v = 200, 128, 700
    b = small(W.EXIT_NORM, n, h, v, 0, "bf16", seed=73, name="range_negative", random_gamma=False)
    ex = b.exits[0]
    # hidden rows near a constant give x_hat near 1 and, with gamma = 1,
    # logits near sum_j W[v][j] = -80 (-74 on average) with a spread of
    # about 2 over the vocabulary, so that softmax rows and their roundings
    # differ from token to token
    rng = np.random.default_rng(5)
    b.hidden[0] = W._store((0.5 + 0.2 * rng.standard_normal((n, h))).astype(np.float32), "bf16")
    w = -80.0 / h + 0.2 * rng.standard_normal((v, h))
    ex.w_out = W._store(w.astype(np.float32), "bf16")
    x = W.decode(b.hidden[0])
    z = x / np.sqrt((x * x).mean(1, keepdims=True) + 1e-5)
    smax = (z @ W.decode(ex.w_out).T).max(1)
    assert smax.max() < -60.0, smax.max()  # every row is out of the unshifted range
    s = run(b)
    total, _ = compare_full(s, b, case="range_negative")
    assert math.isfinite(total)


def test_out_of_range_target_is_reported():
    say("case: target outside the vocabulary")
    from paper_2402_00518_amd import binding as B
    from paper_2402_00518_amd.session import Session
    b = small(W.EXIT_NORM, 100, 64, 300, seed=61, name="bad")
    b.targets[7] = 300
    s = Session.from_batch(b)
    s.step()
    with pytest.raises(B.EEError) as ei:
        s.check_device_error()
    assert ei.value.status == B.EE_ERR_TARGET
    assert math.isnan(s.loss_total.item())
    s.check_device_error()            # the record was cleared
    b.targets[7] = 0
    s2 = Session.from_batch(b)
    s2.step()
    s2.check_device_error()


# ----------------------------------------------------- full-size workloads
def boundary_rows(total, tile=256, extra=None):
    """Rows on both sides of every tile boundary, the whole last tile, and extra rows."""
    edges = [r for k in range(1, (total + tile - 1) // tile) for r in (k * tile - 1, k * tile)]
    last = list(range(((total - 1) // tile) * tile, total))
    rows = np.array(edges + last + ([] if extra is None else list(extra)), dtype=np.int64)
    return np.unique(rows[(rows >= 0) & (rows < total)])


def sampled_compare(name, seed=0, random_gamma=False):
    w = W.WORKLOADS[name]
    say(f"case: {name} full size seed {seed} random_gamma {random_gamma}")
    b = W.make_batch(w, seed, random_gamma=random_gamma)
    s = run(b)
    rows = gpu_row_losses(s)
    exits = O.exits_from_batch(b)
    counts = np.bincount(b.targets, minlength=w.vocab)
    v_rows = boundary_rows(w.vocab, extra=np.concatenate([W.row_sample(w.vocab, 24, seed), np.argsort(counts)[-4:]]))
    i_rows = boundary_rows(w.intermediate, extra=W.row_sample(w.intermediate, 12, seed)) \
        if w.kind == W.EXIT_MLP else None
    case = f"{name}{'_random_gamma' if random_gamma else ''}"
    total = 0.0
    for e, (ex, wt) in enumerate(zip(exits, w.exit_weights)):
        x = W.decode(b.hidden[e])
        ref = O.exit_step_sampled(ex, x, b.targets, wt, v_rows, i_rows)
        sig = EM.step_sigma(ex, x, b.targets, wt, w.dtype, v_rows=v_rows, i_rows=i_rows)
        L = float(ref["loss"])
        total += wt * L
        got = float(s.loss_per_exit[e].item())
        say(f"  exit {e} loss gpu {got:.6f} oracle {L:.6f}")
        assert abs(got - L) <= LOSS_RTOL * abs(L)
        worst = EM.check_elementwise(f"{case} exit {e} row NLL", rows[e], ref["row_loss"], sig["row_loss"],
                                     floor=1e-30)
        record(case, f"exit {e} row NLL (all {w.n_tokens})", worst)
        g = s.grads[e]
        vr = torch.as_tensor(v_rows).cuda()
        checks = [(f"d_w_out ({len(v_rows)} rows)", host(g["d_w_out"][vr]), ref["w_out_rows"], sig["w_out"])]
        if ex.kind != W.EXIT_EMBEDDING:
            checks.append(("d_gamma", host(g["d_gamma"]), ref["gamma"], sig["gamma"]))
        if ex.beta is not None:
            checks.append(("d_beta", host(g["d_beta"]), ref["beta"], sig["beta"]))
        if ex.kind == W.EXIT_MLP:
            ir = torch.as_tensor(i_rows).cuda()
            checks += [("d_gamma_mlp", host(g["d_gamma_mlp"]), ref["gamma_mlp"], sig["gamma_mlp"]),
                       (f"d_w_gate ({len(i_rows)} rows)", host(g["d_w_gate"][ir]), ref["w_gate_rows"], sig["w_gate"]),
                       (f"d_w_up ({len(i_rows)} rows)", host(g["d_w_up"][ir]), ref["w_up_rows"], sig["w_up"]),
                       (f"d_w_down ({len(i_rows)} columns)", host(g["d_w_down"][:, ir]), ref["w_down_cols"],
                        sig["w_down"])]
        for label, got_g, ref_g, sg in checks:
            check_tensor(case, f"exit {e} {label}", got_g, ref_g, sg, GRAD_RTOL)
    assert abs(s.loss_total.item() - total) <= LOSS_RTOL * abs(total)


@pytest.mark.parametrize("name", ["llama7b_norm", "llama7b_norm_2exits", "llama13b_mlp", "llama70b_norm",
                                  "llama7b_layernorm"])
def test_full_size_sampled_parity(name):
    sampled_compare(name)


def test_full_size_random_gamma():
    sampled_compare("llama7b_norm", seed=1, random_gamma=True)
