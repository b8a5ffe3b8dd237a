"""Pins of the fp64 oracle against facts fixed by the paper and by mathematics.

Each test would fail for a plausible mistake in the oracle: a dropped term,
a wrong sign or index, a transposed operand, a wrong reduction or scale.
None of these tests runs the HIP path.
"""

import json
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle as O
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_worked_exits.json")


def rand_exit(kind, h, V, I, rng, scale=0.3, eps=1e-5, random_gamma=True):
    e = O.Exit(kind=kind, w_out=rng.standard_normal((V, h)) * scale, eps=eps)
    if kind in (O.EXIT_NORM, O.EXIT_MLP):
        e.gamma = 1.0 + 0.3 * rng.standard_normal(h) if random_gamma else np.ones(h)
    if kind == O.EXIT_MLP:
        e.gamma_mlp = 1.0 + 0.3 * rng.standard_normal(h) if random_gamma else np.ones(h)
        e.w_gate = rng.standard_normal((I, h)) * scale
        e.w_up = rng.standard_normal((I, h)) * scale
        e.w_down = rng.standard_normal((h, I)) * scale
    return e


def loss_only(e, x, y, w=1.0, m=None):
    return O.exit_step(e, x, y, w, m).loss * w


KINDS = [O.EXIT_EMBEDDING, O.EXIT_NORM, O.EXIT_MLP]


# ------------------------------------------------------------- golden cases
def test_hand_worked_golden():
    """Hand-derived closed forms (tests/golden/hand_worked_exits.json)."""
    fx = json.load(open(GOLDEN))
    for c in fx["cases"]:
        kind = c["kind"]
        e = O.Exit(kind=kind, w_out=np.array(c["w_out"]), eps=c["eps"])
        if "gamma" in c:
            e.gamma = np.array(c["gamma"])
        x = np.array(c["x"])
        y = np.array(c["y"])
        r = O.exit_step(e, x, y, c["exit_weight"])
        assert r.loss == pytest.approx(c["loss"], rel=1e-14, abs=1e-15), c["name"]
        np.testing.assert_allclose(r.row_loss, c["row_loss"], rtol=1e-14, atol=1e-15)
        np.testing.assert_allclose(r.grads["w_out"], c["d_w_out"], rtol=1e-13, atol=1e-15)
        if "d_gamma" in c:
            np.testing.assert_allclose(r.grads["gamma"], c["d_gamma"], rtol=1e-13, atol=1e-15)


# ---------------------------------------------------------- P1 uniform logits
@pytest.mark.parametrize("kind", KINDS)
def test_zero_output_matrix_gives_ln_v_and_closed_form_grads(kind):
    rng = np.random.default_rng(1)
    N, h, V, I = 7, 16, 11, 24
    e = rand_exit(kind, h, V, I, rng)
    e.w_out[:] = 0.0
    x = rng.standard_normal((N, h)) * 2.0
    y = rng.integers(0, V, N)
    w = 0.7
    r = O.exit_step(e, x, y, w)
    assert r.loss == pytest.approx(math.log(V), rel=1e-15)
    np.testing.assert_allclose(r.row_loss, math.log(V), rtol=1e-15)
    # dW_out[v, j] = (w / N) sum_n Z[n, j] (1/V - [y_n = v])
    z = O.exit_forward(e, x)["z"]
    onehot = np.zeros((N, V))
    onehot[np.arange(N), y] = 1.0
    expect = (w / N) * (1.0 / V - onehot).T @ z
    np.testing.assert_allclose(r.grads["w_out"], expect, rtol=1e-12, atol=1e-15)
    for k, g in r.grads.items():
        if k != "w_out":        # dZ = G W_out = 0 kills every other gradient
            assert np.all(g == 0.0), k


# ------------------------------------------------------ P2/P3 row/col sums
def test_seed_rows_sum_to_zero_and_dw_columns_sum_to_zero():
    rng = np.random.default_rng(2)
    N, h, V = 9, 12, 17
    e = rand_exit(O.EXIT_NORM, h, V, 0, rng, scale=1.0)
    x = rng.standard_normal((N, h))
    y = rng.integers(0, V, N)
    s = O.exit_forward(e, x)["s"]
    g = O.logit_grad(s, y, np.full(N, 0.3))
    assert np.max(np.abs(g.sum(axis=1))) < 1e-15
    assert np.all(g[np.arange(N), y] < 0) and np.all(np.delete(g.ravel(), np.arange(N) * V + y) > 0)
    r = O.exit_step(e, x, y, 1.0)
    assert np.max(np.abs(r.grads["w_out"].sum(axis=0))) < 1e-15


# ------------------------------------------------------- P4 finite differences
@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("weighted", [False, True])
def test_central_finite_differences(kind, weighted):
    rng = np.random.default_rng(10 + kind)
    N, h, V, I = 5, 8, 13, 12
    e = rand_exit(kind, h, V, I, rng, scale=0.4)
    x = rng.standard_normal((N, h)) * np.exp(0.5 * rng.standard_normal((N, 1)))
    y = rng.integers(0, V, N)
    m = rng.random(N) if weighted else None
    w = 0.35
    r = O.exit_step(e, x, y, w, m)
    delta = 1e-6
    for name in e.param_names():
        p = getattr(e, name)
        an = r.grads[name]
        fd = np.zeros_like(p)
        for idx in np.ndindex(p.shape):
            old = p[idx]
            p[idx] = old + delta
            lp = loss_only(e, x, y, w, m)
            p[idx] = old - delta
            lm = loss_only(e, x, y, w, m)
            p[idx] = old
            fd[idx] = (lp - lm) / (2 * delta)
        scale = max(1.0, np.max(np.abs(an)))
        assert np.max(np.abs(fd - an)) <= 1e-7 * scale, (name, np.max(np.abs(fd - an)))


def test_finite_differences_two_exits_joint_loss():
    rng = np.random.default_rng(20)
    N, h, V, I = 4, 8, 9, 8
    exits = [rand_exit(O.EXIT_NORM, h, V, I, rng), rand_exit(O.EXIT_MLP, h, V, I, rng)]
    xs = [rng.standard_normal((N, h)), rng.standard_normal((N, h))]
    y = rng.integers(0, V, N)
    ws = [0.25, 0.5]
    total, per = O.multi_exit_step(exits, xs, y, ws)
    delta = 1e-6
    for ei, e in enumerate(exits):
        for name in e.param_names():
            p = getattr(e, name)
            for idx in list(np.ndindex(p.shape))[::3]:
                old = p[idx]
                p[idx] = old + delta
                lp = O.multi_exit_step(exits, xs, y, ws)[0]
                p[idx] = old - delta
                lm = O.multi_exit_step(exits, xs, y, ws)[0]
                p[idx] = old
                fd = (lp - lm) / (2 * delta)
                assert abs(fd - per[ei].grads[name][idx]) < 1e-8, (ei, name, idx)


# -------------------------------------------------- P5 torch autograd (fp64)
@pytest.mark.parametrize("kind", KINDS)
def test_against_torch_autograd(kind):
    rng = np.random.default_rng(30 + kind)
    N, h, V, I, eps = 6, 16, 21, 20, 1e-5
    e = rand_exit(kind, h, V, I, rng, eps=eps)
    x = rng.standard_normal((N, h))
    y = rng.integers(0, V, N)
    w = 0.6
    r = O.exit_step(e, x, y, w)

    tp = {k: torch.tensor(getattr(e, k), requires_grad=True) for k in e.param_names()}
    tx = torch.tensor(x)
    if kind == O.EXIT_MLP:
        u = F.rms_norm(tx, (h,), tp["gamma_mlp"], eps)
        a = F.silu(F.linear(u, tp["w_gate"])) * F.linear(u, tp["w_up"])
        s_in = tx + F.linear(a, tp["w_down"])
    else:
        s_in = tx
    z = F.rms_norm(s_in, (h,), tp["gamma"], eps) if kind != O.EXIT_EMBEDDING else s_in
    logits = F.linear(z, tp["w_out"])
    loss = F.cross_entropy(logits, torch.tensor(y), reduction="mean")
    (w * loss).backward()
    assert r.loss == pytest.approx(loss.item(), rel=1e-13)
    for k in e.param_names():
        np.testing.assert_allclose(r.grads[k], tp[k].grad.numpy(), rtol=1e-10, atol=1e-14)


# ------------------------------------------------ pure-Python brute force
def _py_forward_loss(kind, X, Wout, gamma, y, eps, mlp=None):
    """Loops over scalars only: the definitions written out once more."""
    N, h, V = len(X), len(X[0]), len(Wout)
    total = 0.0
    for n in range(N):
        s_in = list(X[n])
        if kind == O.EXIT_MLP:
            gm, Wg, Wu, Wd = mlp
            rx = 1.0 / math.sqrt(sum(t * t for t in s_in) / h + eps)
            u = [s_in[j] * rx * gm[j] for j in range(h)]
            I = len(Wg)
            act = []
            for i in range(I):
                g = sum(u[j] * Wg[i][j] for j in range(h))
                up = sum(u[j] * Wu[i][j] for j in range(h))
                act.append(g / (1.0 + math.exp(-g)) * up)
            s_in = [s_in[j] + sum(act[i] * Wd[j][i] for i in range(I)) for j in range(h)]
        if kind == O.EXIT_EMBEDDING:
            z = s_in
        else:
            r = 1.0 / math.sqrt(sum(t * t for t in s_in) / h + eps)
            z = [s_in[j] * r * gamma[j] for j in range(h)]
        logits = [sum(z[j] * Wout[v][j] for j in range(h)) for v in range(V)]
        mx = max(logits)
        lse = mx + math.log(sum(math.exp(l - mx) for l in logits))
        total += lse - logits[y[n]]
    return total / N


@pytest.mark.parametrize("kind", KINDS)
def test_pure_python_brute_force_loss(kind):
    rng = np.random.default_rng(40 + kind)
    N, h, V, I, eps = 3, 5, 7, 6, 1e-3
    e = rand_exit(kind, h, V, I, rng, eps=eps)
    x = rng.standard_normal((N, h))
    y = rng.integers(0, V, N)
    mlp = None
    if kind == O.EXIT_MLP:
        mlp = (e.gamma_mlp.tolist(), e.w_gate.tolist(), e.w_up.tolist(), e.w_down.tolist())
    ref = _py_forward_loss(kind, x.tolist(), e.w_out.tolist(),
                           None if e.gamma is None else e.gamma.tolist(), y.tolist(), eps, mlp)
    assert O.exit_step(e, x, y).loss == pytest.approx(ref, rel=1e-13)


# ---------------------------------------------------------- P6 identities
def test_gain_gradient_reordering_identity():
    """sum_n dZ*zhat == sum_v W_out * (G^T zhat): the reordering the GPU uses."""
    rng = np.random.default_rng(50)
    N, h, V = 11, 10, 23
    e = rand_exit(O.EXIT_NORM, h, V, 0, rng)
    x = rng.standard_normal((N, h))
    y = rng.integers(0, V, N)
    f = O.exit_forward(e, x)
    g = O.logit_grad(f["s"], y, np.full(N, 1.0 / N))
    plain = np.sum((g @ e.w_out) * f["z_hat"], axis=0)
    reordered = np.sum(e.w_out * (g.T @ f["z_hat"]), axis=0)
    np.testing.assert_allclose(plain, reordered, rtol=1e-12, atol=1e-16)
    np.testing.assert_allclose(O.exit_step(e, x, y).grads["gamma"], plain, rtol=1e-12)
    # dW_out = (G^T zhat) * gamma: column scale of the gain-free product
    np.testing.assert_allclose(O.exit_step(e, x, y).grads["w_out"],
                               (g.T @ f["z_hat"]) * e.gamma[None, :], rtol=1e-12)


# --------------------------------------------------- P7 RMSNorm invariance
def test_norm_exit_row_scale_invariance():
    rng = np.random.default_rng(60)
    N, h, V = 8, 16, 19
    e = rand_exit(O.EXIT_NORM, h, V, 0, rng, eps=0.0)
    x = rng.standard_normal((N, h))
    y = rng.integers(0, V, N)
    s = np.exp(2.0 * rng.standard_normal((N, 1)))
    a, b = O.exit_step(e, x, y), O.exit_step(e, x * s, y)
    assert a.loss == pytest.approx(b.loss, rel=1e-13)
    np.testing.assert_allclose(a.grads["w_out"], b.grads["w_out"], rtol=1e-11, atol=1e-15)
    e.eps = 1e-5        # eps breaks it, but only slightly for unit-RMS rows
    c, d = O.exit_step(e, x, y), O.exit_step(e, x * 2.0, y)
    assert c.loss != d.loss and abs(c.loss - d.loss) < 1e-4


# ------------------------------------------------ P8 MLP special case
def test_mlp_exit_with_zero_down_projection_is_norm_exit():
    rng = np.random.default_rng(70)
    N, h, V, I = 6, 12, 15, 20
    mlp = rand_exit(O.EXIT_MLP, h, V, I, rng)
    mlp.w_down[:] = 0.0
    norm = O.Exit(kind=O.EXIT_NORM, w_out=mlp.w_out, gamma=mlp.gamma, eps=mlp.eps)
    x = rng.standard_normal((N, h))
    y = rng.integers(0, V, N)
    a, b = O.exit_step(mlp, x, y), O.exit_step(norm, x, y)
    assert a.loss == b.loss
    np.testing.assert_array_equal(a.grads["w_out"], b.grads["w_out"])
    np.testing.assert_array_equal(a.grads["gamma"], b.grads["gamma"])
    assert np.all(a.grads["w_gate"] == 0) and np.all(a.grads["w_up"] == 0)
    assert np.all(a.grads["gamma_mlp"] == 0)
    assert np.any(a.grads["w_down"] != 0)       # the down projection still learns


# ------------------------------------------------- P9 multi-exit linearity
def test_multi_exit_linearity_and_independence():
    rng = np.random.default_rng(80)
    N, h, V, I = 7, 8, 13, 16
    e0, e1 = rand_exit(O.EXIT_NORM, h, V, I, rng), rand_exit(O.EXIT_MLP, h, V, I, rng)
    x0, x1 = rng.standard_normal((N, h)), rng.standard_normal((N, h))
    y = rng.integers(0, V, N)
    total, per = O.multi_exit_step([e0, e1], [x0, x1], y, [0.25, 0.5])
    s0, s1 = O.exit_step(e0, x0, y), O.exit_step(e1, x1, y)
    assert total == pytest.approx(0.25 * s0.loss + 0.5 * s1.loss, rel=1e-15)
    for k in e0.param_names():
        np.testing.assert_allclose(per[0].grads[k], 0.25 * s0.grads[k], rtol=1e-14, atol=1e-18)
    for k in e1.param_names():
        np.testing.assert_allclose(per[1].grads[k], 0.5 * s1.grads[k], rtol=1e-14, atol=1e-18)
    # identical (aliased) parameters and inputs give identical gradients
    total, per = O.multi_exit_step([e0, e0], [x0, x0], y, [1.0, 1.0])
    for k in e0.param_names():
        np.testing.assert_array_equal(per[0].grads[k], per[1].grads[k])


# ------------------------------------------------ P10 token weights
def test_token_weights():
    rng = np.random.default_rng(90)
    N, h, V, I = 10, 8, 11, 12
    e = rand_exit(O.EXIT_MLP, h, V, I, rng)
    x = rng.standard_normal((N, h))
    y = rng.integers(0, V, N)
    a, b = O.exit_step(e, x, y), O.exit_step(e, x, y, token_weights=np.ones(N))
    assert a.loss == b.loss
    m = rng.random(N)
    m[[1, 4]] = 0.0
    full = O.exit_step(e, x, y, token_weights=m)
    keep = m != 0
    sub = O.exit_step(e, x[keep], y[keep], token_weights=m[keep])
    # masked rows contribute nothing; the denominator stays N (reading R1)
    assert full.loss == pytest.approx(sub.loss * keep.sum() / N, rel=1e-13)
    for k in e.param_names():
        np.testing.assert_allclose(full.grads[k], sub.grads[k] * keep.sum() / N, rtol=1e-11, atol=1e-16)
    # linear in m
    m2 = rng.random(N)
    ab = O.exit_step(e, x, y, token_weights=m + 2 * m2)
    one, two = O.exit_step(e, x, y, token_weights=m), O.exit_step(e, x, y, token_weights=m2)
    assert ab.loss == pytest.approx(one.loss + 2 * two.loss, rel=1e-13)


# ---------------------------------------- dynamic token-wise loss weights
def test_dynamic_confidence_weights():
    rng = np.random.default_rng(100)
    N, h, V = 6, 8, 9
    e = rand_exit(O.EXIT_NORM, h, V, 0, rng)
    x = rng.standard_normal((N, h))
    y = rng.integers(0, V, N)
    r = O.exit_step(e, x, y, dynamic_weights=True)
    assert np.all(r.conf >= 1.0 / V) and np.all(r.conf <= 1.0)
    # confidence is the largest softmax entry
    p = np.exp(O.exit_forward(e, x)["s"] - r.lse[:, None])
    np.testing.assert_allclose(r.conf, p.max(axis=1), rtol=1e-14)
    # uniform logits: c = 1/V, so the loss is ln(V)/V
    e.w_out[:] = 0.0
    u = O.exit_step(e, x, y, dynamic_weights=True)
    np.testing.assert_allclose(u.conf, 1.0 / V, rtol=1e-15)
    assert u.loss == pytest.approx(math.log(V) / V, rel=1e-14)
    # the weights are detached: FD of the loss with c frozen at its value
    e = rand_exit(O.EXIT_NORM, h, V, 0, rng)
    r = O.exit_step(e, x, y, dynamic_weights=True)
    c = r.conf.copy()
    delta = 1e-6
    for idx in [(0, 0), (3, 5), (8, 7)]:
        old = e.w_out[idx]
        e.w_out[idx] = old + delta
        lp = O.exit_step(e, x, y, token_weights=c).loss
        e.w_out[idx] = old - delta
        lm = O.exit_step(e, x, y, token_weights=c).loss
        e.w_out[idx] = old
        assert abs((lp - lm) / (2 * delta) - r.grads["w_out"][idx]) < 1e-8


@pytest.mark.parametrize("kind", KINDS)
def test_dynamic_weights_times_token_weights(kind):
    """Reading R20: with caller token weights m, the dynamic weight of row n is
    m_n c_n (c detached).  Pinned by a closed form, masking and central
    finite differences of the loss with the product frozen."""
    rng = np.random.default_rng(105 + kind)
    N, h, V, I = 8, 8, 11, 12
    e = rand_exit(kind, h, V, I, rng)
    x = rng.standard_normal((N, h))
    y = rng.integers(0, V, N)
    m = rng.random(N) + 0.25
    m[[2, 5]] = 0.0
    # all-ones caller weights are the same as none
    a = O.exit_step(e, x, y, dynamic_weights=True)
    b = O.exit_step(e, x, y, token_weights=np.ones(N), dynamic_weights=True)
    assert a.loss == b.loss
    # uniform logits: c = 1/V for every row, so L = ln(V) mean(m) / V
    z = O.Exit(kind=kind, w_out=np.zeros((V, h)), gamma=e.gamma, gamma_mlp=e.gamma_mlp,
               w_gate=e.w_gate, w_up=e.w_up, w_down=e.w_down)
    u = O.exit_step(z, x, y, token_weights=m, dynamic_weights=True)
    assert u.loss == pytest.approx(math.log(V) * np.mean(m) / V, rel=1e-14)
    # masked rows contribute nothing (the denominator stays N)
    full = O.exit_step(e, x, y, 0.7, token_weights=m, dynamic_weights=True)
    keep = m != 0
    sub = O.exit_step(e, x[keep], y[keep], 0.7, token_weights=m[keep], dynamic_weights=True)
    assert full.loss == pytest.approx(sub.loss * keep.sum() / N, rel=1e-13)
    for k in e.param_names():
        np.testing.assert_allclose(full.grads[k], sub.grads[k] * keep.sum() / N, rtol=1e-11, atol=1e-16)
    # the loss is sum_n (m_n c_n) nll_n / N with the product held constant:
    # central differences of that loss give the gradients (times w = 0.7)
    frozen = m * full.conf
    ref = O.exit_step(e, x, y, token_weights=frozen)
    assert full.loss == pytest.approx(ref.loss, rel=1e-14)
    assert full.loss == pytest.approx(float(np.sum(frozen * full.row_loss)) / N, rel=1e-14)
    delta = 1e-6
    for name in e.param_names():
        p = getattr(e, name)
        for idx in [tuple(rng.integers(0, s) for s in p.shape) for _ in range(3)]:
            old = p[idx]
            p[idx] = old + delta
            lp = O.exit_step(e, x, y, token_weights=frozen).loss
            p[idx] = old - delta
            lm = O.exit_step(e, x, y, token_weights=frozen).loss
            p[idx] = old
            fd = 0.7 * (lp - lm) / (2 * delta)
            assert abs(fd - full.grads[name][idx]) <= 1e-7 * max(1.0, abs(fd)), (name, idx)


# ------------------------------------------------------------ structure
def test_chunking_does_not_change_results():
    rng = np.random.default_rng(110)
    N, h, V, I = 13, 8, 10, 12
    e = rand_exit(O.EXIT_MLP, h, V, I, rng)
    x = rng.standard_normal((N, h))
    y = rng.integers(0, V, N)
    a, b = O.exit_step(e, x, y, chunk=1024), O.exit_step(e, x, y, chunk=4)
    assert a.loss == pytest.approx(b.loss, rel=1e-14)
    for k in e.param_names():
        np.testing.assert_allclose(a.grads[k], b.grads[k], rtol=1e-12, atol=1e-16)


@pytest.mark.parametrize("dynamic", [False, True])
@pytest.mark.parametrize("kind", KINDS)
def test_sampled_outputs_match_full(kind, dynamic):
    rng = np.random.default_rng(120 + kind)
    N, h, V, I = 9, 8, 14, 12
    e = rand_exit(kind, h, V, I, rng)
    x = rng.standard_normal((N, h))
    y = rng.integers(0, V, N)
    m = rng.random(N) if dynamic else None
    full = O.exit_step(e, x, y, 0.5, token_weights=m, dynamic_weights=dynamic)
    v_rows, i_rows = np.array([0, 5, 13]), np.array([2, 11])
    smp = O.exit_step_sampled(e, x, y, 0.5, v_rows, i_rows, chunk=4, token_weights=m,
                              dynamic_weights=dynamic)
    assert float(smp["loss"]) == pytest.approx(full.loss, rel=1e-14)
    np.testing.assert_allclose(smp["w_out_rows"], full.grads["w_out"][v_rows], rtol=1e-12)
    if kind != O.EXIT_EMBEDDING:
        np.testing.assert_allclose(smp["gamma"], full.grads["gamma"], rtol=1e-12, atol=1e-16)
    if kind == O.EXIT_MLP:
        np.testing.assert_allclose(smp["gamma_mlp"], full.grads["gamma_mlp"], rtol=1e-12, atol=1e-16)
        np.testing.assert_allclose(smp["w_gate_rows"], full.grads["w_gate"][i_rows], rtol=1e-12)
        np.testing.assert_allclose(smp["w_up_rows"], full.grads["w_up"][i_rows], rtol=1e-12)
        np.testing.assert_allclose(smp["w_down_cols"], full.grads["w_down"][:, i_rows], rtol=1e-12)


def test_empty_batch_is_rejected():
    e = O.Exit(kind=O.EXIT_EMBEDDING, w_out=np.zeros((3, 2)))
    with pytest.raises(ValueError):
        O.exit_step(e, np.zeros((0, 2)), np.zeros(0, dtype=int))


def test_vocab_of_one_has_zero_loss_and_gradient():
    rng = np.random.default_rng(130)
    e = rand_exit(O.EXIT_NORM, 8, 1, 0, rng)
    r = O.exit_step(e, rng.standard_normal((4, 8)), np.zeros(4, dtype=int))
    assert r.loss == 0.0
    assert np.all(r.grads["w_out"] == 0) and np.all(r.grads["gamma"] == 0)


# --------------------------------------- statistics of the synthetic inputs
def test_tiny_workload_loss_near_expectation():
    """W_out ~ N(0, 0.02^2), unit-RMS rows: logits ~ N(0, 0.02^2 h), so
    E[loss] ~ ln V + 0.02^2 h / 2.  A sanity bound on the data, not parity."""
    b = W.make_batch(W.WORKLOADS["tiny_norm_f32"], seed=0)
    e = O.exits_from_batch(b)[0]
    r = O.exit_step(e, W.decode(b.hidden[0]), b.targets)
    expect = math.log(1024) + 0.02 ** 2 * 256 / 2
    assert abs(r.loss - expect) < 0.1


# ------------------------------------------------ LayerNorm flavour of Norm
def rand_layer_exit(kind, h, V, I, rng, bias=True, eps=1e-5):
    e = rand_exit(kind, h, V, I, rng, eps=eps)
    e.norm = "layer"
    if bias:
        e.beta = 0.3 * rng.standard_normal(h)
    return e


@pytest.mark.parametrize("kind,bias", [(O.EXIT_NORM, True), (O.EXIT_NORM, False), (O.EXIT_MLP, True)])
def test_layernorm_against_torch_autograd(kind, bias):
    rng = np.random.default_rng(70 + kind + 2 * bias)
    N, h, V, I, eps = 6, 16, 21, 20, 1e-5
    e = rand_layer_exit(kind, h, V, I, rng, bias=bias, eps=eps)
    x = rng.standard_normal((N, h)) + rng.standard_normal((N, 1)) * 2.0   # rows with offsets
    y = rng.integers(0, V, N)
    w = 0.6
    r = O.exit_step(e, x, y, w)
    tp = {k: torch.tensor(getattr(e, k), requires_grad=True) for k in e.param_names()}
    tx = torch.tensor(x)
    if kind == O.EXIT_MLP:
        u = F.layer_norm(tx, (h,), tp["gamma_mlp"], None, eps)
        a = F.silu(F.linear(u, tp["w_gate"])) * F.linear(u, tp["w_up"])
        s_in = tx + F.linear(a, tp["w_down"])
    else:
        s_in = tx
    z = F.layer_norm(s_in, (h,), tp["gamma"], tp.get("beta"), eps)
    loss = F.cross_entropy(F.linear(z, tp["w_out"]), torch.tensor(y), reduction="mean")
    (w * loss).backward()
    assert r.loss == pytest.approx(loss.item(), rel=1e-13)
    assert set(r.grads) == set(tp)
    for k in e.param_names():
        np.testing.assert_allclose(r.grads[k], tp[k].grad.numpy(), rtol=1e-10, atol=1e-14)


def test_layernorm_finite_differences():
    rng = np.random.default_rng(80)
    N, h, V = 5, 8, 13
    e = rand_layer_exit(O.EXIT_NORM, h, V, 0, rng)
    x = rng.standard_normal((N, h)) + 1.5
    y = rng.integers(0, V, N)
    r = O.exit_step(e, x, y, 0.7)
    for name in ("beta", "gamma"):
        p = getattr(e, name)
        for j in range(h):
            old = p[j]
            p[j] = old + 1e-6
            lp = loss_only(e, x, y, 0.7)
            p[j] = old - 1e-6
            lm = loss_only(e, x, y, 0.7)
            p[j] = old
            assert (lp - lm) / 2e-6 == pytest.approx(r.grads[name][j], rel=1e-6, abs=1e-10)


def test_layernorm_ignores_row_offsets_rmsnorm_does_not():
    rng = np.random.default_rng(81)
    N, h, V = 4, 12, 9
    x = rng.standard_normal((N, h))
    shift = rng.standard_normal((N, 1)) * 3.0
    y = rng.integers(0, V, N)
    e = rand_layer_exit(O.EXIT_NORM, h, V, 0, rng)
    assert O.exit_step(e, x + shift, y).loss == pytest.approx(O.exit_step(e, x, y).loss, rel=1e-9)
    e.norm = "rms"
    assert abs(O.exit_step(e, x + shift, y).loss - O.exit_step(e, x, y).loss) > 1e-3


def test_bias_gradient_reordering_identities():
    """With a bias: sum_n dZ = W_out^T (sum_n G) and dW_out = (G^T zhat) * gamma +
    outer(sum_n G, beta): the reorderings the GPU epilogue uses."""
    rng = np.random.default_rng(82)
    N, h, V = 11, 10, 23
    e = rand_layer_exit(O.EXIT_NORM, h, V, 0, rng)
    x = rng.standard_normal((N, h)) + 0.5
    y = rng.integers(0, V, N)
    f = O.exit_forward(e, x)
    g = O.logit_grad(f["s"], y, np.full(N, 1.0 / N))
    gsum = g.sum(axis=0)
    r = O.exit_step(e, x, y)
    np.testing.assert_allclose(r.grads["beta"], e.w_out.T @ gsum, rtol=1e-12, atol=1e-16)
    np.testing.assert_allclose(r.grads["w_out"], (g.T @ f["z_hat"]) * e.gamma[None, :] + np.outer(gsum, e.beta),
                               rtol=1e-12, atol=1e-16)
    np.testing.assert_allclose(r.grads["gamma"], np.sum(e.w_out * (g.T @ f["z_hat"]), axis=0), rtol=1e-12)


def test_layer_workload_recipe():
    w = W.custom(W.EXIT_NORM, 64, 128, 300, name="ln", norm="layer", bias=True)
    b = W.make_batch(w, 0)
    ex = O.exits_from_batch(b)[0]
    assert ex.norm == "layer" and ex.beta is not None and ex.beta.shape == (128,)
    x = W.decode(b.hidden[0])
    assert np.std(x.mean(axis=1)) > 0.5          # row offsets make centring matter
    w2 = W.custom(W.EXIT_NORM, 64, 128, 300, name="ln")
    assert O.exits_from_batch(W.make_batch(w2, 0))[0].beta is None
