"""Pins of the Adam / learning-rate oracle (oracle/optim.py) against closed
forms, the paper's schedule constants and independent library routines."""

import math

import numpy as np
import pytest
import torch

from oracle import optim as OP


def test_schedule_paper_constants():
    # Sec. 3 "Tuning": 40k iterations, 1% warmup to 1e-4, linear decay to 1e-5.
    T, f = OP.PAPER_ITERATIONS, OP.PAPER_WARMUP_FRACTION
    lr = lambda s: OP.lr_schedule(s, T, f, OP.PAPER_LR_MAX, OP.PAPER_LR_MIN)
    assert lr(1) == pytest.approx(1e-4 / 400, rel=1e-15)
    assert lr(200) == pytest.approx(0.5e-4, rel=1e-15)
    assert lr(400) == pytest.approx(1e-4, rel=1e-15)
    assert lr(20200) == pytest.approx(0.5 * (1e-4 + 1e-5), rel=1e-12)  # halfway through the decay
    assert lr(40000) == pytest.approx(1e-5, rel=1e-15)
    assert lr(50000) == 1e-5
    vals = [lr(s) for s in range(1, T + 1, 97)]
    peak = max(range(len(vals)), key=vals.__getitem__)
    assert all(a <= b for a, b in zip(vals[:peak], vals[1:peak + 1]))
    assert all(a >= b for a, b in zip(vals[peak:], vals[peak + 1:]))


def test_schedule_without_warmup():
    assert OP.lr_schedule(1, 10, 0.0, 1.0, 0.0) == pytest.approx(0.9)
    assert OP.lr_schedule(10, 10, 0.0, 1.0, 0.0) == 0.0


def test_first_step_closed_form():
    # m_hat_1 = g and v_hat_1 = g^2, so the first update is lr g / (|g| + eps).
    rng = np.random.default_rng(0)
    th, g = rng.normal(size=50), rng.normal(size=50) * 1e-3
    z = np.zeros(50)
    out, m, v = OP.adam_step(th, g, z, z, 1, lr=1e-4)
    np.testing.assert_allclose(out, th - 1e-4 * g / (np.abs(g) + 1e-5), rtol=0, atol=1e-18)
    np.testing.assert_allclose(m, 0.1 * g, rtol=1e-14)
    np.testing.assert_allclose(v, 0.05 * g * g, rtol=1e-14)


def test_constant_gradient_closed_form():
    # With a constant g: m_t = (1 - b1^t) g and v_t = (1 - b2^t) g^2, so every
    # bias-corrected update is again lr g / (|g| + eps).
    g = np.array([3e-3, -2e-4, 0.5, -7.0])
    th = np.array([0.1, -0.2, 0.3, 0.0])
    m = v = np.zeros(4)
    for t in range(1, 30):
        new, m, v = OP.adam_step(th, g, m, v, t, lr=1e-3)
        np.testing.assert_allclose(new, th - 1e-3 * g / (np.abs(g) + 1e-5), rtol=1e-12, atol=1e-18)
        np.testing.assert_allclose(m, (1 - 0.9 ** t) * g, rtol=1e-12)
        np.testing.assert_allclose(v, (1 - 0.95 ** t) * g * g, rtol=1e-12)
        th = new


def test_zero_gradient_first_step_is_identity():
    th = np.array([1.0, -2.0, 3.5])
    out, m, v = OP.adam_step(th, np.zeros(3), np.zeros(3), np.zeros(3), 1, lr=1.0)
    np.testing.assert_array_equal(out, th)
    assert not m.any() and not v.any()


def test_matches_torch_adam_over_a_schedule():
    # torch.optim.Adam (fp64, CPU) implements the same published update
    # independently; run 12 updates with the paper's betas/eps and a
    # schedule-driven learning rate.
    rng = np.random.default_rng(1)
    th0 = rng.normal(size=(7, 13))
    grads = [rng.normal(size=(7, 13)) * 10.0 ** rng.uniform(-6, 0) for _ in range(12)]
    p = torch.nn.Parameter(torch.tensor(th0, dtype=torch.float64))
    opt = torch.optim.Adam([p], lr=1.0, betas=(0.9, 0.95), eps=1e-5, weight_decay=0.0,
                           foreach=False, fused=False)
    th, m, v = th0.copy(), np.zeros_like(th0), np.zeros_like(th0)
    for t, g in enumerate(grads, start=1):
        lr = OP.lr_schedule(t, 20, 0.25, 1e-2, 1e-3)
        for group in opt.param_groups:
            group["lr"] = lr
        p.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        th, m, v = OP.adam_step(th, g, m, v, t, lr, 0.9, 0.95, 1e-5)
        np.testing.assert_allclose(th, p.detach().numpy(), rtol=1e-13, atol=1e-16)
        st = opt.state[p]
        np.testing.assert_allclose(m, st["exp_avg"].numpy(), rtol=1e-13, atol=1e-300)
        np.testing.assert_allclose(v, st["exp_avg_sq"].numpy(), rtol=1e-13, atol=1e-300)


def test_round_to_bf16_definition_and_torch():
    one = 1.0
    cases = {one: one, one + 2 ** -8: one, one + 3 * 2 ** -8: one + 2 ** -6,
             one + 2 ** -8 + 2 ** -20: one + 2 ** -7, -2.5: -2.5, 0.0: 0.0}
    for x, want in cases.items():
        assert OP.round_to_bf16(np.array([x]))[0] == want, x
    rng = np.random.default_rng(2)
    x = (rng.normal(size=4096) * 10.0 ** rng.uniform(-30, 30, size=4096)).astype(np.float32)
    want = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(OP.round_to_bf16(x), want)
    assert math.isnan(OP.round_to_bf16(np.array([np.nan]))[0])


def test_mixed_precision_update_paths():
    rng = np.random.default_rng(3)
    master = rng.normal(size=64).astype(np.float32).astype(np.float64)
    param = OP.round_to_bf16(master)
    g = rng.normal(size=64) * 1e-2
    m = rng.normal(size=64) * 1e-3
    v = np.abs(rng.normal(size=64)) * 1e-5
    p1, mst1, m1, v1 = OP.mixed_precision_update(param, master, g, m, v, 5, 1e-4, 0.9, 0.95, 1e-5, True)
    th, mm, vv = OP.adam_step(master, g, m, v, 5, 1e-4)
    np.testing.assert_array_equal(mst1, th.astype(np.float32).astype(np.float64))
    np.testing.assert_array_equal(p1, OP.round_to_bf16(mst1))
    # without a master the stored (bf16) parameter itself is the starting point
    p2, mst2, _, _ = OP.mixed_precision_update(param, None, g, m, v, 5, 1e-4, 0.9, 0.95, 1e-5, True)
    assert mst2 is None
    th2, _, _ = OP.adam_step(param, g, m, v, 5, 1e-4)
    np.testing.assert_array_equal(p2, OP.round_to_bf16(th2.astype(np.float32)))
