"""GPU parity of the fused Adam update (ee_adam_update) against the fp64 oracle.

Bar (u = 2^-24, the fp32 unit roundoff; each bound is twice the worst-case
rounding of the fp32 formula):
  m: 4u (b1 |m_prev| + (1 - b1) |g|)  -- the two terms may cancel;
  v: 4u v  (all terms positive);
  master: a 4u s_m / D + 10u |step| + 2u |p|, with a = lr / (1 - b1^t),
     s_m the m bound's scale, D = sqrt(v_hat) + eps and step = a m / D;
  a bf16 parameter equals the device's own master rounded to nearest even,
  and lies within one bf16 ulp of the oracle's.
"""

import numpy as np
import pytest
import torch

from oracle import optim as OP
from paper_2402_00518_amd import binding as B

pytestmark = pytest.mark.gpu

# The ABI takes fp32 hyper-parameters; the oracle gets the same fp32 values.
f32 = lambda x: float(np.float32(x))
BETA1, BETA2, EPS = f32(OP.PAPER_BETA1), f32(OP.PAPER_BETA2), f32(OP.PAPER_EPS)


def say(msg):
    print(msg, flush=True)


def bf16_of(a32: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a32, dtype=np.float32)).to(torch.bfloat16)


class Case:
    """One parameter tensor with its optimizer state, on the device and as fp64 copies."""

    def __init__(self, rng, numel, dtype, with_master):
        self.numel, self.dtype, self.with_master = numel, dtype, with_master
        master = rng.normal(0.0, 0.02, numel).astype(np.float32)
        grad = (rng.normal(size=numel) * 10.0 ** rng.uniform(-5, -1, size=numel)).astype(np.float32)
        m = (rng.normal(size=numel) * 1e-3).astype(np.float32)
        v = (np.abs(rng.normal(size=numel)) * 1e-5).astype(np.float32)
        if dtype == B.EE_BF16:
            self.param = bf16_of(master).cuda()
            self.param_host = self.param.cpu().double().numpy()
        else:
            self.param = torch.from_numpy(master.copy()).cuda()
            self.param_host = master.astype(np.float64)
        self.master = torch.from_numpy(master.copy()).cuda() if with_master else None
        self.master_host = master.astype(np.float64) if with_master else None
        self.grad = torch.from_numpy(grad).cuda()
        self.m = torch.from_numpy(m).cuda()
        self.v = torch.from_numpy(v).cuda()
        self.grad_host, self.m_host, self.v_host = (grad.astype(np.float64), m.astype(np.float64),
                                                     v.astype(np.float64))

    def resync(self):
        """Take the device's state as the next update's inputs, so every update
        is compared from identical inputs (rounding does not accumulate into
        the comparison)."""
        self.param_host = self.param.cpu().double().numpy()
        if self.with_master:
            self.master_host = self.master.cpu().double().numpy()
        self.m_host = self.m.cpu().double().numpy()
        self.v_host = self.v.cpu().double().numpy()

    def desc(self):
        return B.adam_tensor(self.param, self.grad, self.m, self.v, master=self.master,
                             numel=self.numel, dtype=self.dtype)

    def oracle_update(self, step, lr):
        p0 = self.master_host if self.with_master else self.param_host
        p, mst, m, v = OP.mixed_precision_update(self.param_host, self.master_host, self.grad_host,
                                                 self.m_host, self.v_host, step, lr, BETA1, BETA2,
                                                 EPS, self.dtype == B.EE_BF16)
        # error-bound ingredients (fp64, from the oracle's own values)
        u = 2.0 ** -24
        a = lr / (1.0 - BETA1 ** step)
        s_m = BETA1 * np.abs(self.m_host) + (1.0 - BETA1) * np.abs(self.grad_host)
        D = np.sqrt(v / (1.0 - BETA2 ** step)) + EPS
        upd = a * np.abs(m) / D
        self.tol_m = 2 * 4 * u * s_m + 1e-38
        self.tol_v = 2 * 4 * u * v + 1e-38
        self.tol_p = 2 * (a * 4 * u * s_m / D + 10 * u * upd + 2 * u * np.abs(p0)) + 1e-38
        self.param_host, self.master_host, self.m_host, self.v_host = p, mst, m, v

    def check(self, lr, idx=None):
        sel = (lambda a: a) if idx is None else (lambda a: a[idx])
        m = sel(self.m.cpu().double().numpy())
        v = sel(self.v.cpu().double().numpy())
        def within(got, ref, tol, what):
            bad = np.abs(got - ref) > tol
            assert not bad.any(), (what, int(bad.sum()), got[bad][:4], ref[bad][:4], tol[bad][:4])

        within(m, sel(self.m_host), sel(self.tol_m), "exp_avg")
        within(v, sel(self.v_host), sel(self.tol_v), "exp_avg_sq")
        ref = sel(self.master_host if self.with_master else self.param_host)
        got_param = sel(self.param.cpu().double().numpy())
        if self.with_master:
            got = sel(self.master.cpu().double().numpy())
            within(got, ref, sel(self.tol_p), "master")
            if self.dtype == B.EE_BF16:
                np.testing.assert_array_equal(got_param, OP.round_to_bf16(got))
            else:
                np.testing.assert_array_equal(got_param, got)
        elif self.dtype == B.EE_F32:
            within(got_param, ref, sel(self.tol_p), "param")
        if self.dtype == B.EE_BF16:
            # Round-to-nearest moves each value by at most half a bf16 spacing,
            # so the two rounded parameters differ by at most the masters'
            # difference (bounded by tol_p) plus the spacing at the larger
            # magnitude (8 significant bits).
            big = np.maximum(np.abs(ref), np.abs(got_param)) + sel(self.tol_p)
            spacing = np.exp2(np.floor(np.log2(np.maximum(big, 1e-38))) - 7)
            gap = np.abs(got_param - sel(self.param_host))
            bad = gap > sel(self.tol_p) + spacing
            assert not bad.any(), ("bf16 param", got_param[bad][:4], sel(self.param_host)[bad][:4])


def run_update(cases, step, lr):
    B.ee_adam_update([c.desc() for c in cases], lr, BETA1, BETA2, EPS, step,
                     torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()


def test_ragged_tensors_over_two_launches():
    rng = np.random.default_rng(11)
    sizes = [1, 3, 4095, 4096, 4097, 10000, 70001, 8, 12345, 2]
    kinds = [(B.EE_BF16, True), (B.EE_F32, False), (B.EE_BF16, False)]
    cases = [Case(rng, n, *kinds[i % 3]) for i, n in enumerate(sizes)]
    say(f"case: adam ragged, {len(cases)} tensors, sizes {sizes}")
    lr = f32(1e-3)
    run_update(cases, 7, lr)
    for c in cases:
        c.oracle_update(7, lr)
        c.check(lr)


def test_three_updates_under_the_schedule():
    rng = np.random.default_rng(12)
    cases = [Case(rng, 50000, B.EE_BF16, True), Case(rng, 4096, B.EE_F32, False)]
    say("case: adam, three chained updates")
    for step in (1, 2, 3):
        lr = f32(B.ee_lr_schedule(step, 10, 0.2, 1e-3, 1e-4))
        for c in cases:
            g = (rng.normal(size=c.numel) * 1e-3).astype(np.float32)
            c.grad.copy_(torch.from_numpy(g))
            c.grad_host = g.astype(np.float64)
        run_update(cases, step, lr)
        for c in cases:
            c.oracle_update(step, lr)
            c.check(lr)
            c.resync()


def test_empty_and_zero_gradient():
    rng = np.random.default_rng(13)
    c = Case(rng, 5000, B.EE_BF16, True)
    c.grad.zero_()
    c.grad_host[:] = 0.0
    c.m.zero_(); c.m_host[:] = 0.0
    c.v.zero_(); c.v_host[:] = 0.0
    before = c.master.clone()
    say("case: adam, zero gradient at step 1")
    B.ee_adam_update([c.desc(), B.adam_tensor(c.param, c.grad, c.m, c.v, numel=0)], 1e-3, BETA1, BETA2,
                     EPS, 1, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert torch.equal(c.master, before)
    assert not c.m.any() and not c.v.any()


def test_full_size_output_matrix_sampled():
    # The 7B-shape output matrix (V = 32000, h = 4096): 131 M elements in one
    # tensor; compare 200k sampled elements.
    numel = 32000 * 4096
    rng = np.random.default_rng(14)
    say(f"case: adam full-size W_out, numel={numel}")
    c = Case(rng, numel, B.EE_BF16, True)
    lr = f32(1e-4)
    run_update([c], 400, lr)
    idx = np.unique(np.concatenate([rng.integers(0, numel, 200000), [0, numel - 1, numel // 2]]))
    for name in ("param_host", "master_host", "grad_host", "m_host", "v_host"):
        setattr(c, name, getattr(c, name)[idx])
    c.oracle_update(400, lr)
    # compare on the sampled indices only
    sampled = type("S", (), {})()
    sampled.m = c.m[torch.from_numpy(idx).cuda()]
    sampled.v = c.v[torch.from_numpy(idx).cuda()]
    sampled.param = c.param[torch.from_numpy(idx).cuda()]
    sampled.master = c.master[torch.from_numpy(idx).cuda()]
    c.m, c.v, c.param, c.master = sampled.m, sampled.v, sampled.param, sampled.master
    c.check(lr)
