"""The C ABI without a GPU: the library loads, exports every declared symbol,
and rejects bad arguments before anything is enqueued.

Pointers here are fake device addresses: validation only compares and
aligns them, it never dereferences them, and no call reaches a HIP launch.
"""

import ctypes
import os
import re

import pytest

from paper_2402_00518_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ee_tuning.h")

pytestmark = pytest.mark.skipif(not os.path.exists(B.LIB_PATH),
                                reason="libeetune.so not built (run __graft_entry__.build())")

GB = 1 << 30


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ee_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert set(names) == set(B.EXPORTS)
    L = B.lib()
    for n in names:
        assert hasattr(L, n), n
        assert ctypes.cast(getattr(L, n), ctypes.c_void_p).value


def test_version_and_status_strings():
    assert B.ee_abi_version() == B.EE_ABI_VERSION == 2
    for s in range(10):
        assert B.ee_status_string(s)
    assert "unknown" in B.ee_status_string(99)


def fake_exit(kind=B.EE_EXIT_NORM, dtype=B.EE_BF16, h=256, V=1000, I=0, base=0x10_0000_0000):
    """Parameters at distinct, far-apart fake addresses."""
    return B.make_exit(kind, dtype, h, V, I if kind == B.EE_EXIT_MLP else 0, 1e-5,
                       w_out=base, gamma=base + GB, gamma_mlp=base + 2 * GB,
                       w_gate=base + 3 * GB, w_up=base + 4 * GB, w_down=base + 5 * GB)


def fake_grads(base=0x20_0000_0000):
    return B.make_grads(base, base + GB, base + 2 * GB, base + 3 * GB, base + 4 * GB, base + 5 * GB)


X = 0x30_0000_0000
Y = 0x31_0000_0000
LOSS = 0x32_0000_0000
WS = 0x40_0000_0000
N = 300


def fwd(e, **kw):
    a = dict(hidden=X, targets=Y, token_w=None, n_tokens=N, exit_weight=1.0, flags=0, ws=WS,
             ws_bytes=1 << 32, loss=LOSS, row_loss=None, stream=None)
    a.update(kw)
    return B.ee_head_forward_loss(e, check=False, **a)


def expect(status, code, needle):
    assert status == code, (status, B.ee_last_error())
    assert needle in B.ee_last_error(), B.ee_last_error()


def test_workspace_bytes():
    e = fake_exit()
    a = B.ee_workspace_bytes([e], 100)
    b = B.ee_workspace_bytes([e], 5000)
    assert 0 < a < b
    m = fake_exit(B.EE_EXIT_MLP, I=512)
    assert B.ee_workspace_bytes([e, m], 100) == B.ee_workspace_bytes([m], 100) > a
    # the dominant region is the [V][N_pad] logits/seed buffer
    assert b >= 1000 * 5056 * 2
    with pytest.raises(B.EEError, match="hidden"):
        B.ee_workspace_bytes([fake_exit(h=100)], 10)
    assert B.lib().ee_workspace_bytes(0, (B.EeExit * 1)(), 10) == 0


@pytest.mark.parametrize("field,value,code,needle", [
    ("hidden", 100, B.EE_ERR_SHAPE, "hidden"),
    ("hidden", 0, B.EE_ERR_SHAPE, "hidden"),
    ("vocab", 0, B.EE_ERR_SHAPE, "vocab"),
    ("vocab", (1 << 20) + 1, B.EE_ERR_SHAPE, "vocab"),
    ("dtype", 7, B.EE_ERR_DTYPE, "dtype"),
    ("kind", B.EE_EXIT_LAYER, B.EE_ERR_UNSUPPORTED, "Layer"),
    ("kind", 9, B.EE_ERR_UNSUPPORTED, "kind"),
    ("intermediate", 64, B.EE_ERR_SHAPE, "intermediate"),
    ("rms_eps", -1.0, B.EE_ERR_SHAPE, "rms_eps"),
    ("rms_eps", float("nan"), B.EE_ERR_SHAPE, "rms_eps"),
    ("norm", 5, B.EE_ERR_UNSUPPORTED, "norm"),
    ("beta", 0x10_8000_0000, B.EE_ERR_SHAPE, "beta"),            # a bias without LayerNorm
    ("w_out", None, B.EE_ERR_NULL, "w_out"),
    ("gamma", None, B.EE_ERR_NULL, "gamma"),
    ("w_out", 0x10_0000_0008, B.EE_ERR_ALIGN, "w_out"),
])
def test_forward_rejects_bad_exit(field, value, code, needle):
    e = fake_exit()
    setattr(e, field, value)
    expect(fwd(e), code, needle)


def test_layernorm_is_for_norm_exits_and_needs_a_bias_gradient():
    e = fake_exit(B.EE_EXIT_MLP, I=512)
    e.norm = B.EE_NORM_LAYER
    expect(fwd(e), B.EE_ERR_UNSUPPORTED, "LayerNorm")
    e = fake_exit(B.EE_EXIT_EMBEDDING)
    e.norm = B.EE_NORM_LAYER
    expect(fwd(e), B.EE_ERR_UNSUPPORTED, "LayerNorm")
    e = fake_exit()
    e.norm = B.EE_NORM_LAYER
    e.beta = 0x10_8000_0008
    expect(fwd(e), B.EE_ERR_ALIGN, "beta")
    e.beta = 0x10_8000_0000
    expect(fwd(e, ws_bytes=16), B.EE_ERR_WORKSPACE, "workspace")        # a valid LayerNorm exit
    assert B.ee_workspace_bytes([e], 100) > B.ee_workspace_bytes([fake_exit()], 100)
    g = fake_grads()
    g.d_beta = None
    st = B.ee_head_backward(e, 100, 0x60_0000_0000, 1 << 32, g, 0, None, check=False)
    expect(st, B.EE_ERR_NULL, "d_beta")


def test_mlp_exit_needs_its_weights():
    e = fake_exit(B.EE_EXIT_MLP, I=512)
    e.w_down = None
    expect(fwd(e), B.EE_ERR_NULL, "w_down")
    e = fake_exit(B.EE_EXIT_MLP, I=500)
    expect(fwd(e), B.EE_ERR_SHAPE, "intermediate")


def test_embedding_exit_needs_no_gain():
    e = fake_exit(B.EE_EXIT_EMBEDDING)
    e.gamma = None
    expect(fwd(e, ws_bytes=16), B.EE_ERR_WORKSPACE, "workspace")  # got past the exit checks


@pytest.mark.parametrize("kw,code,needle", [
    (dict(hidden=None), B.EE_ERR_NULL, "hidden"),
    (dict(targets=None), B.EE_ERR_NULL, "targets"),
    (dict(loss=None), B.EE_ERR_NULL, "loss"),
    (dict(ws=None), B.EE_ERR_NULL, "workspace"),
    (dict(hidden=X + 4), B.EE_ERR_ALIGN, "hidden"),
    (dict(token_w=Y + 2 * GB + 8), B.EE_ERR_ALIGN, "token_w"),
    (dict(n_tokens=0), B.EE_ERR_SHAPE, "n_tokens"),
    (dict(n_tokens=-5), B.EE_ERR_SHAPE, "n_tokens"),
    (dict(n_tokens=(1 << 20) + 1), B.EE_ERR_SHAPE, "n_tokens"),
    (dict(flags=2), B.EE_ERR_UNSUPPORTED, "flags"),
    (dict(exit_weight=float("inf")), B.EE_ERR_SHAPE, "exit_weight"),
    (dict(ws_bytes=1000), B.EE_ERR_WORKSPACE, "workspace"),
    (dict(loss=WS + 1024), B.EE_ERR_ALIAS, "loss"),
    (dict(row_loss=X + 64), B.EE_ERR_ALIAS, "hidden"),
    (dict(loss=0x10_0000_0000 + 4096), B.EE_ERR_ALIAS, "w_out"),
])
def test_forward_rejects_bad_arguments(kw, code, needle):
    expect(fwd(fake_exit(), **kw), code, needle)


def bwd(e, g, **kw):
    a = dict(n_tokens=N, ws=WS, ws_bytes=1 << 32, grads=g, accumulate=0, stream=None)
    a.update(kw)
    return B.ee_head_backward(e, check=False, **a)


def test_backward_rejects_bad_arguments():
    e, g = fake_exit(), fake_grads()
    g2 = fake_grads()
    g2.d_gamma = None
    expect(bwd(e, g2), B.EE_ERR_NULL, "d_gamma")
    expect(bwd(e, g, accumulate=2), B.EE_ERR_SHAPE, "accumulate")
    expect(bwd(e, g, ws_bytes=100), B.EE_ERR_WORKSPACE, "workspace")
    g3 = fake_grads()
    g3.d_gamma = g3.d_w_out + 1024            # inside d_w_out
    expect(bwd(e, g3), B.EE_ERR_ALIAS, "d_gamma")
    g4 = fake_grads()
    g4.d_w_out = e.w_out                     # a gradient written over its parameter
    expect(bwd(e, g4), B.EE_ERR_ALIAS, "w_out")
    g5 = fake_grads()
    g5.d_w_out = WS + 4096                   # over the workspace
    expect(bwd(e, g5), B.EE_ERR_ALIAS, "workspace")
    g6 = fake_grads()
    g6.d_w_out += 4
    expect(bwd(e, g6), B.EE_ERR_ALIGN, "d_w_out")
    m = fake_exit(B.EE_EXIT_MLP, I=512)
    g7 = fake_grads()
    g7.d_w_up = None
    expect(bwd(m, g7), B.EE_ERR_NULL, "d_w_up")


def step(exits, grads, **kw):
    a = dict(hidden=[X + i * GB for i in range(len(exits))], targets=Y, token_w=None, n_tokens=N,
             exit_weights=[1.0] * len(exits), flags=0, grads=grads, accumulate=0, ws=WS,
             ws_bytes=1 << 32, loss_total=LOSS, loss_per_exit=LOSS + 256, stream=None)
    a.update(kw)
    return B.ee_multi_exit_step(exits, check=False, **a)


def test_multi_exit_step_rejects_bad_arguments():
    e0, e1 = fake_exit(), fake_exit(base=0x50_0000_0000)
    g0, g1 = fake_grads(), fake_grads(0x60_0000_0000)
    assert B.lib().ee_multi_exit_step(0, None, None, None, None, 1, None, 0, None, 0, None, 0,
                                      None, None, None) == B.EE_ERR_SHAPE
    e1.vocab = 999
    expect(step([e0, e1], [g0, g1]), B.EE_ERR_SHAPE, "vocabulary")
    e1 = fake_exit(base=0x50_0000_0000, dtype=B.EE_F32)
    expect(step([e0, e1], [g0, g1]), B.EE_ERR_DTYPE, "dtype")
    e1 = fake_exit(base=0x50_0000_0000)
    expect(step([e0, e1], [g0, g0]), B.EE_ERR_ALIAS, "d_w_out")       # shared gradient buffers
    expect(step([e0, e1], [g0, g1], exit_weights=[1.0, float("nan")]), B.EE_ERR_SHAPE, "exit_weights")
    expect(step([e0, e1], [g0, g1], loss_per_exit=LOSS), B.EE_ERR_ALIAS, "loss")
    expect(step([e0, e1], [g0, g1], ws_bytes=4096), B.EE_ERR_WORKSPACE, "workspace")
    expect(step([e0, e1], [g0, g1], hidden=[X, None]), B.EE_ERR_NULL, "hidden")


def test_check_device_error_validates_before_touching_the_device():
    assert B.ee_check_device_error(None, 1 << 20, None, check=False) == B.EE_ERR_NULL
    assert B.ee_check_device_error(WS, 16, None, check=False) == B.EE_ERR_WORKSPACE


def test_missing_library_fails_loudly(tmp_path, monkeypatch):
    monkeypatch.setattr(B, "_lib", None)
    monkeypatch.setattr(B, "LIB_PATH", str(tmp_path / "libeetune.so"))
    with pytest.raises(RuntimeError, match="missing"):
        B.lib()


# ------------------------------------------------------------ Adam update
def fake_adam(i=0, numel=1000, dtype=B.EE_BF16, master=True):
    base = 0x40_0000_0000 + i * 8 * GB
    return B.adam_tensor(param=base, grad=base + GB, exp_avg=base + 2 * GB, exp_avg_sq=base + 3 * GB,
                         master=(base + 4 * GB) if master else None, numel=numel, dtype=dtype)


def adam_status(tensors, lr=1e-4, b1=0.9, b2=0.95, eps=1e-5, step=1):
    return B.ee_adam_update(tensors, lr, b1, b2, eps, step, None, check=False)


def test_adam_nothing_to_do_is_ok():
    assert adam_status([]) == B.EE_OK
    assert adam_status([fake_adam(numel=0), fake_adam(1, numel=0)]) == B.EE_OK


@pytest.mark.parametrize("kw,code,needle", [
    (dict(lr=float("nan")), B.EE_ERR_SHAPE, "lr"),
    (dict(b1=1.0), B.EE_ERR_SHAPE, "beta1"),
    (dict(b2=-0.1), B.EE_ERR_SHAPE, "beta1"),
    (dict(eps=-1.0), B.EE_ERR_SHAPE, "eps"),
    (dict(step=0), B.EE_ERR_SHAPE, "step"),
])
def test_adam_rejects_bad_hyperparameters(kw, code, needle):
    assert adam_status([fake_adam()], **kw) == code
    assert needle in B.ee_last_error()


def test_adam_rejects_bad_tensors():
    t = fake_adam(); t.param = None
    assert adam_status([t]) == B.EE_ERR_NULL and "param" in B.ee_last_error()
    t = fake_adam(); t.grad = 0x40_0000_0008
    assert adam_status([t]) == B.EE_ERR_ALIGN and "grad" in B.ee_last_error()
    t = fake_adam(); t.master = 0x40_0000_0004
    assert adam_status([t]) == B.EE_ERR_ALIGN
    t = fake_adam(); t.dtype = 7
    assert adam_status([t]) == B.EE_ERR_DTYPE
    t = fake_adam(); t.numel = -1
    assert adam_status([t]) == B.EE_ERR_SHAPE
    t = fake_adam(); t.reserved = 1
    assert adam_status([t]) == B.EE_ERR_SHAPE


def test_adam_rejects_aliasing():
    t = fake_adam(); t.exp_avg_sq = t.exp_avg + 512       # m and v overlap
    assert adam_status([t]) == B.EE_ERR_ALIAS
    t = fake_adam(); t.grad = t.param                     # written param over the gradient
    assert adam_status([t]) == B.EE_ERR_ALIAS
    a, b = fake_adam(0), fake_adam(1)
    b.master = a.master + 16                              # two tensors share a master
    assert adam_status([a, b]) == B.EE_ERR_ALIAS
    a, b = fake_adam(0), fake_adam(1)
    b.grad = a.grad                                        # shared read-only gradient is fine for validation
    b.param = a.param + 1024                               # but overlapping params (2000 bytes each) are not
    assert adam_status([a, b]) == B.EE_ERR_ALIAS


def test_lr_schedule_matches_the_oracle():
    from oracle import optim as OP
    for T, f, hi, lo in ((40000, 0.01, 1e-4, 1e-5), (10, 0.0, 1.0, 0.0), (37, 0.3, 2.0, 0.5)):
        for s in sorted({1, 2, int(f * T), int(f * T) + 1, T // 2, T - 1, T, T + 3}):
            if s < 1:
                continue
            assert B.ee_lr_schedule(s, T, f, hi, lo) == pytest.approx(OP.lr_schedule(s, T, f, hi, lo),
                                                                      rel=1e-15, abs=1e-300)
    import math
    assert math.isnan(B.ee_lr_schedule(0, 10, 0.1, 1.0, 0.0))
    assert math.isnan(B.ee_lr_schedule(1, 10, 1.0, 1.0, 0.0))


# ------------------------------------------------------------ decode decision
def decide_status(e, n=4, threshold=0.5, token=0x50_0000_0000, conf=0x51_0000_0000, flag=0x52_0000_0000,
                  ws=0x60_0000_0000, ws_bytes=1 << 32, hidden=X):
    return B.ee_exit_decide(e, hidden, n, threshold, token, conf, flag, ws, ws_bytes, None, check=False)


def test_decode_workspace_bytes():
    e = fake_exit()
    a, b = B.ee_decode_workspace_bytes(e, 1), B.ee_decode_workspace_bytes(e, 64)
    assert 0 < a < b
    m = fake_exit(kind=B.EE_EXIT_MLP, I=128)
    assert B.ee_decode_workspace_bytes(m, 8) > B.ee_decode_workspace_bytes(fake_exit(), 8)
    with pytest.raises(B.EEError):
        B.ee_decode_workspace_bytes(e, 0)


def test_decide_rejects_bad_arguments():
    e = fake_exit()
    assert decide_status(e, n=0) == B.EE_ERR_SHAPE
    assert decide_status(e, threshold=float("nan")) == B.EE_ERR_SHAPE
    assert decide_status(e, token=None) == B.EE_ERR_NULL
    assert decide_status(e, conf=0x51_0000_0004) == B.EE_ERR_ALIGN
    assert decide_status(e, ws_bytes=16) == B.EE_ERR_WORKSPACE
    assert decide_status(e, flag=0x50_0000_0000) == B.EE_ERR_ALIAS          # flag over token
    assert decide_status(e, token=X) == B.EE_ERR_ALIAS                       # output over the hidden states
    assert decide_status(e, ws=0x10_0000_0000) == B.EE_ERR_ALIAS             # workspace over W_out
    bad = fake_exit(); bad.kind = B.EE_EXIT_LAYER
    assert decide_status(bad) == B.EE_ERR_UNSUPPORTED


def static_status(e, n=4, threshold=0.5, token=0x50_0000_0000, conf=0x51_0000_0000, flag=0x52_0000_0000,
                  hidden=X):
    return B.ee_exit_decide_static(e, hidden, n, threshold, token, conf, flag, None, check=False)


def test_decide_static_rejects_before_touching_the_device():
    """The entry point without a workspace validates like ee_exit_decide and
    refuses calls whose workspace would not fit its fixed array; all of this
    happens before it looks up the array or enqueues anything."""
    e = fake_exit(h=8192, V=32000)
    fit = max(n for n in range(1, 4096) if B.ee_decode_workspace_bytes(e, n) <= B.EE_STATIC_SCRATCH_BYTES)
    assert fit >= 1000                                        # about 1100 rows of a 70B-shaped Norm exit
    expect(static_status(e, n=fit + 1), B.EE_ERR_WORKSPACE, "fixed")
    assert static_status(e, n=0) == B.EE_ERR_SHAPE
    assert static_status(e, threshold=float("nan")) == B.EE_ERR_SHAPE
    assert static_status(e, token=None) == B.EE_ERR_NULL
    assert static_status(e, conf=0x51_0000_0004) == B.EE_ERR_ALIGN
    assert static_status(e, flag=0x50_0000_0000) == B.EE_ERR_ALIAS         # flag over token
    assert static_status(e, token=X) == B.EE_ERR_ALIAS                      # output over the hidden states
    bad = fake_exit(); bad.kind = B.EE_EXIT_LAYER
    assert static_status(bad) == B.EE_ERR_UNSUPPORTED


def test_mlp_exit_hidden_limit():
    e = fake_exit(B.EE_EXIT_MLP, h=8256, I=512)
    expect(fwd(e), B.EE_ERR_SHAPE, "MLP exit needs hidden")
