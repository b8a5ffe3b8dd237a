"""ctypes binding of libeetune.so: the C ABI of include/ee_tuning.h, same names.

Argument marshalling only.  Every step of the exit-head path runs in the HIP
kernels behind the library; there is no Python or CPU fallback.  Pointer
arguments accept torch tensors (their data_ptr()), plain integers or None.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libeetune.so")

EE_OK = 0
EE_ERR_NULL = 1
EE_ERR_SHAPE = 2
EE_ERR_DTYPE = 3
EE_ERR_ALIGN = 4
EE_ERR_WORKSPACE = 5
EE_ERR_ALIAS = 6
EE_ERR_UNSUPPORTED = 7
EE_ERR_TARGET = 8
EE_ERR_HIP = 9

EE_F32 = 0
EE_BF16 = 1

EE_EXIT_EMBEDDING = 0
EE_EXIT_NORM = 1
EE_EXIT_MLP = 2
EE_EXIT_LAYER = 3

EE_FLAG_DYNAMIC_TOKEN_WEIGHTS = 1

EE_NORM_RMS = 0
EE_NORM_LAYER = 1

EE_ABI_VERSION = 2

# Every symbol include/ee_tuning.h declares.
EXPORTS = (
    "ee_workspace_bytes", "ee_head_forward_loss", "ee_head_backward",
    "ee_multi_exit_step", "ee_check_device_error", "ee_status_string",
    "ee_last_error", "ee_abi_version", "ee_profile_start", "ee_profile_stop",
    "ee_adam_update", "ee_lr_schedule", "ee_decode_workspace_bytes", "ee_exit_decide",
    "ee_exit_decide_static",
)
# Size of the fixed workspace array of ee_exit_decide_static, per GPU.
EE_STATIC_SCRATCH_BYTES = 32 << 20


class EeExit(ctypes.Structure):
    _fields_ = [
        ("kind", ctypes.c_int32), ("dtype", ctypes.c_int32),
        ("hidden", ctypes.c_int64), ("vocab", ctypes.c_int64),
        ("intermediate", ctypes.c_int64), ("rms_eps", ctypes.c_float),
        ("norm", ctypes.c_int32),
        ("w_out", ctypes.c_void_p), ("gamma", ctypes.c_void_p),
        ("gamma_mlp", ctypes.c_void_p), ("w_gate", ctypes.c_void_p),
        ("w_up", ctypes.c_void_p), ("w_down", ctypes.c_void_p),
        ("beta", ctypes.c_void_p),
    ]


class EeExitGrads(ctypes.Structure):
    _fields_ = [
        ("d_w_out", ctypes.c_void_p), ("d_gamma", ctypes.c_void_p),
        ("d_gamma_mlp", ctypes.c_void_p), ("d_w_gate", ctypes.c_void_p),
        ("d_w_up", ctypes.c_void_p), ("d_w_down", ctypes.c_void_p),
        ("d_beta", ctypes.c_void_p),
    ]


class EeAdamTensor(ctypes.Structure):
    _fields_ = [
        ("param", ctypes.c_void_p), ("master", ctypes.c_void_p), ("grad", ctypes.c_void_p),
        ("exp_avg", ctypes.c_void_p), ("exp_avg_sq", ctypes.c_void_p),
        ("numel", ctypes.c_int64), ("dtype", ctypes.c_int32), ("reserved", ctypes.c_int32),
    ]


class EeKernelTime(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char_p), ("launches", ctypes.c_int32),
                ("total_ms", ctypes.c_double)]


class EEError(RuntimeError):
    def __init__(self, status: int, func: str, detail: str):
        super().__init__(f"{func} -> {status} ({status_string(status)}): {detail}")
        self.status = status


_lib = None


def lib() -> ctypes.CDLL:
    """Load libeetune.so once.  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build the HIP extension first "
                "(python -m paper_2402_00518_amd.build)")
        L = ctypes.CDLL(LIB_PATH)
        vp, i64, f32, u32, i32 = (ctypes.c_void_p, ctypes.c_int64, ctypes.c_float,
                                  ctypes.c_uint32, ctypes.c_int)
        P = ctypes.POINTER
        L.ee_workspace_bytes.argtypes = [i32, P(EeExit), i64]
        L.ee_workspace_bytes.restype = ctypes.c_size_t
        L.ee_head_forward_loss.argtypes = [P(EeExit), vp, vp, vp, i64, f32, u32, vp,
                                           ctypes.c_size_t, vp, vp, vp]
        L.ee_head_forward_loss.restype = i32
        L.ee_head_backward.argtypes = [P(EeExit), i64, vp, ctypes.c_size_t,
                                       P(EeExitGrads), i32, vp]
        L.ee_head_backward.restype = i32
        L.ee_multi_exit_step.argtypes = [i32, P(EeExit), P(vp), vp, vp, i64, P(f32), u32,
                                         P(EeExitGrads), i32, vp, ctypes.c_size_t, vp, vp, vp]
        L.ee_multi_exit_step.restype = i32
        L.ee_check_device_error.argtypes = [vp, ctypes.c_size_t, vp]
        L.ee_check_device_error.restype = i32
        L.ee_status_string.argtypes = [i32]
        L.ee_status_string.restype = ctypes.c_char_p
        L.ee_last_error.argtypes = []
        L.ee_last_error.restype = ctypes.c_char_p
        L.ee_abi_version.argtypes = []
        L.ee_abi_version.restype = i32
        L.ee_profile_start.argtypes = []
        L.ee_profile_start.restype = i32
        L.ee_profile_stop.argtypes = [P(EeKernelTime), i32]
        L.ee_profile_stop.restype = i32
        L.ee_adam_update.argtypes = [i32, P(EeAdamTensor), f32, f32, f32, f32, i64, vp]
        L.ee_adam_update.restype = i32
        L.ee_lr_schedule.argtypes = [i64, i64, ctypes.c_double, ctypes.c_double, ctypes.c_double]
        L.ee_lr_schedule.restype = ctypes.c_double
        L.ee_decode_workspace_bytes.argtypes = [P(EeExit), i64]
        L.ee_decode_workspace_bytes.restype = ctypes.c_size_t
        L.ee_exit_decide.argtypes = [P(EeExit), vp, i64, f32, vp, vp, vp, vp, ctypes.c_size_t, vp]
        L.ee_exit_decide.restype = i32
        L.ee_exit_decide_static.argtypes = [P(EeExit), vp, i64, f32, vp, vp, vp, vp]
        L.ee_exit_decide_static.restype = i32
        _lib = L
    return _lib


def ptr(x) -> Optional[int]:
    """Device address of a tensor, an integer address, or None for NULL."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def status_string(s: int) -> str:
    return lib().ee_status_string(s).decode()


def ee_status_string(s: int) -> str:
    return status_string(s)


def ee_last_error() -> str:
    return lib().ee_last_error().decode()


def ee_abi_version() -> int:
    return lib().ee_abi_version()


def _check(status: int, func: str) -> int:
    if status != EE_OK:
        raise EEError(status, func, ee_last_error())
    return status


def _exits_array(exits: Sequence[EeExit]):
    arr = (EeExit * len(exits))()
    for i, e in enumerate(exits):
        arr[i] = e
    return arr


def ee_workspace_bytes(exits: Sequence[EeExit], n_tokens: int) -> int:
    n = lib().ee_workspace_bytes(len(exits), _exits_array(exits), n_tokens)
    if n == 0:
        raise EEError(EE_ERR_SHAPE, "ee_workspace_bytes", ee_last_error())
    return n


def ee_head_forward_loss(e: EeExit, hidden, targets, token_w, n_tokens: int, exit_weight: float,
                         flags: int, ws, ws_bytes: int, loss, row_loss, stream, check=True) -> int:
    s = lib().ee_head_forward_loss(ctypes.byref(e), ptr(hidden), ptr(targets), ptr(token_w),
                                   n_tokens, exit_weight, flags, ptr(ws), ws_bytes, ptr(loss),
                                   ptr(row_loss), stream)
    return _check(s, "ee_head_forward_loss") if check else s


def ee_head_backward(e: EeExit, n_tokens: int, ws, ws_bytes: int, grads: EeExitGrads,
                     accumulate: int, stream, check=True) -> int:
    s = lib().ee_head_backward(ctypes.byref(e), n_tokens, ptr(ws), ws_bytes,
                               ctypes.byref(grads), accumulate, stream)
    return _check(s, "ee_head_backward") if check else s


def ee_multi_exit_step(exits: Sequence[EeExit], hidden: Sequence, targets, token_w, n_tokens: int,
                       exit_weights: Sequence[float], flags: int, grads: Sequence[EeExitGrads],
                       accumulate: int, ws, ws_bytes: int, loss_total, loss_per_exit, stream,
                       check=True) -> int:
    ne = len(exits)
    hs = (ctypes.c_void_p * ne)(*[ptr(h) for h in hidden])
    ws_arr = (ctypes.c_float * ne)(*exit_weights)
    gs = (EeExitGrads * ne)()
    for i, g in enumerate(grads):
        gs[i] = g
    s = lib().ee_multi_exit_step(ne, _exits_array(exits), hs, ptr(targets), ptr(token_w), n_tokens,
                                 ws_arr, flags, gs, accumulate, ptr(ws), ws_bytes, ptr(loss_total),
                                 ptr(loss_per_exit), stream)
    return _check(s, "ee_multi_exit_step") if check else s


def ee_check_device_error(ws, ws_bytes: int, stream, check=True) -> int:
    s = lib().ee_check_device_error(ptr(ws), ws_bytes, stream)
    return _check(s, "ee_check_device_error") if check else s


def ee_profile_start() -> None:
    _check(lib().ee_profile_start(), "ee_profile_start")


def ee_profile_stop(capacity: int = 64) -> dict:
    """{kernel name: (launches, total milliseconds)} since ee_profile_start()."""
    arr = (EeKernelTime * capacity)()
    n = lib().ee_profile_stop(arr, capacity)
    if n < 0:
        raise EEError(EE_ERR_HIP, "ee_profile_stop", ee_last_error())
    return {arr[i].name.decode(): (arr[i].launches, arr[i].total_ms) for i in range(n)}


# ----------------------------------------------------------- construction
def make_exit(kind: int, dtype: int, hidden: int, vocab: int, intermediate: int = 0,
              rms_eps: float = 1e-5, w_out=None, gamma=None, gamma_mlp=None, w_gate=None,
              w_up=None, w_down=None, beta=None, norm: int = EE_NORM_RMS) -> EeExit:
    return EeExit(kind, dtype, hidden, vocab, intermediate, rms_eps, norm, ptr(w_out), ptr(gamma),
                  ptr(gamma_mlp), ptr(w_gate), ptr(w_up), ptr(w_down), ptr(beta))


def make_grads(d_w_out=None, d_gamma=None, d_gamma_mlp=None, d_w_gate=None, d_w_up=None,
               d_w_down=None, d_beta=None) -> EeExitGrads:
    return EeExitGrads(ptr(d_w_out), ptr(d_gamma), ptr(d_gamma_mlp), ptr(d_w_gate), ptr(d_w_up),
                       ptr(d_w_down), ptr(d_beta))


def adam_tensor(param, grad, exp_avg, exp_avg_sq, master=None, numel: Optional[int] = None,
                dtype: Optional[int] = None) -> EeAdamTensor:
    """Descriptor of one parameter tensor for ee_adam_update.  With torch
    tensors, numel and dtype default to the parameter's."""
    if numel is None:
        numel = param.numel()
    if dtype is None:
        import torch
        dtype = EE_BF16 if param.dtype == torch.bfloat16 else EE_F32
    return EeAdamTensor(ptr(param), ptr(master), ptr(grad), ptr(exp_avg), ptr(exp_avg_sq),
                        int(numel), int(dtype), 0)


def ee_adam_update(tensors: Sequence[EeAdamTensor], lr: float, beta1: float, beta2: float,
                   eps: float, step: int, stream, check=True) -> int:
    arr = (EeAdamTensor * max(1, len(tensors)))(*tensors)
    s = lib().ee_adam_update(len(tensors), arr, lr, beta1, beta2, eps, step, stream)
    return _check(s, "ee_adam_update") if check else s


def ee_lr_schedule(step: int, total_steps: int, warmup_fraction: float, lr_max: float,
                   lr_min: float) -> float:
    return lib().ee_lr_schedule(step, total_steps, warmup_fraction, lr_max, lr_min)


def ee_decode_workspace_bytes(e: EeExit, n_rows: int) -> int:
    n = lib().ee_decode_workspace_bytes(ctypes.byref(e), n_rows)
    if n == 0:
        raise EEError(EE_ERR_SHAPE, "ee_decode_workspace_bytes", ee_last_error())
    return n


def ee_exit_decide(e: EeExit, hidden, n_rows: int, threshold: float, token, confidence, exit_flag,
                   ws, ws_bytes: int, stream, check=True) -> int:
    s = lib().ee_exit_decide(ctypes.byref(e), ptr(hidden), n_rows, threshold, ptr(token),
                             ptr(confidence), ptr(exit_flag), ptr(ws), ws_bytes, stream)
    return _check(s, "ee_exit_decide") if check else s


def ee_exit_decide_static(e: EeExit, hidden, n_rows: int, threshold: float, token, confidence, exit_flag,
                          stream, check=True) -> int:
    s = lib().ee_exit_decide_static(ctypes.byref(e), ptr(hidden), n_rows, threshold, ptr(token),
                                    ptr(confidence), ptr(exit_flag), stream)
    return _check(s, "ee_exit_decide_static") if check else s
