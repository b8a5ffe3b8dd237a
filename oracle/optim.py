"""Plain fp64 CPU oracle of the exit-parameter update -- TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg import
this module; the product path never does, and nothing here is shared with it.

What it computes (EE-Tuning, arXiv 2402.00518):
  * Sec. 2.2, "Computational efficiency": each tuning iteration ends with an
    update of every exit's parameters from their gradients.
  * Sec. 3, "Tuning": the optimiser is Adam with beta1 = 0.9, beta2 = 0.95,
    eps = 1e-5, under a learning-rate schedule with linear warmup over the
    first 1% of the iterations to a maximum of 1e-4 and linear decay to a
    minimum of 1e-5.

Adam is the update of Kingma and Ba (2015, Algorithm 1):
    m_t = beta1 m_{t-1} + (1 - beta1) g_t
    v_t = beta2 v_{t-1} + (1 - beta2) g_t^2
    theta_t = theta_{t-1} - lr_t * m_hat_t / (sqrt(v_hat_t) + eps),
    m_hat_t = m_t / (1 - beta1^t),  v_hat_t = v_t / (1 - beta2^t).

Readings where the paper is silent (also listed in the design notes):
  R14 no weight decay and no gradient clipping (neither is mentioned);
      eps is added after the square root, as in Kingma and Ba;
  R15 the schedule counts updates from 1; W = floor(warmup_fraction * T)
      warmup updates with lr = lr_max * s / W, then
      lr = lr_min + (lr_max - lr_min) (T - s) / (T - W) up to s = T, and
      lr_min after T;
  R16 mixed precision keeps fp32 master weights and fp32 moments; a bf16
      parameter is the master rounded to nearest even.  Without a master,
      the parameter itself is read, updated and written back.
"""

from __future__ import annotations

import math
from typing import Optional, Tuple

import numpy as np

PAPER_BETA1 = 0.9
PAPER_BETA2 = 0.95
PAPER_EPS = 1e-5
PAPER_LR_MAX = 1e-4
PAPER_LR_MIN = 1e-5
PAPER_WARMUP_FRACTION = 0.01
PAPER_ITERATIONS = 40000


def lr_schedule(step: int, total_steps: int, warmup_fraction: float, lr_max: float,
                lr_min: float) -> float:
    """Learning rate of update number `step` (1-based), Sec. 3 "Tuning" (R15)."""
    warmup = int(math.floor(warmup_fraction * total_steps))
    if step <= warmup:
        return lr_max * step / warmup
    if step <= total_steps:
        return lr_min + (lr_max - lr_min) * (total_steps - step) / (total_steps - warmup)
    return lr_min


def adam_step(theta: np.ndarray, grad: np.ndarray, m: np.ndarray, v: np.ndarray, step: int,
              lr: float, beta1: float = PAPER_BETA1, beta2: float = PAPER_BETA2,
              eps: float = PAPER_EPS) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """One Adam update in fp64; returns (theta_t, m_t, v_t).  Inputs are not modified."""
    theta = np.asarray(theta, dtype=np.float64)
    g = np.asarray(grad, dtype=np.float64)
    m_t = beta1 * np.asarray(m, dtype=np.float64) + (1.0 - beta1) * g
    v_t = beta2 * np.asarray(v, dtype=np.float64) + (1.0 - beta2) * g * g
    m_hat = m_t / (1.0 - beta1 ** step)
    v_hat = v_t / (1.0 - beta2 ** step)
    return theta - lr * m_hat / (np.sqrt(v_hat) + eps), m_t, v_t


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """fp32 values rounded to the nearest bfloat16 (ties to even), returned as
    float64.  Written from the format's definition: keep the top 16 bits of
    the binary32 pattern, rounding on the 16 dropped bits."""
    f = np.asarray(x, dtype=np.float32)
    bits = f.view(np.uint32).astype(np.uint64)
    lower = bits & 0xFFFF
    upper = bits >> 16
    round_up = (lower > 0x8000) | ((lower == 0x8000) & ((upper & 1) == 1))
    upper = upper + round_up.astype(np.uint64)
    nan = np.isnan(f)
    out = (upper.astype(np.uint32) << 16).view(np.float32)
    out = np.where(nan, np.float32(np.nan), out)
    return out.astype(np.float64)


def mixed_precision_update(param: np.ndarray, master: Optional[np.ndarray], grad: np.ndarray,
                           m: np.ndarray, v: np.ndarray, step: int, lr: float, beta1: float,
                           beta2: float, eps: float, param_bf16: bool):
    """The update of one parameter tensor as stored (R16).

    param: the stored parameter values (decoded to float64); master: fp32
    master values (float64) or None.  Returns (param_t, master_t or None,
    m_t, v_t); every returned tensor is rounded to its storage type
    (param to bf16 when param_bf16, everything else to fp32)."""
    src = master if master is not None else param
    theta, m_t, v_t = adam_step(src, grad, m, v, step, lr, beta1, beta2, eps)
    theta32 = theta.astype(np.float32).astype(np.float64)
    param_t = round_to_bf16(theta32) if param_bf16 else theta32
    master_t = theta32 if master is not None else None
    return (param_t, master_t, m_t.astype(np.float32).astype(np.float64),
            v_t.astype(np.float32).astype(np.float64))
