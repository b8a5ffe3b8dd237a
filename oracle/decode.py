"""Plain fp64 CPU oracle of the early-exit decision at decode -- TEST
INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg import
this module; the product path never does, and nothing here is shared with it.

What it computes (EE-Tuning, arXiv 2402.00518, Sec. 3 "Inference"): decoding
is greedy, and an exit emits its most likely next token as soon as the
maximum next-token probability at that exit is above a pre-set threshold; a
threshold of 1 disables early exits.  For each row n of the hidden states at
one exit:
    S_n        = exit(hidden_n) W_out^T             (exit_forward, Sec. 2.1)
    token_n    = argmax_v S_n[v]                     (lowest id among ties)
    conf_n     = max_v softmax(S_n)[v] = exp(max_v S_n - logsumexp_v S_n)
    exit_n     = conf_n > threshold                  ("above": strict)

Readings (also listed in the design notes):
  R17 "above" is strict, so threshold 1 never exits (a probability is at
      most 1);
  R18 ties of the maximum logit go to the lowest token id.
"""

from __future__ import annotations

from typing import Dict

import numpy as np

from .ee_oracle import Exit, exit_forward, log_sum_exp


def exit_decide(e: Exit, x: np.ndarray, threshold: float) -> Dict[str, np.ndarray]:
    """Decision of one exit for every row of x ([N][h], decoded to float64).

    Returns logits [N][V], token [N] (int64), confidence [N] and exit [N]
    (bool)."""
    logits = exit_forward(e, np.asarray(x, dtype=np.float64))["s"]
    token = np.argmax(logits, axis=1)            # first (lowest) index of the maximum
    conf = np.exp(logits.max(axis=1) - log_sum_exp(logits))
    return {"logits": logits, "token": token, "confidence": conf, "exit": conf > threshold}
