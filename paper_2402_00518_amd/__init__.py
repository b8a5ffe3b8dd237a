"""MI355X-native EE-Tuning exit-head training step (arXiv 2402.00518).

The computation lives in libeetune.so (HIP kernels for gfx950 behind the C
ABI of include/ee_tuning.h).  ``binding`` exposes that ABI under the same
names; ``session`` keeps device buffers in torch tensors.
"""

from . import binding  # noqa: F401
from .binding import (  # noqa: F401
    EE_BF16, EE_EXIT_EMBEDDING, EE_EXIT_LAYER, EE_EXIT_MLP, EE_EXIT_NORM, EE_F32,
    EE_FLAG_DYNAMIC_TOKEN_WEIGHTS, EEError, ee_abi_version, ee_check_device_error,
    ee_head_backward, ee_head_forward_loss, ee_last_error, ee_multi_exit_step,
    ee_status_string, ee_workspace_bytes,
)

__all__ = [
    "binding", "EEError", "ee_abi_version", "ee_check_device_error", "ee_head_backward",
    "ee_head_forward_loss", "ee_last_error", "ee_multi_exit_step", "ee_status_string",
    "ee_workspace_bytes",
]
