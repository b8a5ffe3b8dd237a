"""Device-resident buffers for the exit-head step, owned by torch.

torch provides device memory and the stream; every computation is a call
into libeetune.so through the binding.  A Session holds one step's inputs
(hidden states, targets, token weights), the exits' parameters, their fp32
gradients, the loss outputs and the workspace.
"""

from __future__ import annotations

from typing import List, Optional, Sequence

import numpy as np
import torch

from . import binding as B


def to_device(arr: np.ndarray, device) -> torch.Tensor:
    """numpy storage array (float32, int32, or uint16 bf16 bits) -> device tensor."""
    arr = np.ascontiguousarray(arr)
    if arr.dtype == np.uint16:
        return torch.from_numpy(arr.view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(arr).to(device)


def current_stream() -> int:
    return torch.cuda.current_stream().cuda_stream


class Session:
    """All buffers of a multi-exit step over one batch.

    ``exits`` is a list of dicts with the storage arrays ``w_out`` and, per
    kind, ``gamma``, ``gamma_mlp``, ``w_gate``, ``w_up``, ``w_down``.
    """

    def __init__(self, kind: int, dtype: int, hidden: int, vocab: int, intermediate: int,
                 eps: float, exits: Sequence[dict], hidden_states: Sequence[np.ndarray],
                 targets: np.ndarray, token_weights: Optional[np.ndarray] = None,
                 exit_weights: Sequence[float] = (1.0,), device: str = "cuda:0",
                 kinds: Optional[Sequence[int]] = None, norm: int = B.EE_NORM_RMS):
        self.device = torch.device(device)
        self.n_tokens = int(len(targets))
        self.hidden, self.vocab, self.intermediate = hidden, vocab, intermediate
        self.dtype = dtype
        self.exit_weights = [float(w) for w in exit_weights]
        kinds = list(kinds) if kinds is not None else [kind] * len(exits)
        self.kinds = kinds
        self.params: List[dict] = []
        self.grads: List[dict] = []
        self.c_exits: List[B.EeExit] = []
        self.c_grads: List[B.EeExitGrads] = []
        for k, p in zip(kinds, exits):
            t = {name: to_device(a, self.device) for name, a in p.items() if a is not None}
            self.params.append(t)
            inter = intermediate if k == B.EE_EXIT_MLP else 0
            self.c_exits.append(B.make_exit(k, dtype, hidden, vocab, inter, eps, norm=norm, **t))
            g = {"d_w_out": torch.zeros(vocab, hidden, dtype=torch.float32, device=self.device)}
            if k != B.EE_EXIT_EMBEDDING:
                g["d_gamma"] = torch.zeros(hidden, dtype=torch.float32, device=self.device)
            if "beta" in t:
                g["d_beta"] = torch.zeros(hidden, dtype=torch.float32, device=self.device)
            if k == B.EE_EXIT_MLP:
                g["d_gamma_mlp"] = torch.zeros(hidden, dtype=torch.float32, device=self.device)
                g["d_w_gate"] = torch.zeros(intermediate, hidden, dtype=torch.float32, device=self.device)
                g["d_w_up"] = torch.zeros(intermediate, hidden, dtype=torch.float32, device=self.device)
                g["d_w_down"] = torch.zeros(hidden, intermediate, dtype=torch.float32, device=self.device)
            self.grads.append(g)
            self.c_grads.append(B.make_grads(**g))
        self.x = [to_device(h, self.device) for h in hidden_states]
        self.targets = to_device(np.asarray(targets, dtype=np.int32), self.device)
        self.token_w = None if token_weights is None else \
            to_device(np.asarray(token_weights, dtype=np.float32), self.device)
        self.ws_bytes = B.ee_workspace_bytes(self.c_exits, self.n_tokens)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=self.device)
        ne = len(exits)
        self.loss_total = torch.zeros(1, dtype=torch.float32, device=self.device)
        self.loss_per_exit = torch.zeros(max(ne, 1), dtype=torch.float32, device=self.device)
        # L_e of ee_head_forward_loss, one 16-byte aligned slot per exit
        self.loss_fwd = torch.zeros(max(ne, 1), 4, dtype=torch.float32, device=self.device)
        self.row_loss = torch.zeros(self.n_tokens, dtype=torch.float32, device=self.device)
        self.opt_state: Optional[List[dict]] = None

    @classmethod
    def from_batch(cls, batch, device: str = "cuda:0") -> "Session":
        """Upload a workloads.Batch."""
        w = batch.workload
        dtype = B.EE_F32 if w.dtype == "f32" else B.EE_BF16
        exits = []
        for p in batch.exits:
            d = {"w_out": p.w_out, "gamma": p.gamma, "gamma_mlp": p.gamma_mlp,
                 "w_gate": p.w_gate, "w_up": p.w_up, "w_down": p.w_down, "beta": p.beta}
            exits.append({k: v for k, v in d.items() if v is not None})
        norm = B.EE_NORM_LAYER if w.norm == "layer" else B.EE_NORM_RMS
        return cls(w.kind, dtype, w.hidden, w.vocab, w.intermediate, w.eps, exits, batch.hidden,
                   batch.targets, batch.token_weights, w.exit_weights, device, norm=norm)

    # ------------------------------------------------------------ ABI calls
    def step(self, flags: int = 0, accumulate: int = 0, stream: Optional[int] = None):
        """One ee_multi_exit_step over every exit, enqueued on the stream."""
        B.ee_multi_exit_step(self.c_exits, self.x, self.targets, self.token_w, self.n_tokens,
                             self.exit_weights, flags, self.c_grads, accumulate, self.ws,
                             self.ws_bytes, self.loss_total, self.loss_per_exit,
                             current_stream() if stream is None else stream)

    def forward(self, e: int = 0, flags: int = 0, row_loss: bool = True, stream: Optional[int] = None):
        """ee_head_forward_loss of exit e: L_e into loss_fwd[e, 0], the per-row
        NLL into row_loss."""
        B.ee_head_forward_loss(self.c_exits[e], self.x[e], self.targets, self.token_w,
                               self.n_tokens, self.exit_weights[e], flags, self.ws, self.ws_bytes,
                               self.loss_fwd[e, :1], self.row_loss if row_loss else None,
                               current_stream() if stream is None else stream)

    def backward(self, e: int = 0, accumulate: int = 0, stream: Optional[int] = None):
        B.ee_head_backward(self.c_exits[e], self.n_tokens, self.ws, self.ws_bytes, self.c_grads[e],
                           accumulate, current_stream() if stream is None else stream)

    def check_device_error(self):
        B.ee_check_device_error(self.ws, self.ws_bytes, current_stream())

    # ------------------------------------------------------------ optimizer
    def init_optimizer(self, master: bool = True):
        """Adam state for every exit parameter: zero moments and, with
        `master`, an fp32 master copy of each parameter."""
        self.opt_state = []
        for params in self.params:
            st = {}
            for name, p in params.items():
                st[name] = {
                    "m": torch.zeros(p.shape, dtype=torch.float32, device=self.device),
                    "v": torch.zeros(p.shape, dtype=torch.float32, device=self.device),
                    "master": p.float().clone() if master else None,
                }
            self.opt_state.append(st)

    def adam_tensors(self) -> List[B.EeAdamTensor]:
        out = []
        for params, grads, st in zip(self.params, self.grads, self.opt_state):
            for name, p in params.items():
                s = st[name]
                out.append(B.adam_tensor(p, grads["d_" + name], s["m"], s["v"], master=s["master"]))
        return out

    def update(self, step: int, lr: float, beta1: float = 0.9, beta2: float = 0.95, eps: float = 1e-5,
               stream: Optional[int] = None):
        """One ee_adam_update over every exit parameter (Sec. 3 hyper-parameters by default)."""
        if self.opt_state is None:
            self.init_optimizer()
        B.ee_adam_update(self.adam_tensors(), lr, beta1, beta2, eps, step,
                         current_stream() if stream is None else stream)
