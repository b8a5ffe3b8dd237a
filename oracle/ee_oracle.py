"""Plain fp64 CPU oracle of the EE-Tuning exit-head training step.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the
benchmark's CPU-baseline leg may import this module.  The product path
(the HIP library and its Python binding) never calls it and shares no code
with it.

What it computes (EE-Tuning, arXiv 2402.00518):
  * Sec. 2 "Preliminaries": the autoregressive LM loss, the negative
    log-likelihood of each next token.  Targets arrive already shifted: row n
    of the hidden states predicts targets[n].
  * Sec. 2.1 "Architectures of early exits": an exit maps a hidden state in
    R^h to logits in R^V.  Embedding = one h x V output matrix; Norm = a
    normalisation module in front of it; MLP = a backbone-shaped MLP in front
    of Norm.  Fig. 2's caption: modules are residual with pre-normalisation.
    Sec. 3.2: the normalisation is RMSNorm, following Llama 2.
  * Remark in Sec. 2.1: output matrices are untied (each exit owns W_out).
  * Sec. 2.2: the backbone is frozen; each exit is tuned by backpropagation
    into its own parameters only, independently of the other exits.
  * Sec. 1: exits' losses are combined as a weighted sum.
  * Sec. 2.3 "Dynamic token-wise loss weights" and Appendix A.3 "Dynamic
    token-wise loss weighting": each token's NLL may be weighted by a
    detached confidence c_t, the maximum next-token probability.

Readings where the paper is silent (each also listed in the design notes):
  R1 loss over tokens is the MEAN over the N rows (token weights multiply,
     the denominator stays N);
  R2 L = sum_e w_e L_e, un-normalised;
  R3 RMSNorm r = (mean_j s_j^2 + eps)^(-1/2), eps inside the root;
  R4 MLP exit: Y = X + W_d^T-projection of SwiGLU(RMSNorm_mlp(X)), then the
     exit RMSNorm and W_out, two separate gains;
  R5 SwiGLU: A = silu(U W_g^T) * (U W_u^T), silu(t) = t sigmoid(t), no biases;
  R6 W_out is stored [V][h] (the paper's h x V matrix, transposed storage);
  R19 LayerNorm flavour (Sec. 2.1 names LayerNorm or RMSNorm): s_hat =
     (s - mean_j s_j) (mean_j (s_j - mean)^2 + eps)^(-1/2) (biased variance,
     eps inside the root), z = s_hat * gamma + beta with an optional bias;
     an exit uses one normalisation type for all its norms;
  R20 dynamic token-wise weights combined with caller token weights: the
     two multiply, m_n = token_w[n] c_n (the paper has c_n alone; a caller
     weight of 0 keeps a row masked).

Pins (tests/test_oracle.py): a hand-worked golden example, closed forms at
W_out = 0, central finite differences, torch autograd in fp64, pure-Python
brute force, invariances and reordering identities.  The MLP exit's
arithmetic is pinned the same way, and with W_d = 0 it reduces to the Norm
exit; but Fig. 2 itself is not in the paper's text, so that R4 is the
paper's module (rather than another residual pre-norm MLP) is parity
unpinned.

Every array here is float64; inputs are decoded exactly from their storage
format before use.  Backward uses the plain chain rule (dZ = G W_out etc.),
not the reorderings the GPU path uses.
"""

from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Sequence

import numpy as np

EXIT_EMBEDDING = 0
EXIT_NORM = 1
EXIT_MLP = 2

CHUNK_ROWS = 1024


# ----------------------------------------------------------- elementwise maps
def sigmoid(t: np.ndarray) -> np.ndarray:
    """Logistic function, evaluated without overflow for either sign."""
    out = np.empty_like(t)
    pos = t >= 0
    out[pos] = 1.0 / (1.0 + np.exp(-t[pos]))
    e = np.exp(t[~pos])
    out[~pos] = e / (1.0 + e)
    return out


def silu(t: np.ndarray) -> np.ndarray:
    """SiLU (swish) gate of the SwiGLU MLP: t * sigmoid(t)."""
    return t * sigmoid(t)


def silu_grad(t: np.ndarray) -> np.ndarray:
    """d silu / dt = sigmoid(t) * (1 + t * (1 - sigmoid(t)))."""
    s = sigmoid(t)
    return s * (1.0 + t * (1.0 - s))


# ------------------------------------------------------------------- RMSNorm
def rms_inv(s: np.ndarray, eps: float) -> np.ndarray:
    """RMSNorm scale r_n = (mean_j s[n,j]^2 + eps)^(-1/2) (reading R3)."""
    return 1.0 / np.sqrt(np.mean(s * s, axis=1) + eps)


def layer_stats(s: np.ndarray, eps: float):
    """LayerNorm row statistics: mean and r = (mean_j (s_j - mean)^2 + eps)^(-1/2)
    (biased variance, eps inside the root)."""
    mu = np.mean(s, axis=1)
    c = s - mu[:, None]
    return mu, 1.0 / np.sqrt(np.mean(c * c, axis=1) + eps)


def norm_forward(e: "Exit", s: np.ndarray, gain: np.ndarray, bias: Optional[np.ndarray]):
    """The exit's normalisation of rows s: (s_hat, r, z) with z = s_hat * gain (+ bias)."""
    if e.norm == "layer":
        mu, r = layer_stats(s, e.eps)
        s_hat = (s - mu[:, None]) * r[:, None]
    else:
        r = rms_inv(s, e.eps)
        s_hat = s * r[:, None]
    z = s_hat * gain[None, :]
    if bias is not None:
        z = z + bias[None, :]
    return s_hat, r, z


def layernorm_backward(d_hat: np.ndarray, s_hat: np.ndarray, r: np.ndarray) -> np.ndarray:
    """ds for s_hat = (s - mean(s)) r:  r (d_hat - mean_j d_hat - s_hat mean_j(d_hat s_hat))."""
    return r[:, None] * (d_hat - np.mean(d_hat, axis=1, keepdims=True)
                         - s_hat * np.mean(d_hat * s_hat, axis=1, keepdims=True))


def rmsnorm_backward(d_hat: np.ndarray, s_hat: np.ndarray, r: np.ndarray) -> np.ndarray:
    """Gradient w.r.t. the RMSNorm input s, given dL/d(s_hat) with s_hat = r s.

    ds = r * (d_hat - s_hat * mean_j(d_hat * s_hat)).
    """
    proj = np.mean(d_hat * s_hat, axis=1, keepdims=True)
    return r[:, None] * (d_hat - s_hat * proj)


# -------------------------------------------------------------- parameters
@dataclasses.dataclass
class Exit:
    """One exit's parameters, float64 (Sec. 2.1 architectures)."""

    kind: int
    w_out: np.ndarray                       # [V][h]
    gamma: Optional[np.ndarray] = None      # [h]  exit RMSNorm gain
    gamma_mlp: Optional[np.ndarray] = None  # [h]  MLP pre-norm gain
    w_gate: Optional[np.ndarray] = None     # [I][h]
    w_up: Optional[np.ndarray] = None       # [I][h]
    w_down: Optional[np.ndarray] = None     # [h][I]
    eps: float = 1e-5
    norm: str = "rms"                       # "rms" or "layer" (Sec. 2.1: LayerNorm or RMSNorm)
    beta: Optional[np.ndarray] = None       # [h]  LayerNorm bias of the exit norm, or None

    @property
    def hidden(self) -> int:
        return self.w_out.shape[1]

    @property
    def vocab(self) -> int:
        return self.w_out.shape[0]

    def param_names(self) -> List[str]:
        names = ["w_out"]
        if self.kind in (EXIT_NORM, EXIT_MLP):
            names.append("gamma")
        if self.kind in (EXIT_NORM, EXIT_MLP) and self.beta is not None:
            names.append("beta")
        if self.kind == EXIT_MLP:
            names += ["gamma_mlp", "w_gate", "w_up", "w_down"]
        return names


# ---------------------------------------------------------------- forward
def exit_forward(e: Exit, x: np.ndarray) -> Dict[str, np.ndarray]:
    """Exit forward for a block of rows x [n][h]; returns every intermediate.

    Z is what the output matrix sees; S = Z W_out^T are the logits.
    """
    f: Dict[str, np.ndarray] = {"x": x}
    if e.kind == EXIT_MLP:
        u_hat, r_x, u = norm_forward(e, x, e.gamma_mlp, None)   # pre-norm (Fig. 2 caption)
        hg = u @ e.w_gate.T                          # gate projection
        hu = u @ e.w_up.T                            # up projection
        a = silu(hg) * hu                            # SwiGLU (R5)
        y = x + a @ e.w_down.T                       # residual (R4)
        f.update(r_x=r_x, u_hat=u_hat, u=u, hg=hg, hu=hu, a=a, y=y)
        s_in = y
    else:
        s_in = x
    if e.kind in (EXIT_NORM, EXIT_MLP):
        z_hat, r, z = norm_forward(e, s_in, e.gamma, e.beta)     # exit Norm (Sec. 2.1, 3.2)
        f.update(r=r, z_hat=z_hat)
    else:
        z = s_in                                     # Embedding exit
    f["z"] = z
    f["s"] = z @ e.w_out.T                           # logits [n][V]
    return f


def log_sum_exp(s: np.ndarray) -> np.ndarray:
    """Row-wise log sum_v exp(s[n, v]), shifted by the row max."""
    mx = np.max(s, axis=1)
    return mx + np.log(np.sum(np.exp(s - mx[:, None]), axis=1))


def softmax(s: np.ndarray) -> np.ndarray:
    return np.exp(s - log_sum_exp(s)[:, None])


def token_nll(s: np.ndarray, y: np.ndarray) -> np.ndarray:
    """Per-row negative log-likelihood of the target token (Sec. 2)."""
    return log_sum_exp(s) - s[np.arange(s.shape[0]), y]


def confidence(s: np.ndarray) -> np.ndarray:
    """Maximum next-token probability per row (dynamic token weights)."""
    return np.exp(np.max(s, axis=1) - log_sum_exp(s))


# ------------------------------------------------------------------ backward
def exit_backward(e: Exit, f: Dict[str, np.ndarray], g: np.ndarray) -> Dict[str, np.ndarray]:
    """Gradients of every exit parameter given the logit gradient g = dL/dS.

    Plain chain rule through S = Z W_out^T and the modules in front of it.
    Nothing flows into the hidden states x (frozen backbone, Sec. 2.2).
    """
    grads: Dict[str, np.ndarray] = {}
    grads["w_out"] = g.T @ f["z"]                    # dL/dW_out  [V][h]
    if e.kind == EXIT_EMBEDDING:
        return grads
    dz = g @ e.w_out                                 # dL/dZ      [n][h]
    grads["gamma"] = np.sum(dz * f["z_hat"], axis=0)
    if e.beta is not None:
        grads["beta"] = np.sum(dz, axis=0)
    if e.kind == EXIT_NORM:
        return grads
    d_zhat = dz * e.gamma[None, :]
    norm_bwd = layernorm_backward if e.norm == "layer" else rmsnorm_backward
    dy = norm_bwd(d_zhat, f["z_hat"], f["r"])        # through the exit norm
    # y = x + a W_d^T: the residual branch carries no parameters.
    grads["w_down"] = dy.T @ f["a"]                  # [h][I]
    da = dy @ e.w_down                               # [n][I]
    d_hg = da * f["hu"] * silu_grad(f["hg"])
    d_hu = da * silu(f["hg"])
    grads["w_gate"] = d_hg.T @ f["u"]                # [I][h]
    grads["w_up"] = d_hu.T @ f["u"]                  # [I][h]
    du = d_hg @ e.w_gate + d_hu @ e.w_up             # [n][h]
    grads["gamma_mlp"] = np.sum(du * f["u_hat"], axis=0)
    return grads


def logit_grad(s: np.ndarray, y: np.ndarray, scale: np.ndarray) -> np.ndarray:
    """dL/dS for L = sum_n scale_n * nll_n: scale_n * (softmax - onehot)."""
    p = softmax(s)
    p[np.arange(s.shape[0]), y] -= 1.0
    return p * scale[:, None]


# ------------------------------------------------------------ token weights
def row_weights(conf: np.ndarray, token_weights: Optional[np.ndarray], r0: int, r1: int,
                dynamic_weights: bool) -> np.ndarray:
    """Loss weight m_n of rows r0..r1-1.

    The caller's token weights (all ones when None; a zero masks a row,
    reading R9) times, with ``dynamic_weights``, the detached confidence c_n,
    the maximum next-token probability (Sec. 2.3 "Dynamic token-wise loss
    weights"; Appendix A.3 gives the weighted loss -sum_t c_t log P(x_t | x_<t)).
    The paper weights by c_t alone, i.e. all caller weights one; with caller
    weights the two multiply (reading R20), so a masked row stays masked.
    c_n is treated as a constant: no gradient flows through it.
    """
    m = np.ones(r1 - r0) if token_weights is None else \
        np.asarray(token_weights[r0:r1], dtype=np.float64).copy()
    if dynamic_weights:
        m = m * conf
    return m


# ---------------------------------------------------------- one exit, all rows
@dataclasses.dataclass
class ExitResult:
    loss: float                        # L_e (unweighted, mean over N rows)
    row_loss: np.ndarray               # [N] nll per row
    grads: Dict[str, np.ndarray]       # already multiplied by the exit weight
    lse: np.ndarray                    # [N] log-sum-exp per row
    conf: np.ndarray                   # [N] max probability per row


def exit_step(e: Exit, x: np.ndarray, y: np.ndarray, exit_weight: float = 1.0,
              token_weights: Optional[np.ndarray] = None,
              dynamic_weights: bool = False,
              chunk: int = CHUNK_ROWS) -> ExitResult:
    """Loss L_e = (1/N) sum_n m_n nll_n and the gradients of exit_weight * L_e.

    m_n = token_weights[n] (all ones when None); with ``dynamic_weights`` each
    m_n is further multiplied by the detached confidence c_n (reading R20, see
    row_weights).  Rows are processed in chunks; gradients are sums over
    chunks, which is the same triple sum reordered by rows only.
    """
    n = x.shape[0]
    if n == 0:
        raise ValueError("the loss is a mean over tokens: N must be positive")
    grads: Dict[str, np.ndarray] = {}
    row_loss = np.empty(n)
    lse = np.empty(n)
    conf = np.empty(n)
    total = 0.0
    for r0 in range(0, n, chunk):
        r1 = min(n, r0 + chunk)
        f = exit_forward(e, x[r0:r1])
        s = f["s"]
        nll = token_nll(s, y[r0:r1])
        c = confidence(s)
        m = row_weights(c, token_weights, r0, r1, dynamic_weights)
        row_loss[r0:r1] = nll
        lse[r0:r1] = log_sum_exp(s)
        conf[r0:r1] = c
        total += float(np.sum(m * nll))
        g = logit_grad(s, y[r0:r1], exit_weight * m / n)
        for k, v in exit_backward(e, f, g).items():
            grads[k] = v if k not in grads else grads[k] + v
    return ExitResult(total / n, row_loss, grads, lse, conf)


def multi_exit_step(exits: Sequence[Exit], xs: Sequence[np.ndarray], y: np.ndarray,
                    exit_weights: Sequence[float],
                    token_weights: Optional[np.ndarray] = None,
                    dynamic_weights: bool = False):
    """All exits of one step: L = sum_e w_e L_e and each exit's gradients.

    Exits are independent (Sec. 2.2): each one's gradient depends only on its
    own hidden states and parameters.
    """
    per = [exit_step(e, x, y, w, token_weights, dynamic_weights)
           for e, x, w in zip(exits, xs, exit_weights)]
    total = sum(w * r.loss for w, r in zip(exit_weights, per))
    return total, per


# ------------------------------------------------- sampled outputs, any size
def exit_step_sampled(e: Exit, x: np.ndarray, y: np.ndarray, exit_weight: float,
                      v_rows: np.ndarray, i_rows: Optional[np.ndarray] = None,
                      token_weights: Optional[np.ndarray] = None,
                      chunk: int = CHUNK_ROWS, dynamic_weights: bool = False) -> Dict[str, np.ndarray]:
    """Loss, per-row NLL, full gains' gradients and sampled weight-gradient rows.

    Computes the forward for every row (the loss needs all of them), dL/dS
    and dL/dZ for every row, then only the requested rows of the weight
    gradients, each by its definition:
      dW_out[v, :] = sum_n G[n, v] Z[n, :]                (v in v_rows)
      dW_gate[i, :], dW_up[i, :], dW_down[:, i]           (i in i_rows)
    gamma and gamma_mlp gradients are computed in full.
    """
    n = x.shape[0]
    out: Dict[str, np.ndarray] = {}
    row_loss = np.empty(n)
    lse = np.empty(n)
    total = 0.0
    acc: Dict[str, np.ndarray] = {}

    def add(k, v):
        acc[k] = v if k not in acc else acc[k] + v

    for r0 in range(0, n, chunk):
        r1 = min(n, r0 + chunk)
        f = exit_forward(e, x[r0:r1])
        s = f["s"]
        nll = token_nll(s, y[r0:r1])
        m = row_weights(confidence(s), token_weights, r0, r1, dynamic_weights)
        row_loss[r0:r1] = nll
        lse[r0:r1] = log_sum_exp(s)
        total += float(np.sum(m * nll))
        g = logit_grad(s, y[r0:r1], exit_weight * m / n)
        add("w_out_rows", g[:, v_rows].T @ f["z"])
        if e.kind == EXIT_EMBEDDING:
            continue
        dz = g @ e.w_out
        add("gamma", np.sum(dz * f["z_hat"], axis=0))
        if e.beta is not None:
            add("beta", np.sum(dz, axis=0))
        if e.kind == EXIT_NORM:
            continue
        d_zhat = dz * e.gamma[None, :]
        norm_bwd = layernorm_backward if e.norm == "layer" else rmsnorm_backward
        dy = norm_bwd(d_zhat, f["z_hat"], f["r"])
        da = dy @ e.w_down
        d_hg = da * f["hu"] * silu_grad(f["hg"])
        d_hu = da * silu(f["hg"])
        du = d_hg @ e.w_gate + d_hu @ e.w_up
        add("gamma_mlp", np.sum(du * f["u_hat"], axis=0))
        if i_rows is not None:
            add("w_gate_rows", d_hg[:, i_rows].T @ f["u"])
            add("w_up_rows", d_hu[:, i_rows].T @ f["u"])
            add("w_down_cols", dy.T @ f["a"][:, i_rows])   # [h][len(i_rows)]
    out.update(acc)
    out["loss"] = np.array(total / n)
    out["row_loss"] = row_loss
    out["lse"] = lse
    return out
