"""Seeded synthetic inputs for the early-exit head training step.

This module only draws random numbers and packs them into the storage
formats both sides read (fp32, or bf16 bit patterns as uint16).  It holds
none of the method's arithmetic: no norm, no projection, no softmax.  The
HIP path and the fp64 oracle decode the very same bits.

Workload shapes follow the Llama-2 models the paper tunes (Sec. 3, "Models"
and "Tuning": batch 16 x sequence 2048, Llama 2-Chat 7B/13B/70B).  Real
hidden states and the pre-training corpus are not available, so:
  * hidden states X[n, :] = s_n * z_n with z ~ N(0, 1) and a per-row
    lognormal(0, 0.5) scale s_n, mimicking the spread of hidden-state norms
    across tokens;
  * weights ~ N(0, 0.02^2), the usual GPT initialisation (the paper's
    "random" init, Sec. 2.1);
  * targets follow a truncated Zipf law P(rank k) ~ k^-1.1 over the vocab,
    mapped to token ids by a seeded permutation (natural-language token
    frequencies without clustering the frequent ids in one vocab tile).
"""

from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional

import numpy as np

ROOT_SEED = 240200518

EXIT_EMBEDDING = 0
EXIT_NORM = 1
EXIT_MLP = 2

DTYPE_F32 = "f32"
DTYPE_BF16 = "bf16"


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shape and distribution recipe of one synthetic exit-head step."""

    name: str
    kind: int              # EXIT_* of every exit
    n_tokens: int          # N = batch x sequence
    hidden: int            # h
    vocab: int             # V
    intermediate: int      # I (MLP exits), else 0
    dtype: str             # storage dtype of hidden states and weights
    exit_weights: tuple    # w_e per exit
    row_scale: bool        # per-row lognormal(0, 0.5) scale on X
    zipf: bool             # Zipf(1.1) targets, else uniform
    eps: float = 1e-5      # RMSNorm epsilon (Llama-2 value)
    norm: str = "rms"      # exit normalisation: "rms" or "layer" (LayerNorm, Norm exits)
    bias: bool = False     # LayerNorm with a bias beta

    @property
    def n_exits(self) -> int:
        return len(self.exit_weights)


# The five workloads: a tiny fp32 case and Llama-2 7B/13B/70B-shaped cases.
WORKLOADS: Dict[str, Workload] = {
    "tiny_norm_f32": Workload("tiny_norm_f32", EXIT_NORM, 512, 256, 1024, 0,
                              DTYPE_F32, (1.0,), False, False),
    "llama7b_norm": Workload("llama7b_norm", EXIT_NORM, 4096, 4096, 32000, 0,
                             DTYPE_BF16, (1.0,), True, True),
    "llama7b_norm_2exits": Workload("llama7b_norm_2exits", EXIT_NORM, 4096, 4096,
                                    32000, 0, DTYPE_BF16, (0.25, 0.5), True, True),
    "llama13b_mlp": Workload("llama13b_mlp", EXIT_MLP, 4096, 5120, 32000, 13824,
                             DTYPE_BF16, (1.0,), True, True),
    "llama70b_norm": Workload("llama70b_norm", EXIT_NORM, 8192, 8192, 32000, 0,
                              DTYPE_BF16, (1.0,), True, True),
    # the LayerNorm flavour of the Norm exit (with bias) at the 7B shape
    "llama7b_layernorm": Workload("llama7b_layernorm", EXIT_NORM, 4096, 4096, 32000, 0,
                                  DTYPE_BF16, (1.0,), True, True, norm="layer", bias=True),
}
WORKLOAD_ORDER = list(WORKLOADS)


def custom(kind: int, n_tokens: int, hidden: int, vocab: int, intermediate: int = 0,
           dtype: str = DTYPE_BF16, exit_weights=(1.0,), row_scale: bool = True,
           zipf: bool = True, eps: float = 1e-5, name: str = "custom", norm: str = "rms",
           bias: bool = False) -> Workload:
    """A workload of arbitrary shape drawn with the same recipe."""
    return Workload(name, kind, n_tokens, hidden, vocab, intermediate, dtype,
                    tuple(float(w) for w in exit_weights), row_scale, zipf, eps, norm, bias)


# ---------------------------------------------------------------- bf16 bits
def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round to nearest, ties to even).

    Returns the 16-bit patterns as uint16.  NaN stays NaN (quiet bit set).
    """
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    rounded = (u + 0x7FFF + lsb) >> 16
    nan = np.isnan(a)
    out = rounded.astype(np.uint16)
    if nan.any():
        out[nan] = ((u[nan] >> 16) | 0x40).astype(np.uint16)
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Decode bfloat16 bit patterns (uint16) exactly to float32."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def decode(arr: np.ndarray) -> np.ndarray:
    """Storage array (float32, or uint16 bf16 bits) -> exact float64 values."""
    if arr.dtype == np.uint16:
        return bf16_bits_to_f32(arr).astype(np.float64)
    return np.asarray(arr, dtype=np.float64)


def _store(a32: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == DTYPE_BF16:
        return f32_to_bf16_bits(a32)
    return np.ascontiguousarray(a32, dtype=np.float32)


# ------------------------------------------------------------------ drawing
def _normal(rng: np.random.Generator, shape, std: float = 1.0) -> np.ndarray:
    out = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        out *= np.float32(std)
    return out


def zipf_targets(rng: np.random.Generator, n: int, vocab: int, s: float = 1.1) -> np.ndarray:
    """Truncated Zipf over ranks 1..V, ranks mapped to ids by a permutation."""
    ranks = np.arange(1, vocab + 1, dtype=np.float64)
    p = ranks ** (-s)
    cdf = np.cumsum(p)
    cdf /= cdf[-1]
    u = rng.random(n)
    rank_idx = np.minimum(np.searchsorted(cdf, u, side="right"), vocab - 1)
    perm = rng.permutation(vocab)
    return perm[rank_idx].astype(np.int32)


@dataclasses.dataclass
class ExitParams:
    """One exit's parameters in storage format (bf16 bits or fp32)."""

    kind: int
    w_out: np.ndarray                    # [V][h]
    gamma: Optional[np.ndarray] = None   # [h]   exit norm gain (Norm, MLP)
    beta: Optional[np.ndarray] = None    # [h]   LayerNorm bias (Norm exit with bias)
    gamma_mlp: Optional[np.ndarray] = None  # [h] MLP pre-norm gain (MLP)
    w_gate: Optional[np.ndarray] = None  # [I][h]
    w_up: Optional[np.ndarray] = None    # [I][h]
    w_down: Optional[np.ndarray] = None  # [h][I]


@dataclasses.dataclass
class Batch:
    """Everything one step consumes."""

    workload: Workload
    hidden: List[np.ndarray]   # per exit, [N][h] storage format
    targets: np.ndarray        # [N] int32
    exits: List[ExitParams]
    token_weights: Optional[np.ndarray] = None   # [N] float32 or None


def make_batch(w: Workload, seed: int = 0, random_gamma: bool = False,
               token_weights: bool = False) -> Batch:
    """Draw one seeded batch for workload ``w``.

    Streams are spawned from SeedSequence([ROOT_SEED, seed, salt]) in a fixed
    order: targets (and token weights); then per exit X, row scales, W_out,
    gamma, and for MLP exits gamma_mlp, W_gate, W_up, W_down.
    """
    salt = sum((i + 1) * ord(c) for i, c in enumerate(w.name)) & 0xFFFFFFFF
    ss = np.random.SeedSequence([ROOT_SEED, int(seed), salt])
    n_streams = 2 + w.n_exits * 9
    streams = [np.random.Generator(np.random.PCG64(c)) for c in ss.spawn(n_streams)]
    it = iter(streams)

    rng_y = next(it)
    if w.zipf:
        y = zipf_targets(rng_y, w.n_tokens, w.vocab)
    else:
        y = rng_y.integers(0, w.vocab, size=w.n_tokens, dtype=np.int64).astype(np.int32)
    rng_m = next(it)
    m = None
    if token_weights:
        m = rng_m.random(w.n_tokens, dtype=np.float32)
        m[rng_m.random(w.n_tokens) < 0.1] = 0.0   # some masked tokens

    hidden, exits = [], []
    per_exit = [[next(it) for _ in range(8)] for _ in range(w.n_exits)]
    extra = [next(it) for _ in range(w.n_exits)]     # LayerNorm offsets and bias
    for (rx, rs, rw, rg, rgm, rwg, rwu, rwd), rb in zip(per_exit, extra):
        x = _normal(rx, (w.n_tokens, w.hidden))
        if w.row_scale:
            s = np.exp(0.5 * rs.standard_normal(w.n_tokens)).astype(np.float32)
            x *= s[:, None]
        if w.norm == "layer":
            # a per-row offset, so that the mean-centring of LayerNorm matters
            x += rb.standard_normal(w.n_tokens).astype(np.float32)[:, None]
        hidden.append(_store(x, w.dtype))
        w_out = _store(_normal(rw, (w.vocab, w.hidden), 0.02), w.dtype)
        p = ExitParams(kind=w.kind, w_out=w_out)
        if w.kind in (EXIT_NORM, EXIT_MLP):
            g = (1.0 + _normal(rg, (w.hidden,), 0.1)) if random_gamma \
                else np.ones(w.hidden, np.float32)
            p.gamma = _store(g, w.dtype)
        if w.kind == EXIT_NORM and w.norm == "layer" and w.bias:
            p.beta = _store(_normal(rb, (w.hidden,), 0.1), w.dtype)
        if w.kind == EXIT_MLP:
            gm = (1.0 + _normal(rgm, (w.hidden,), 0.1)) if random_gamma \
                else np.ones(w.hidden, np.float32)
            p.gamma_mlp = _store(gm, w.dtype)
            p.w_gate = _store(_normal(rwg, (w.intermediate, w.hidden), 0.02), w.dtype)
            p.w_up = _store(_normal(rwu, (w.intermediate, w.hidden), 0.02), w.dtype)
            p.w_down = _store(_normal(rwd, (w.hidden, w.intermediate), 0.02), w.dtype)
        exits.append(p)
    return Batch(w, hidden, y, exits, m)


def row_sample(n_tokens: int, count: int, seed: int = 0) -> np.ndarray:
    """Sorted, seeded sample of distinct row indices (always includes the last row)."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([ROOT_SEED, 7, seed])))
    count = min(count, n_tokens)
    idx = rng.choice(n_tokens, size=count, replace=False)
    idx[-1] = n_tokens - 1
    return np.unique(idx)
