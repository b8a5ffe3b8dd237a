// Fused epilogues of the exit-head GEMMs.  Each receives the wave's 2 x 2
// block of 32 x 32 fp32 accumulators and the tile context (see gemm.h for
// the accumulator-to-(row, col) map).
#pragma once

#include "gemm.h"

namespace ee {

// Logits, transposed: C[v][n] = S[n][v] = Z[n] . W_out[v]  (rows = vocab ids,
// columns = tokens).  Per (vocab tile, token) it keeps the online-softmax
// partials m = max_v S and l = sum_v exp(S - m) over the tile's rows, stores
// P = exp(S - m) (the only copy of the logits that reaches memory) and
// captures the fp32 logit of each token's target (next-token NLL, Sec. 2).
template <typename T>
struct EpiLogits {
  struct Params {
    T *P;               // [V][ldp]
    int64_t ldp;        // padded token count
    float *part_m;      // [tiles over V][ldp]
    float *part_l;      // [tiles over V][ldp]
    float *tgt;         // [ldp] target logit
    const int32_t *targets;
  };
  __device__ static void apply(const Params &p, f32x16_t (&acc)[2][2], const TileCtx &t) {
    int y[2];
    float mx[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int col = t.col(j);
      y[j] = col < t.N ? p.targets[col] : -1;
      mx[j] = -INFINITY;
    }
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = t.row(i, v);
        if (row < t.M) {
#pragma unroll
          for (int j = 0; j < 2; ++j) {
            const float a = acc[i][j][v];
            mx[j] = fmaxf(mx[j], a);
            if (row == y[j]) p.tgt[t.col(j)] = a;
          }
        }
      }
    tile_col_reduce<true>(t, mx);
    float sm[2] = {0.0f, 0.0f};
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = t.row(i, v);
        if (row < t.M) {
#pragma unroll
          for (int j = 0; j < 2; ++j) {
            const int col = t.col(j);
            const float e = fast_exp(acc[i][j][v] - mx[j]);
            sm[j] += e;
            if (col < t.N) p.P[static_cast<int64_t>(row) * p.ldp + col] = from_f32<T>(e);
          }
        }
      }
    tile_col_reduce<false>(t, sm);
    if (t.wave_m == 0 && t.lane < 32) {
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int col = t.col(j);
        if (col < t.N) {
          p.part_m[static_cast<int64_t>(t.tile_m) * p.ldp + col] = mx[j];
          p.part_l[static_cast<int64_t>(t.tile_m) * p.ldp + col] = sm[j];
        }
      }
    }
  }
};

// Weight gradient with a gain folded in:  C = G^T X_hat (rows = output rows
// of the weight, columns = hidden features).
//   dW[r][j]      = C[r][j] * gain[j]          (gain == NULL: no scale)
//   part[tile][j] = sum_{r in tile} W[r][j] * C[r][j]
// The partials sum over tiles to the gain's gradient, because
//   sum_n dZ[n][j] x_hat[n][j] = sum_r W[r][j] (G^T x_hat)[r][j],
// the same triple sum reordered; no dZ GEMM is needed for it.
template <typename T>
struct EpiWeightGrad {
  struct Params {
    float *dW;          // [M][ldw]
    int64_t ldw;
    const T *gain;      // [N] or NULL
    const T *W;         // [M][ldw] or NULL (no gain-gradient partials)
    float *part;        // [tiles over M][ldw]
    int accumulate;
  };
  __device__ static void apply(const Params &p, f32x16_t (&acc)[2][2], const TileCtx &t) {
    float g[2], dg[2] = {0.0f, 0.0f};
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int col = t.col(j);
      g[j] = (p.gain != nullptr && col < t.N) ? to_f32(p.gain[col]) : 1.0f;
    }
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = t.row(i, v);
        if (row >= t.M) continue;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int col = t.col(j);
          if (col >= t.N) continue;
          const int64_t o = static_cast<int64_t>(row) * p.ldw + col;
          const float c = acc[i][j][v];
          const float d = c * g[j];
          p.dW[o] = p.accumulate ? p.dW[o] + d : d;
          if (p.W != nullptr) dg[j] += to_f32(p.W[o]) * c;
        }
      }
    if (p.W != nullptr) {
      tile_col_reduce<false>(t, dg);
      if (t.wave_m == 0 && t.lane < 32) {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int col = t.col(j);
          if (col < t.N) p.part[static_cast<int64_t>(t.tile_m) * p.ldw + col] = dg[j];
        }
      }
    }
  }
};

// fp32 store with optional residual (Y = X + C) and accumulation (dW += C).
// Rows at or beyond `rows` are not stored (the GEMM may run over padding).
template <typename T>
struct EpiStoreF32 {
  struct Params {
    float *C;
    int64_t ldc;
    const T *residual;  // same layout as C, or NULL
    int64_t ldr;
    int rows;
    int accumulate;
  };
  __device__ static void apply(const Params &p, f32x16_t (&acc)[2][2], const TileCtx &t) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = t.row(i, v);
        if (row >= p.rows) continue;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int col = t.col(j);
          if (col >= t.N) continue;
          float c = acc[i][j][v];
          if (p.residual != nullptr) c += to_f32(p.residual[static_cast<int64_t>(row) * p.ldr + col]);
          const int64_t o = static_cast<int64_t>(row) * p.ldc + col;
          p.C[o] = p.accumulate ? p.C[o] + c : c;
        }
      }
  }
};

// Store in the element type (gate projection H_g of the SwiGLU MLP).
template <typename T>
struct EpiStoreT {
  struct Params {
    T *C;
    int64_t ldc;
  };
  __device__ static void apply(const Params &p, f32x16_t (&acc)[2][2], const TileCtx &t) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = t.row(i, v);
        if (row >= t.M) continue;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int col = t.col(j);
          if (col < t.N) p.C[static_cast<int64_t>(row) * p.ldc + col] = from_f32<T>(acc[i][j][v]);
        }
      }
  }
};

// Up projection H_u with the SwiGLU product: A = silu(H_g) * H_u.
template <typename T>
struct EpiSwiGLU {
  struct Params {
    const T *Hg;
    T *Hu;
    T *A;
    int64_t ld;
  };
  __device__ static void apply(const Params &p, f32x16_t (&acc)[2][2], const TileCtx &t) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = t.row(i, v);
        if (row >= t.M) continue;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int col = t.col(j);
          if (col >= t.N) continue;
          const int64_t o = static_cast<int64_t>(row) * p.ld + col;
          const float hu = acc[i][j][v];
          const float hg = to_f32(p.Hg[o]);
          p.Hu[o] = from_f32<T>(hu);
          p.A[o] = from_f32<T>(silu_f(hg) * hu);
        }
      }
  }
};

// Backward of the SwiGLU product from dA = dY W_down:
//   dH_g = dA * H_u * silu'(H_g),   dH_u = dA * silu(H_g).
template <typename T>
struct EpiSwiGLUBwd {
  struct Params {
    const T *Hg;
    const T *Hu;
    T *dHg;
    T *dHu;
    int64_t ld;
  };
  __device__ static void apply(const Params &p, f32x16_t (&acc)[2][2], const TileCtx &t) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = t.row(i, v);
        if (row >= t.M) continue;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int col = t.col(j);
          if (col >= t.N) continue;
          const int64_t o = static_cast<int64_t>(row) * p.ld + col;
          const float da = acc[i][j][v];
          const float hg = to_f32(p.Hg[o]);
          const float hu = to_f32(p.Hu[o]);
          p.dHg[o] = from_f32<T>(da * hu * silu_grad_f(hg));
          p.dHu[o] = from_f32<T>(da * silu_f(hg));
        }
      }
  }
};

}  // namespace ee
