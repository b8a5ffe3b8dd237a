// Fused epilogues of the exit-head GEMMs.  Each receives the wave's MB x NB
// blocks of 32 x 32 fp32 accumulators and the tile context (see gemm.h for
// the accumulator-to-(row, col) map).  Accumulators are only ever indexed
// with compile-time indices (for_each_acc), so they stay in registers.
#pragma once

#include "gemm.h"

namespace ee {

// f(row, col, j, value) for every accumulator element of the lane; j is the
// lane's column slot (0..NB-1).
template <class Cfg, class F>
__device__ __forceinline__ void for_each_acc(f32x16_t (&acc)[Cfg::MB][Cfg::NB], const TileCtx<Cfg> &t, F &&f) {
  static_for<Cfg::MB>([&](auto i) EE_ALWAYS_INLINE {
    static_for<16>([&](auto v) EE_ALWAYS_INLINE {
      const int row = t.row(i, v);
      static_for<Cfg::NB>([&](auto j) EE_ALWAYS_INLINE { f(row, t.col(j), static_cast<int>(j), acc[i][j][decltype(v)::value]); });
    });
  });
}

// Same, with operands the epilogue reads from memory: for each 32-row block
// first every load(row_c, col_c) of the block is issued (rows and columns
// clamped into [0, rows) x [0, cols), so no load is predicated), then
// f(row, col, j, value, loaded) runs for the block.  Loads therefore never
// wait behind the stores of the same block.
template <class Cfg, class L, class F>
__device__ __forceinline__ void for_each_acc_loaded(f32x16_t (&acc)[Cfg::MB][Cfg::NB], const TileCtx<Cfg> &t, int rows,
                                                    int cols, L &&load, F &&f) {
  using V = decltype(load(0, 0));
  static_for<Cfg::MB>([&](auto i) EE_ALWAYS_INLINE {
    V pre[16][Cfg::NB];
    static_for<16>([&](auto v) EE_ALWAYS_INLINE {
      const int row = min(t.row(i, v), rows - 1);
      static_for<Cfg::NB>([&](auto j) EE_ALWAYS_INLINE { pre[v][j] = load(row, min(t.col(j), cols - 1)); });
    });
    static_for<16>([&](auto v) EE_ALWAYS_INLINE {
      const int row = t.row(i, v);
      static_for<Cfg::NB>([&](auto j) EE_ALWAYS_INLINE {
        f(row, t.col(j), static_cast<int>(j), acc[i][j][decltype(v)::value], pre[v][j]);
      });
    });
  });
}

struct F2 {
  float a, b;
};

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
  template <class Cfg>
  __device__ __forceinline__ static void apply(const Params &p, f32x16_t (&acc)[Cfg::MB][Cfg::NB], const TileCtx<Cfg> &t) {
    constexpr int NB = Cfg::NB;
    int y[NB];
    float mx[NB], sm[NB];
    static_for<NB>([&](auto j) EE_ALWAYS_INLINE {
      const int col = t.col(j);
      y[j] = col < t.N ? p.targets[col] : -1;
      mx[j] = -INFINITY;
      sm[j] = 0.0f;
    });
    for_each_acc<Cfg>(acc, t, [&](int row, int col, int j, float a) EE_ALWAYS_INLINE {
      if (row < t.M) {
        mx[j] = fmaxf(mx[j], a);
        if (row == y[j]) p.tgt[col] = a;
      }
    });
    tile_col_reduce<true, Cfg>(t, mx);
    for_each_acc<Cfg>(acc, t, [&](int row, int col, int j, float a) EE_ALWAYS_INLINE {
      if (row < t.M) {
        const float e = fast_exp(a - mx[j]);
        sm[j] += e;
        if (col < t.N) p.P[static_cast<int64_t>(row) * p.ldp + col] = from_f32<T>(e);
      }
    });
    tile_col_reduce<false, Cfg>(t, sm);
    if (t.wave_m == 0 && t.lane < 32) {
      static_for<NB>([&](auto j) EE_ALWAYS_INLINE {
        const int col = t.col(j);
        if (col < t.N) {
          p.part_m[static_cast<int64_t>(t.tile_m) * p.ldp + col] = mx[j];
          p.part_l[static_cast<int64_t>(t.tile_m) * p.ldp + col] = sm[j];
        }
      });
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
  template <class Cfg>
  __device__ __forceinline__ static void apply(const Params &p, f32x16_t (&acc)[Cfg::MB][Cfg::NB], const TileCtx<Cfg> &t) {
    constexpr int NB = Cfg::NB;
    float g[NB], dg[NB];
    with_flag(p.gain != nullptr, [&](auto G_) EE_ALWAYS_INLINE {
      static_for<NB>([&](auto j) EE_ALWAYS_INLINE {
        g[j] = decltype(G_)::value ? to_f32(p.gain[min(t.col(j), t.N - 1)]) : 1.0f;
        dg[j] = 0.0f;
      });
    });
    const bool with_w = p.W != nullptr;
    with_flag(with_w, [&](auto W_) EE_ALWAYS_INLINE {
      with_flag(p.accumulate != 0, [&](auto A_) EE_ALWAYS_INLINE {
        constexpr bool kW = decltype(W_)::value, kAcc = decltype(A_)::value;
        for_each_acc_loaded<Cfg>(
            acc, t, t.M, t.N,
            [&](int row, int col) EE_ALWAYS_INLINE {
              const int64_t o = static_cast<int64_t>(row) * p.ldw + col;
              F2 r{0.0f, 0.0f};
              if constexpr (kW) r.a = to_f32(p.W[o]);
              if constexpr (kAcc) r.b = p.dW[o];
              return r;
            },
            [&](int row, int col, int j, float c, F2 in) EE_ALWAYS_INLINE {
              if (row < t.M && col < t.N) {
                p.dW[static_cast<int64_t>(row) * p.ldw + col] = in.b + c * g[j];
                if constexpr (kW) dg[j] += in.a * c;
              }
            });
      });
    });
    if (with_w) {
      tile_col_reduce<false, Cfg>(t, dg);
      if (t.wave_m == 0 && t.lane < 32) {
        static_for<NB>([&](auto j) EE_ALWAYS_INLINE {
          const int col = t.col(j);
          if (col < t.N) p.part[static_cast<int64_t>(t.tile_m) * p.ldw + col] = dg[j];
        });
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
  template <class Cfg>
  __device__ __forceinline__ static void apply(const Params &p, f32x16_t (&acc)[Cfg::MB][Cfg::NB], const TileCtx<Cfg> &t) {
    with_flag(p.residual != nullptr, [&](auto R_) EE_ALWAYS_INLINE {
      with_flag(p.accumulate != 0, [&](auto A_) EE_ALWAYS_INLINE {
        constexpr bool kRes = decltype(R_)::value, kAcc = decltype(A_)::value;
        if constexpr (!kRes && !kAcc) {
          for_each_acc<Cfg>(acc, t, [&](int row, int col, int, float a) EE_ALWAYS_INLINE {
            if (row < p.rows && col < t.N) p.C[static_cast<int64_t>(row) * p.ldc + col] = a;
          });
        } else {
          for_each_acc_loaded<Cfg>(
              acc, t, p.rows, t.N,
              [&](int row, int col) EE_ALWAYS_INLINE {
                float r = 0.0f;
                if constexpr (kRes) r += to_f32(p.residual[static_cast<int64_t>(row) * p.ldr + col]);
                if constexpr (kAcc) r += p.C[static_cast<int64_t>(row) * p.ldc + col];
                return r;
              },
              [&](int row, int col, int, float a, float in) EE_ALWAYS_INLINE {
                if (row < p.rows && col < t.N) p.C[static_cast<int64_t>(row) * p.ldc + col] = a + in;
              });
        }
      });
    });
  }
};

// Store in the element type (gate projection H_g of the SwiGLU MLP).
template <typename T>
struct EpiStoreT {
  struct Params {
    T *C;
    int64_t ldc;
  };
  template <class Cfg>
  __device__ __forceinline__ static void apply(const Params &p, f32x16_t (&acc)[Cfg::MB][Cfg::NB], const TileCtx<Cfg> &t) {
    for_each_acc<Cfg>(acc, t, [&](int row, int col, int, float a) EE_ALWAYS_INLINE {
      if (row < t.M && col < t.N) p.C[static_cast<int64_t>(row) * p.ldc + col] = from_f32<T>(a);
    });
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
  template <class Cfg>
  __device__ __forceinline__ static void apply(const Params &p, f32x16_t (&acc)[Cfg::MB][Cfg::NB], const TileCtx<Cfg> &t) {
    for_each_acc_loaded<Cfg>(
        acc, t, t.M, t.N,
        [&](int row, int col) EE_ALWAYS_INLINE { return to_f32(p.Hg[static_cast<int64_t>(row) * p.ld + col]); },
        [&](int row, int col, int, float hu, float hg) EE_ALWAYS_INLINE {
          if (row < t.M && col < t.N) {
            const int64_t o = static_cast<int64_t>(row) * p.ld + col;
            p.Hu[o] = from_f32<T>(hu);
            p.A[o] = from_f32<T>(silu_f(hg) * hu);
          }
        });
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
  template <class Cfg>
  __device__ __forceinline__ static void apply(const Params &p, f32x16_t (&acc)[Cfg::MB][Cfg::NB], const TileCtx<Cfg> &t) {
    for_each_acc_loaded<Cfg>(
        acc, t, t.M, t.N,
        [&](int row, int col) EE_ALWAYS_INLINE {
          const int64_t o = static_cast<int64_t>(row) * p.ld + col;
          return F2{to_f32(p.Hg[o]), to_f32(p.Hu[o])};
        },
        [&](int row, int col, int, float da, F2 h) EE_ALWAYS_INLINE {
          if (row < t.M && col < t.N) {
            const int64_t o = static_cast<int64_t>(row) * p.ld + col;
            p.dHg[o] = from_f32<T>(da * h.b * silu_grad_f(h.a));
            p.dHu[o] = from_f32<T>(da * silu_f(h.a));
          }
        });
  }
};

}  // namespace ee
