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

// Row-vector form, for outputs stored transposed (C[m][n] at ptr[n*ld + m]):
// a lane's accumulator rows 4q..4q+3 of a block are consecutive, so they
// are one 8-byte (bf16) or 16-byte (fp32) access there.  f(row0, col, j,
// vals, loaded) runs for every such group after all load(row0_c, col_c) of
// the 32-row block have been issued (row0 and col clamped into the problem;
// the row count must be a multiple of 4).
template <class Cfg, class L, class F>
__device__ __forceinline__ void for_each_acc4_loaded(f32x16_t (&acc)[Cfg::MB][Cfg::NB], const TileCtx<Cfg> &t,
                                                     L &&load, F &&f) {
  using V = decltype(load(0, 0));
  static_for<Cfg::MB>([&](auto i) EE_ALWAYS_INLINE {
    V pre[4][Cfg::NB];
    static_for<4>([&](auto q) EE_ALWAYS_INLINE {
      const int row0 = min(t.row(i, 4 * q), t.M - 4);
      static_for<Cfg::NB>([&](auto j) EE_ALWAYS_INLINE { pre[q][j] = load(row0, min(t.col(j), t.N - 1)); });
    });
    static_for<4>([&](auto q) EE_ALWAYS_INLINE {
      constexpr int v0 = 4 * decltype(q)::value;
      const int row0 = t.row(i, v0);
      static_for<Cfg::NB>([&](auto j) EE_ALWAYS_INLINE {
        const f32x4_t c = {acc[i][j][v0], acc[i][j][v0 + 1], acc[i][j][v0 + 2], acc[i][j][v0 + 3]};
        f(row0, t.col(j), static_cast<int>(j), c, pre[q][j]);
      });
    });
  });
}

// Four consecutive elements as fp32, and back.
__device__ __forceinline__ f32x4_t load4(const float *p) { return *reinterpret_cast<const f32x4_t *>(p); }
__device__ __forceinline__ f32x4_t load4(const bf16_t *p) {
  const u32x2_t u = *reinterpret_cast<const u32x2_t *>(p);
  return f32x4_t{__uint_as_float(u[0] << 16), __uint_as_float(u[0] & 0xFFFF0000u), __uint_as_float(u[1] << 16),
                 __uint_as_float(u[1] & 0xFFFF0000u)};
}
__device__ __forceinline__ void store4(float *p, f32x4_t v) { *reinterpret_cast<f32x4_t *>(p) = v; }
__device__ __forceinline__ void store4(bf16_t *p, f32x4_t v) {
  const u32x2_t u = {static_cast<uint32_t>(f32_to_bf16(v[0])) | (static_cast<uint32_t>(f32_to_bf16(v[1])) << 16),
                     static_cast<uint32_t>(f32_to_bf16(v[2])) | (static_cast<uint32_t>(f32_to_bf16(v[3])) << 16)};
  *reinterpret_cast<u32x2_t *>(p) = u;
}

struct F2 {
  float a, b;
};

struct V2 {
  f32x4_t a, b;
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
// With a LayerNorm bias b (z = x_hat * gain + b), Z = X_hat * gain + 1 b^T, so
//   dW[r][j]       += gsum[r] * b[j]               (gsum[r] = sum_n G[n][r])
//   part_b[tile][j] = sum_{r in tile} W[r][j] * gsum[r]   (sums to d b)
template <typename T>
struct EpiWeightGrad {
  struct Params {
    float *dW;          // [M][ldw]
    int64_t ldw;
    const T *gain;      // [N] or NULL
    const T *W;         // [M][ldw] or NULL (no gain-gradient partials)
    float *part;        // [tiles over M][ldw]
    int accumulate;
    const float *gsum;  // [M] with a bias, else NULL
    const T *bias;      // [N] or NULL
    float *part_b;      // [tiles over M][ldw] with a bias
  };
  struct In {
    float w, old, gs;
  };
  template <class Cfg>
  __device__ __forceinline__ static void apply(const Params &p, f32x16_t (&acc)[Cfg::MB][Cfg::NB], const TileCtx<Cfg> &t) {
    constexpr int NB = Cfg::NB;
    float g[NB], dg[NB], bt[NB], db[NB];
    with_flag(p.gain != nullptr, [&](auto G_) EE_ALWAYS_INLINE {
      static_for<NB>([&](auto j) EE_ALWAYS_INLINE {
        g[j] = decltype(G_)::value ? to_f32(p.gain[min(t.col(j), t.N - 1)]) : 1.0f;
        dg[j] = 0.0f;
        db[j] = 0.0f;
        bt[j] = 0.0f;
      });
    });
    const bool with_w = p.W != nullptr;
    const bool with_b = p.bias != nullptr;
    if (with_b) static_for<NB>([&](auto j) EE_ALWAYS_INLINE { bt[j] = to_f32(p.bias[min(t.col(j), t.N - 1)]); });
    auto body = [&](auto W_, auto A_, auto B_) EE_ALWAYS_INLINE {
          constexpr bool kW = decltype(W_)::value, kAcc = decltype(A_)::value, kB = decltype(B_)::value;
          for_each_acc_loaded<Cfg>(
              acc, t, t.M, t.N,
              [&](int row, int col) EE_ALWAYS_INLINE {
                const int64_t o = static_cast<int64_t>(row) * p.ldw + col;
                In r{0.0f, 0.0f, 0.0f};
                if constexpr (kW) r.w = to_f32(p.W[o]);
                if constexpr (kAcc) r.old = p.dW[o];
                if constexpr (kB) r.gs = p.gsum[row];
                return r;
              },
              [&](int row, int col, int j, float c, In in) EE_ALWAYS_INLINE {
                if (row < t.M && col < t.N) {
                  float v = in.old + c * g[j];
                  if constexpr (kB) v += in.gs * bt[j];
                  p.dW[static_cast<int64_t>(row) * p.ldw + col] = v;
                  if constexpr (kW) dg[j] += in.w * c;
                  if constexpr (kW && kB) db[j] += in.w * in.gs;
                }
              });
    };
    // A bias comes with W (the bias gradient needs W): six variants.
    with_flag(with_w, [&](auto W_) EE_ALWAYS_INLINE {
      with_flag(p.accumulate != 0, [&](auto A_) EE_ALWAYS_INLINE {
        if constexpr (decltype(W_)::value)
          with_flag(with_b, [&](auto B_) EE_ALWAYS_INLINE { body(W_, A_, B_); });
        else
          body(W_, A_, std::false_type{});
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
      if (with_b) {
        tile_col_reduce<false, Cfg>(t, db);
        if (t.wave_m == 0 && t.lane < 32) {
          static_for<NB>([&](auto j) EE_ALWAYS_INLINE {
            const int col = t.col(j);
            if (col < t.N) p.part_b[static_cast<int64_t>(t.tile_m) * p.ldw + col] = db[j];
          });
        }
      }
    }
  }
};

// fp32 store with optional accumulation (dW += C).  Rows at or beyond
// `rows` are not stored (the GEMM may run over padding).  With split K,
// slice z of the product goes to C + z * zstride (partial sums).
template <typename T>
struct EpiStoreF32 {
  struct Params {
    float *C;
    int64_t ldc;
    int rows;
    int accumulate;
    int64_t zstride;
  };
  template <class Cfg>
  __device__ __forceinline__ static void apply(const Params &p0, f32x16_t (&acc)[Cfg::MB][Cfg::NB], const TileCtx<Cfg> &t) {
    Params p = p0;
    p.C += t.kz * p.zstride;
    with_flag(p.accumulate != 0, [&](auto A_) EE_ALWAYS_INLINE {
      if constexpr (!decltype(A_)::value) {
        for_each_acc<Cfg>(acc, t, [&](int row, int col, int, float a) EE_ALWAYS_INLINE {
          if (row < p.rows && col < t.N) p.C[static_cast<int64_t>(row) * p.ldc + col] = a;
        });
      } else {
        for_each_acc_loaded<Cfg>(
            acc, t, p.rows, t.N,
            [&](int row, int col) EE_ALWAYS_INLINE { return p.C[static_cast<int64_t>(row) * p.ldc + col]; },
            [&](int row, int col, int, float a, float in) EE_ALWAYS_INLINE {
              if (row < p.rows && col < t.N) p.C[static_cast<int64_t>(row) * p.ldc + col] = a + in;
            });
      }
    });
  }
};

// The SwiGLU MLP's GEMMs run transposed: rows of C are features (I or h)
// and columns are tokens, while every activation is stored token-major
// ([N][I] or [N][h]), so each lane's four consecutive rows are one vector
// access.  Feature counts are multiples of 64, so a group of four rows is
// either wholly inside the problem or wholly outside.

// Gate projection: H_g[n][i] = C[i][n], stored in the element type.
template <typename T>
struct EpiStoreTr {
  struct Params {
    T *C;          // [N][ldc]
    int64_t ldc;
  };
  template <class Cfg>
  __device__ __forceinline__ static void apply(const Params &p, f32x16_t (&acc)[Cfg::MB][Cfg::NB], const TileCtx<Cfg> &t) {
    for_each_acc4_loaded<Cfg>(
        acc, t, [&](int, int) EE_ALWAYS_INLINE { return 0; },
        [&](int row0, int col, int, f32x4_t c, int) EE_ALWAYS_INLINE {
          if (row0 < t.M && col < t.N) store4(p.C + static_cast<int64_t>(col) * p.ldc + row0, c);
        });
  }
};

// Up projection with the SwiGLU product, untransposed (rows of C are
// tokens): H_u = C, A = silu(H_g) * H_u.  Lanes 0-31 of each access cover 32
// consecutive features of one token row.
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

// Up projection with the SwiGLU product: H_u[n][i] = C[i][n],
// A[n][i] = silu(H_g[n][i]) * H_u[n][i].
template <typename T>
struct EpiSwiGLUTr {
  struct Params {
    const T *Hg;
    T *Hu;
    T *A;
    int64_t ld;
  };
  template <class Cfg>
  __device__ __forceinline__ static void apply(const Params &p, f32x16_t (&acc)[Cfg::MB][Cfg::NB], const TileCtx<Cfg> &t) {
    for_each_acc4_loaded<Cfg>(
        acc, t, [&](int row0, int col) EE_ALWAYS_INLINE { return load4(p.Hg + static_cast<int64_t>(col) * p.ld + row0); },
        [&](int row0, int col, int, f32x4_t hu, f32x4_t hg) EE_ALWAYS_INLINE {
          if (row0 < t.M && col < t.N) {
            const int64_t o = static_cast<int64_t>(col) * p.ld + row0;
            store4(p.Hu + o, hu);
            f32x4_t a;
            static_for<4>([&](auto e) EE_ALWAYS_INLINE {
              constexpr int E = decltype(e)::value;
              a[E] = silu_f(hg[E]) * hu[E];
            });
            store4(p.A + o, a);
          }
        });
  }
};

// Down projection with the residual: Y[n][j] = X[n][j] + C[j][n]  (fp32 out).
template <typename T>
struct EpiResidualTr {
  struct Params {
    float *Y;       // [N][ld]
    const T *X;     // [N][ld]
    int64_t ld;
  };
  template <class Cfg>
  __device__ __forceinline__ static void apply(const Params &p, f32x16_t (&acc)[Cfg::MB][Cfg::NB], const TileCtx<Cfg> &t) {
    for_each_acc4_loaded<Cfg>(
        acc, t, [&](int row0, int col) EE_ALWAYS_INLINE { return load4(p.X + static_cast<int64_t>(col) * p.ld + row0); },
        [&](int row0, int col, int, f32x4_t c, f32x4_t x) EE_ALWAYS_INLINE {
          if (row0 < t.M && col < t.N) store4(p.Y + static_cast<int64_t>(col) * p.ld + row0, c + x);
        });
  }
};

// Backward of the SwiGLU product from dA[n][i] = C[i][n] (C = W_down^T dY^T):
//   dH_g = dA * H_u * silu'(H_g),   dH_u = dA * silu(H_g).
template <typename T>
struct EpiSwiGLUBwdTr {
  struct Params {
    const T *Hg;
    const T *Hu;
    T *dHg;
    T *dHu;
    int64_t ld;
  };
  template <class Cfg>
  __device__ __forceinline__ static void apply(const Params &p, f32x16_t (&acc)[Cfg::MB][Cfg::NB], const TileCtx<Cfg> &t) {
    for_each_acc4_loaded<Cfg>(
        acc, t,
        [&](int row0, int col) EE_ALWAYS_INLINE {
          const int64_t o = static_cast<int64_t>(col) * p.ld + row0;
          return V2{load4(p.Hg + o), load4(p.Hu + o)};
        },
        [&](int row0, int col, int, f32x4_t da, V2 h) EE_ALWAYS_INLINE {
          if (row0 < t.M && col < t.N) {
            const int64_t o = static_cast<int64_t>(col) * p.ld + row0;
            f32x4_t dg, du;
            static_for<4>([&](auto e) EE_ALWAYS_INLINE {
              constexpr int E = decltype(e)::value;
              dg[E] = da[E] * h.b[E] * silu_grad_f(h.a[E]);
              du[E] = da[E] * silu_f(h.a[E]);
            });
            store4(p.dHg + o, dg);
            store4(p.dHu + o, du);
          }
        });
  }
};

}  // namespace ee
