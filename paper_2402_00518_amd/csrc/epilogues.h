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

// Four consecutive elements as fp32, and back.
__device__ __forceinline__ f32x4_t load4(const float *p) { return *reinterpret_cast<const f32x4_t *>(p); }
__device__ __forceinline__ f32x4_t load4(const bf16_t *p) {
  const u32x2_t u = *reinterpret_cast<const u32x2_t *>(p);
  return f32x4_t{__uint_as_float(u[0] << 16), __uint_as_float(u[0] & 0xFFFF0000u), __uint_as_float(u[1] << 16),
                 __uint_as_float(u[1] & 0xFFFF0000u)};
}
__device__ __forceinline__ void store4(float *p, f32x4_t v) { *reinterpret_cast<f32x4_t *>(p) = v; }
__device__ __forceinline__ void store4(bf16_t *p, f32x4_t v) {
  // two values per hardware convert (round to nearest even)
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  typedef __bf16 b16x2_t __attribute__((ext_vector_type(2)));
  const b16x2_t lo = __builtin_convertvector((f32x2_t{v[0], v[1]}), b16x2_t);
  const b16x2_t hi = __builtin_convertvector((f32x2_t{v[2], v[3]}), b16x2_t);
  *reinterpret_cast<u32x2_t *>(p) = u32x2_t{__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi)};
}

// ------------------------------------------------ row-slot reductions
// A lane holds accumulator element v of block (i, j) for NB columns j at one
// row per "slot" k = i * 16 + v: wave row i*32 + (v/4)*8 + (lane/32)*4 + v%4.
// Rows are shared by the 32 lanes of equal lane / 32 (each holding other
// columns), so a per-row reduction over the wave's columns is a reduction
// over those 32 lanes.
__device__ __forceinline__ int slot_row(int k, int lane) {
  const int i = k >> 4, v = k & 15;
  return i * 32 + (v >> 2) * 8 + (lane >> 5) * 4 + (v & 3);
}

// Reduce-scatter of N row slots over the 32 lanes that share them: five
// butterfly steps (lane bits 4..0), each halving the values a lane keeps, so
// N/2 + N/4 + ... + N/32 shuffles instead of 5 N.  On return v[x], x < N/32,
// is the total (sum or max) of slot base + (N/32) * (lane % 32) + x, where
// the caller's slots are base .. base + N - 1.
template <bool IsMax, int N>
__device__ __forceinline__ void slot_reduce_scatter(float (&v)[N], int lane) {
  static_assert(N >= 32 && (N & (N - 1)) == 0, "slots must be a power of two >= 32");
  static_for<5>([&](auto st) EE_ALWAYS_INLINE {
    constexpr int S = decltype(st)::value;
    constexpr int BIT = 4 - S, H = (N >> S) / 2;
    const bool hi = (lane >> BIT) & 1;
    static_for<H>([&](auto kk) EE_ALWAYS_INLINE {
      constexpr int K = decltype(kk)::value;
      const float send = hi ? v[K] : v[K + H];
      const float keep = hi ? v[K + H] : v[K];
      const float recv = __shfl_xor(send, 1 << BIT);
      v[K] = IsMax ? fmaxf(keep, recv) : keep + recv;
    });
  });
}

// Four consecutive elements, raw (converted at use so that a batch of loads
// is not split by conversions waiting on each of them).
__device__ __forceinline__ u32x2_t raw4(const bf16_t *p) { return *reinterpret_cast<const u32x2_t *>(p); }
__device__ __forceinline__ f32x4_t raw4(const float *p) { return *reinterpret_cast<const f32x4_t *>(p); }
__device__ __forceinline__ f32x4_t cvt4(u32x2_t u) {
  return f32x4_t{__uint_as_float(u[0] << 16), __uint_as_float(u[0] & 0xFFFF0000u), __uint_as_float(u[1] << 16),
                 __uint_as_float(u[1] & 0xFFFF0000u)};
}
__device__ __forceinline__ f32x4_t cvt4(f32x4_t v) { return v; }
template <typename T> struct Raw4Of;
template <> struct Raw4Of<bf16_t> { using type = u32x2_t; };
template <> struct Raw4Of<float> { using type = f32x4_t; };
template <typename T> using Raw4 = typename Raw4Of<T>::type;

// Logits: C[n][v] = S[n][v] = Z[n] . W_out[v] (rows = tokens, columns =
// vocab ids).  For every token and every WN-column slice of the vocabulary
// (one wave's columns) it keeps the online-softmax partials
// m = max_v S and l = sum_v exp(S - m), stores P = exp(S - m) (the only copy
// of the logits that reaches memory) at P[v][n], four tokens per 8- or
// 16-byte store, and captures the fp32 logit of each token's target
// (next-token NLL, Sec. 2).  Rows are handled in parts of two blocks (32
// slots), each reduced over the wave's columns by a reduce-scatter (one row
// per lane) and broadcast back through the wave's own LDS rows.
template <typename T>
struct EpiLogits {
  struct Params {
    T *P;               // [V][ldp]
    int64_t ldp;        // padded token count (multiple of 4)
    float *part_m;      // [V / WN][ldp]
    float *part_l;      // [V / WN][ldp]
    float *tgt;         // [ldp] target logit
    const int32_t *targets;
  };
  template <class Cfg>
  __device__ __forceinline__ static void apply(const Params &p, f32x16_t (&acc)[Cfg::MB][Cfg::NB], const TileCtx<Cfg> &t) {
    constexpr int NB = Cfg::NB, NPART = Cfg::MB / 2;  // parts of two blocks
    constexpr float kLog2e = 1.4426950408889634f;
    const int lane = t.lane, lo = lane & 31, hw = lane >> 5;
    const int wave = t.wave_m * Cfg::WAVES_N + t.wave_n;
    int *ylds = reinterpret_cast<int *>(t.smem);                                   // [BM] tile tokens' targets
    float *wl = reinterpret_cast<float *>(t.smem) + Cfg::BM + wave * Cfg::WM;     // this wave's rows
    __syncthreads();  // every wave is past its last fragment reads
    if (threadIdx.x < Cfg::BM) {
      const int r = t.m0 + static_cast<int>(threadIdx.x);
      ylds[threadIdx.x] = r < t.M ? p.targets[r] : -1;
    }
    __syncthreads();
    const int cbase = t.n0 + t.wave_n * Cfg::WN;  // first column of the wave
    const int64_t ct = cbase / Cfg::WN;           // its partial slice
    const int rbase = t.wave_m * Cfg::WM + hw * 4;  // tile row of the lane's slot 0
    // Does any of the wave's rows have its target among the wave's columns?
    // (rare: WN of V columns), so capture code runs in few waves.
    bool hit = false;
    static_for<Cfg::WM / 64>([&](auto h) EE_ALWAYS_INLINE {
      const int y = ylds[t.wave_m * Cfg::WM + 64 * decltype(h)::value + lane];
      hit = hit || static_cast<unsigned>(y - cbase) < static_cast<unsigned>(Cfg::WN);
    });
    const bool capture = __any(hit);
    const bool interior = t.m0 + Cfg::BM <= t.M && cbase + Cfg::WN <= t.N;
    with_flag(interior, [&](auto IN_) EE_ALWAYS_INLINE {
      constexpr bool kIn = decltype(IN_)::value;
      int col[NB];
      bool cok[NB];
      T *pcol[NB];  // P[col][m0 + rbase]: the group (I, Q) adds I*32 + Q*8
      static_for<NB>([&](auto j) EE_ALWAYS_INLINE {
        col[j] = t.col(j);
        cok[j] = kIn || col[j] < t.N;
        pcol[j] = p.P + static_cast<int64_t>(min(col[j], t.N - 1)) * p.ldp + t.m0 + rbase;
      });
      static_for<NPART>([&](auto hf) EE_ALWAYS_INLINE {
        constexpr int I0 = decltype(hf)::value * 2;
        // keep each part's accumulator reads inside the part (register pressure)
        __builtin_amdgcn_sched_barrier(0);
        float mx[32], sm[32];
        static_for<2>([&](auto ii) EE_ALWAYS_INLINE {
          constexpr int I = I0 + decltype(ii)::value;
          static_for<16>([&](auto v) EE_ALWAYS_INLINE {
            constexpr int V = decltype(v)::value;
            float m = -INFINITY;
            static_for<NB>([&](auto j) EE_ALWAYS_INLINE {
              if (cok[j]) m = fmaxf(m, acc[I][j][V]);
            });
            mx[decltype(ii)::value * 16 + V] = m;
          });
        });
        if (capture) {
          static_for<2>([&](auto ii) EE_ALWAYS_INLINE {
            constexpr int I = I0 + decltype(ii)::value;
            static_for<4>([&](auto q) EE_ALWAYS_INLINE {
              constexpr int Q = decltype(q)::value;
              const int r0 = rbase + I * 32 + Q * 8;
              const int4 y4 = *reinterpret_cast<const int4 *>(ylds + r0);
              const int yv[4] = {y4.x, y4.y, y4.z, y4.w};
              static_for<4>([&](auto e) EE_ALWAYS_INLINE {
                constexpr int E = decltype(e)::value;
                static_for<NB>([&](auto j) EE_ALWAYS_INLINE {
                  if (cok[j] && col[j] == yv[E]) p.tgt[t.m0 + r0 + E] = acc[I][j][Q * 4 + E];
                });
              });
            });
          });
        }
        slot_reduce_scatter<true>(mx, lane);
        wl[slot_row(I0 * 16 + lo, lane)] = mx[0];
        // the rows read back below are this wave's own: a wave-scope fence
        // suffices (the other waves go on with their parts)
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        // P = exp(S - m) = exp2(S log2e - m log2e), four tokens per store; row sums
        static_for<2>([&](auto ii) EE_ALWAYS_INLINE {
          constexpr int I = I0 + decltype(ii)::value;
          static_for<4>([&](auto q) EE_ALWAYS_INLINE {
            constexpr int Q = decltype(q)::value;
            const f32x4_t ml = *reinterpret_cast<const f32x4_t *>(wl + I * 32 + Q * 8 + hw * 4) * kLog2e;
            const bool rok = kIn || t.m0 + rbase + I * 32 + Q * 8 < t.M;
            f32x4_t s4 = {0.0f, 0.0f, 0.0f, 0.0f};
            static_for<NB>([&](auto j) EE_ALWAYS_INLINE {
              f32x4_t e4;
              static_for<4>([&](auto e) EE_ALWAYS_INLINE {
                constexpr int E = decltype(e)::value;
                const float x = __builtin_amdgcn_exp2f(fmaf(acc[I][j][Q * 4 + E], kLog2e, -ml[E]));
                e4[E] = cok[j] ? x : 0.0f;
              });
              if (cok[j] && rok) store4(pcol[j] + (I * 32 + Q * 8), e4);
              s4 += e4;
            });
            static_for<4>([&](auto e) EE_ALWAYS_INLINE {
              sm[decltype(ii)::value * 16 + Q * 4 + decltype(e)::value] = s4[decltype(e)::value];
            });
          });
        });
        slot_reduce_scatter<false>(sm, lane);
        const int row = t.m0 + t.wave_m * Cfg::WM + slot_row(I0 * 16 + lo, lane);
        if (cbase < t.N && row < t.M) {
          p.part_m[ct * p.ldp + row] = mx[0];
          p.part_l[ct * p.ldp + row] = sm[0];
        }
      });
    });
  }
};

// Weight gradient with a gain folded in, computed transposed:
// C = X_hat^T G (rows = features j of the weight's rows, columns = output
// rows r), stored as dW[r][j] four features per 16-byte store.
//   dW[r][j]      = C[j][r] * gain[j]          (gain == NULL: no scale)
//   part[s][j]    = sum_{r in slice s} W[r][j] * C[j][r]
// with slices s of WN output rows (one wave's columns).  The partials sum
// over slices to the gain's gradient, because
//   sum_n dZ[n][j] x_hat[n][j] = sum_r W[r][j] (G^T x_hat)[r][j],
// the same triple sum reordered; no dZ GEMM is needed for it.
// With a LayerNorm bias b (z = x_hat * gain + b), Z = X_hat * gain + 1 b^T, so
//   dW[r][j]       += gsum[r] * b[j]               (gsum[r] = sum_n G[n][r])
//   part_b[s][j]    = sum_{r in slice s} W[r][j] * gsum[r]   (sums to d b)
// Rows are handled in parts of two blocks (32 slots, one row per lane after
// the reduce-scatter); the W loads of each 32-row block are issued while the
// previous block is processed.
template <typename T>
struct EpiWeightGrad {
  struct Params {
    float *dW;          // [N][ldw]
    int64_t ldw;
    const T *gain;      // [M] or NULL
    const T *W;         // [N][ldw] or NULL (no gain-gradient partials)
    float *part;        // [N / WN][ldw]
    int accumulate;
    const float *gsum;  // [N] with a bias, else NULL
    const T *bias;      // [M] or NULL
    float *part_b;      // [N / WN][ldw] with a bias
  };
  template <class Cfg>
  __device__ __forceinline__ static void apply(const Params &p, f32x16_t (&acc)[Cfg::MB][Cfg::NB], const TileCtx<Cfg> &t) {
    constexpr int NB = Cfg::NB, NPART = Cfg::MB / 2;
    const int lane = t.lane, lo = lane & 31, hw = lane >> 5;
    const int cbase = t.n0 + t.wave_n * Cfg::WN;
    const int64_t ct = cbase / Cfg::WN;
    const int rbase = t.m0 + t.wave_m * Cfg::WM + hw * 4;  // feature of the lane's slot 0
    const bool interior = t.m0 + Cfg::BM <= t.M && cbase + Cfg::WN <= t.N;
    // The tile's gain and bias as fp32 in LDS, so that the stores below do
    // not wait on a global load per group of four features (a line's four
    // pieces then reach L2 close together, rather than spread over several
    // load latencies during which it may be evicted half-written).
    float *gl = reinterpret_cast<float *>(t.smem);  // [BM] gain, [BM] bias
    __syncthreads();  // every wave is past its last fragment reads
    if (threadIdx.x < Cfg::BM) {
      const int r = min(t.m0 + static_cast<int>(threadIdx.x), t.M - 1);
      gl[threadIdx.x] = p.gain != nullptr ? to_f32(p.gain[r]) : 1.0f;
      gl[Cfg::BM + threadIdx.x] = p.bias != nullptr ? to_f32(p.bias[r]) : 0.0f;
    }
    __syncthreads();
    auto body = [&](auto IN_, auto W_, auto A_, auto B_, auto G_) EE_ALWAYS_INLINE {
      constexpr bool kIn = decltype(IN_)::value, kW = decltype(W_)::value, kAcc = decltype(A_)::value;
      constexpr bool kB = decltype(B_)::value, kG = decltype(G_)::value;
      int col[NB];
      bool cok[NB];
      float gs[NB];
      float *dcol[NB];      // dW[col][rbase]: group (I, Q) adds I*32 + Q*8
      const T *wcol[NB];    // W[col][rbase]
      static_for<NB>([&](auto j) EE_ALWAYS_INLINE {
        col[j] = t.col(j);
        cok[j] = kIn || col[j] < t.N;
        const int64_t o = static_cast<int64_t>(min(col[j], t.N - 1)) * p.ldw + rbase;
        dcol[j] = p.dW + o;
        wcol[j] = kW ? p.W + o : nullptr;
        gs[j] = kB ? p.gsum[min(col[j], t.N - 1)] : 0.0f;
      });
      // Offset of group (I, Q) from rbase, moved back into [0, M - 4] at the
      // problem's last rows (edge tiles only; such groups are not stored).
      auto goff = [&](int I, int Q) EE_ALWAYS_INLINE {
        const int o = I * 32 + Q * 8;
        return kIn ? o : min(o, t.M - 4 - rbase);
      };
      // W of one 32-row block, double-buffered: the block after the current
      // one is always in flight (two blocks of registers, no spills).
      Raw4<T> w[2][4][NB];
      auto load_w = [&](auto blk) EE_ALWAYS_INLINE {
        constexpr int I = decltype(blk)::value;
        if constexpr (kW && I < Cfg::MB) {
          static_for<4>([&](auto q) EE_ALWAYS_INLINE {
            const int o = goff(I, decltype(q)::value);
            static_for<NB>([&](auto j) EE_ALWAYS_INLINE { w[I % 2][decltype(q)::value][j] = raw4(wcol[j] + o); });
          });
        }
      };
      load_w(std::integral_constant<int, 0>{});
      static_for<NPART>([&](auto hf) EE_ALWAYS_INLINE {
        constexpr int H = decltype(hf)::value, I0 = H * 2;
        __builtin_amdgcn_sched_barrier(0);
        float dg[32], db[32];
        static_for<2>([&](auto ii) EE_ALWAYS_INLINE {
          constexpr int II = decltype(ii)::value, I = I0 + II;
          load_w(std::integral_constant<int, I + 1>{});
          static_for<4>([&](auto q) EE_ALWAYS_INLINE {
            constexpr int Q = decltype(q)::value;
            const int o = goff(I, Q);
            const bool rok = kIn || rbase + I * 32 + Q * 8 < t.M;
            const int lo4 = rbase - t.m0 + o;  // tile row of the group (o clamped at the problem's edge)
            const f32x4_t g4 = kG ? *reinterpret_cast<const f32x4_t *>(gl + lo4) : f32x4_t{1.0f, 1.0f, 1.0f, 1.0f};
            const f32x4_t b4 = kB ? *reinterpret_cast<const f32x4_t *>(gl + Cfg::BM + lo4) : f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
            f32x4_t sg = {0.0f, 0.0f, 0.0f, 0.0f}, sb = {0.0f, 0.0f, 0.0f, 0.0f};
            static_for<NB>([&](auto j) EE_ALWAYS_INLINE {
              const f32x4_t c = {acc[I][j][Q * 4], acc[I][j][Q * 4 + 1], acc[I][j][Q * 4 + 2], acc[I][j][Q * 4 + 3]};
              f32x4_t v = c * g4;
              if constexpr (kAcc) v += raw4(dcol[j] + o);
              if constexpr (kB) v += gs[j] * b4;
              if (cok[j] && rok) store4(dcol[j] + o, v);
              if constexpr (kW) {
                const f32x4_t wv = cvt4(w[I % 2][Q][j]);
                if (cok[j]) {
                  sg += wv * c;
                  if constexpr (kB) sb += wv * gs[j];
                }
              }
            });
            static_for<4>([&](auto e) EE_ALWAYS_INLINE {
              constexpr int K = II * 16 + Q * 4 + decltype(e)::value;
              dg[K] = sg[decltype(e)::value];
              db[K] = sb[decltype(e)::value];
            });
          });
        });
        if constexpr (kW) {
          slot_reduce_scatter<false>(dg, lane);
          if constexpr (kB) slot_reduce_scatter<false>(db, lane);
          const int row = t.m0 + t.wave_m * Cfg::WM + slot_row(I0 * 16 + lo, lane);
          if (cbase < t.N && row < t.M) {
            p.part[ct * p.ldw + row] = dg[0];
            if constexpr (kB) p.part_b[ct * p.ldw + row] = db[0];
          }
        }
      });
    };
    // A bias comes with W (the bias gradient needs W).
    with_flag(interior, [&](auto IN_) EE_ALWAYS_INLINE {
      with_flag(p.gain != nullptr, [&](auto G_) EE_ALWAYS_INLINE {
        with_flag(p.W != nullptr, [&](auto W_) EE_ALWAYS_INLINE {
          with_flag(p.accumulate != 0, [&](auto A_) EE_ALWAYS_INLINE {
            if constexpr (decltype(W_)::value)
              with_flag(p.bias != nullptr, [&](auto B_) EE_ALWAYS_INLINE { body(IN_, W_, A_, B_, G_); });
            else
              body(IN_, W_, A_, std::false_type{}, G_);
          });
        });
      });
    });
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

// Plain store in the element type, untransposed: C[row][col] (gate
// projection with tokens as rows: H_g[n][i]).  Lanes 0-31 of each store
// cover 32 consecutive columns of one row.
template <typename T>
struct EpiStore {
  struct Params {
    T *C;          // [M][ldc]
    int64_t ldc;
  };
  template <class Cfg>
  __device__ __forceinline__ static void apply(const Params &p, f32x16_t (&acc)[Cfg::MB][Cfg::NB], const TileCtx<Cfg> &t) {
    for_each_acc<Cfg>(acc, t, [&](int row, int col, int, float a) EE_ALWAYS_INLINE {
      if (row < t.M && col < t.N) p.C[static_cast<int64_t>(row) * p.ldc + col] = from_f32<T>(a);
    });
  }
};

// Down projection with the residual, untransposed (rows of C are tokens,
// columns features): Y[n][j] = X[n][j] + C[n][j]  (fp32 out; lanes 0-31 of a
// store write one 128-byte line).  With split K, slice z of the product goes
// to Y + z * zstride and only slice 0 adds X (the slices are partial sums
// the exit-norm statistics add).
template <typename T>
struct EpiResidual {
  struct Params {
    float *Y;       // [N][ld]
    const T *X;     // [N][ld]
    int64_t ld;
    int64_t zstride;
  };
  template <class Cfg>
  __device__ __forceinline__ static void apply(const Params &p, f32x16_t (&acc)[Cfg::MB][Cfg::NB], const TileCtx<Cfg> &t) {
    float *Y = p.Y + t.kz * p.zstride;
    if (t.kz == 0) {
      for_each_acc_loaded<Cfg>(
          acc, t, t.M, t.N,
          [&](int row, int col) EE_ALWAYS_INLINE { return p.X[static_cast<int64_t>(row) * p.ld + col]; },
          [&](int row, int col, int, float a, T x) EE_ALWAYS_INLINE {
            if (row < t.M && col < t.N) Y[static_cast<int64_t>(row) * p.ld + col] = a + to_f32(x);
          });
    } else {
      for_each_acc<Cfg>(acc, t, [&](int row, int col, int, float a) EE_ALWAYS_INLINE {
        if (row < t.M && col < t.N) Y[static_cast<int64_t>(row) * p.ld + col] = a;
      });
    }
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

// Backward of the SwiGLU product, untransposed (rows of C = dA = dY W_down
// are tokens, columns features i; lanes 0-31 of each access cover 32
// consecutive features of one token):
//   dH_g = dA * H_u * silu'(H_g),   dH_u = dA * silu(H_g).
template <typename T>
struct EpiSwiGLUBwd {
  struct Params {
    const T *Hg;   // [N][ld]
    const T *Hu;
    T *dHg;
    T *dHu;
    int64_t ld;
  };
  struct H2 {
    T g, u;
  };
  template <class Cfg>
  __device__ __forceinline__ static void apply(const Params &p, f32x16_t (&acc)[Cfg::MB][Cfg::NB], const TileCtx<Cfg> &t) {
    for_each_acc_loaded<Cfg>(
        acc, t, t.M, t.N,
        [&](int row, int col) EE_ALWAYS_INLINE {
          const int64_t o = static_cast<int64_t>(row) * p.ld + col;
          return H2{p.Hg[o], p.Hu[o]};
        },
        [&](int row, int col, int, float da, H2 h) EE_ALWAYS_INLINE {
          if (row < t.M && col < t.N) {
            const int64_t o = static_cast<int64_t>(row) * p.ld + col;
            float sv, sg;
            silu_and_grad(to_f32(h.g), sv, sg);
            p.dHg[o] = from_f32<T>(da * to_f32(h.u) * sg);
            p.dHu[o] = from_f32<T>(da * sv);
          }
        });
  }
};

}  // namespace ee
