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

// The first butterfly step of the reductions below, over lane bit 4, for
// H slot pairs (K, K + H): lanes with the bit clear keep slot K, the others
// slot K + H, each combined with its partner's value of the same slot.  One
// v_permlane16_swap per pair exchanges exactly those two values (the
// partner's copy of the kept slot lands in the other register), so no lane
// selects what to send: v[K] = op(first, second) in either half.
template <bool IsMax, int H, int N>
__device__ __forceinline__ void slot_step_bit4(float (&v)[N]) {
  static_for<H>([&](auto kk) EE_ALWAYS_INLINE {
    constexpr int K = decltype(kk)::value;
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v[K]), __float_as_uint(v[K + H]), false, false);
    const float a = __uint_as_float(r[0]), b = __uint_as_float(r[1]);
    v[K] = IsMax ? fmaxf(a, b) : a + b;
  });
}

// Reduce-scatter of N row slots over the 32 lanes that share them: five
// butterfly steps (lane bits 4..0), each halving the values a lane keeps, so
// N/2 + N/4 + ... + N/32 shuffles instead of 5 N.  On return v[x], x < N/32,
// is the total (sum or max) of slot base + (N/32) * (lane % 32) + x, where
// the caller's slots are base .. base + N - 1.
template <bool IsMax, int N>
__device__ __forceinline__ void slot_reduce_scatter(float (&v)[N], int lane) {
  static_assert(N >= 32 && (N & (N - 1)) == 0, "slots must be a power of two >= 32");
  slot_step_bit4<IsMax, N / 2>(v);
  static_for<4>([&](auto st0) EE_ALWAYS_INLINE {
    constexpr int S = decltype(st0)::value + 1;
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

// Sum of 16 row slots (one 32-row block) over the 32 lanes that share them:
// four halving exchanges (lane bits 4..1) and a full one over bit 0, after
// which v[0] of lanes 2 s and 2 s + 1 of each half-wave is the total of
// slot s.
__device__ __forceinline__ void slot_reduce16(float (&v)[16], int lane) {
  slot_step_bit4<false, 8>(v);
  static_for<3>([&](auto st0) EE_ALWAYS_INLINE {
    constexpr int S = decltype(st0)::value + 1;
    constexpr int BIT = 4 - S, H = 8 >> S;
    const bool hi = (lane >> BIT) & 1;
    static_for<H>([&](auto kk) EE_ALWAYS_INLINE {
      constexpr int K = decltype(kk)::value;
      const float send = hi ? v[K] : v[K + H];
      const float keep = hi ? v[K + H] : v[K];
      v[K] = keep + __shfl_xor(send, 1 << BIT);
    });
  });
  v[0] += __shfl_xor(v[0], 1);
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
// of the logits that reaches memory) at P[v][n], tokens contiguous, and
// captures the fp32 logit of each token's target (next-token NLL, Sec. 2).
// With shift0 the store and the sums take no shift at all, P = exp(S) and
// l = sum_v exp(S): the form in which the weight-gradient GEMM can use P as
// it is (see the cross-entropy reduce); m, then needed only for the
// confidence of dynamic token weights, is computed and stored only if
// shift0 == 1 (2: no maxima at all).  Rows are handled in parts of two
// blocks (32 slots), each reduced over the wave's columns by a
// reduce-scatter (one row per lane) and, for the shifted form, broadcast
// back through the wave's own LDS rows.  A part's 64 tokens are one 128-byte
// line of a bf16 P row: in bf16 the part's P values pass through 8 KB of
// the wave's LDS ([64 vocab ids][64 tokens], 16-byte chunks XOR-swizzled by
// the vocab id) and leave in whole lines, eight lanes per line (a lane's own
// four tokens would touch 32 lines per store); fp32 P is stored directly,
// four tokens per 16-byte store.  Token columns past M up to ldp may be
// written with finite values (the seed zeroes them).
template <typename T>
struct EpiLogits {
  struct Params {
    T *P;               // [V][ldp]
    int64_t ldp;        // padded token count (multiple of 8)
    float *part_m;      // [V / WN][ldp]
    float *part_l;      // [V / WN][ldp]
    float *tgt;         // [ldp] target logit
    const int32_t *targets;
    int shift0;         // 1, 2: P = exp(S) instead of exp(S - m); 2: and no maxima
  };
  template <class Cfg>
  __device__ __forceinline__ static void apply(const Params &p, f32x16_t (&acc)[Cfg::MB][Cfg::NB], const TileCtx<Cfg> &t) {
    constexpr int NB = Cfg::NB, NPART = Cfg::MB / 2;  // parts of two blocks
    constexpr float kLog2e = 1.4426950408889634f;
    constexpr bool kStage = std::is_same<T, bf16_t>::value;
    constexpr int kStageOff = 8192;  // after the targets and the row broadcasts
    static_assert((Cfg::BM + Cfg::THREADS / 64 * Cfg::WM) * 4 <= kStageOff, "broadcast rows fit below the staging");
    static_assert(!kStage || (Cfg::WN == 64 && kStageOff + Cfg::THREADS / 64 * 8192 <= 2 * Cfg::STAGE_BYTES),
                  "8 KB of staging per wave");
    const int lane = t.lane, lo = lane & 31, hw = lane >> 5;
    const int wave = t.wave_m * Cfg::WAVES_N + t.wave_n;
    int *ylds = reinterpret_cast<int *>(t.smem);                                   // [BM] tile tokens' targets
    float *wl = reinterpret_cast<float *>(t.smem) + Cfg::BM + wave * Cfg::WM;     // this wave's rows
    char *stage = t.smem + kStageOff + wave * 8192;                               // this wave's P lines
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
    auto shift_modes = [&](auto &&f) EE_ALWAYS_INLINE {
      if (p.shift0 == 0)
        f(std::false_type{}, std::true_type{});
      else if (p.shift0 == 1)
        f(std::true_type{}, std::true_type{});
      else
        f(std::true_type{}, std::false_type{});
    };
    shift_modes([&](auto S0_, auto MX_) EE_ALWAYS_INLINE {
    with_flag(interior, [&](auto IN_) EE_ALWAYS_INLINE {
      constexpr bool kIn = decltype(IN_)::value, kShift0 = decltype(S0_)::value, kMax = decltype(MX_)::value;
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
        if constexpr (kMax) {
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
        }
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
        if constexpr (kMax) slot_reduce_scatter<true>(mx, lane);
        if constexpr (!kShift0) {
          wl[slot_row(I0 * 16 + lo, lane)] = mx[0];
          // the rows read back below are this wave's own: a wave-scope fence
          // suffices (the other waves go on with their parts)
          __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
          __builtin_amdgcn_wave_barrier();
          __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        }
        // P = exp(S - m) = exp2(S log2e - m log2e) (m = 0 with shift0), four
        // tokens per store; row sums
        static_for<2>([&](auto ii) EE_ALWAYS_INLINE {
          constexpr int I = I0 + decltype(ii)::value;
          static_for<4>([&](auto q) EE_ALWAYS_INLINE {
            constexpr int Q = decltype(q)::value;
            const f32x4_t ml = kShift0 ? f32x4_t{0.0f, 0.0f, 0.0f, 0.0f}
                                       : *reinterpret_cast<const f32x4_t *>(wl + I * 32 + Q * 8 + hw * 4) * kLog2e;
            const bool rok = kIn || t.m0 + rbase + I * 32 + Q * 8 < t.M;
            f32x4_t s4 = {0.0f, 0.0f, 0.0f, 0.0f};
            static_for<NB>([&](auto j) EE_ALWAYS_INLINE {
              f32x4_t e4;
              static_for<4>([&](auto e) EE_ALWAYS_INLINE {
                constexpr int E = decltype(e)::value;
                const float x = __builtin_amdgcn_exp2f(fmaf(acc[I][j][Q * 4 + E], kLog2e, -ml[E]));
                e4[E] = cok[j] ? x : 0.0f;
              });
              if constexpr (kStage) {
                // vocab id fw = j * 32 + lane % 32 of the wave, tokens 32 ii + 8 Q + 4 hw + 0..3
                const int fw = decltype(j)::value * 32 + lo;
                store4(reinterpret_cast<T *>(stage + fw * 128 + (((decltype(ii)::value * 4 + Q) ^ (fw & 7)) << 4) + hw * 8),
                       e4);
              } else if (cok[j] && rok) {
                store4(pcol[j] + (I * 32 + Q * 8), e4);
              }
              s4 += e4;
            });
            static_for<4>([&](auto e) EE_ALWAYS_INLINE {
              sm[decltype(ii)::value * 16 + Q * 4 + decltype(e)::value] = s4[decltype(e)::value];
            });
          });
        });
        if constexpr (kStage) {
          // the lines read back are this wave's own: a wave-scope fence suffices
          __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
          __builtin_amdgcn_wave_barrier();
          __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
          const int tok0 = t.m0 + t.wave_m * Cfg::WM + I0 * 32;  // the part's first token
          static_for<8>([&](auto it) EE_ALWAYS_INLINE {
            const int c = decltype(it)::value * 64 + lane;  // chunk: vocab id c / 8, tokens 8 (c % 8) ..
            const int fw = c >> 3, k = c & 7;
            const u32x4_t v = *reinterpret_cast<const u32x4_t *>(stage + fw * 128 + ((k ^ (fw & 7)) << 4));
            const int col = cbase + fw, tok = tok0 + k * 8;
            if (col < t.N && tok < p.ldp) *reinterpret_cast<u32x4_t *>(p.P + static_cast<int64_t>(col) * p.ldp + tok) = v;
          });
          // the next part overwrites the staging lines
          __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
          __builtin_amdgcn_wave_barrier();
          __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        }
        slot_reduce_scatter<false>(sm, lane);
        const int row = t.m0 + t.wave_m * Cfg::WM + slot_row(I0 * 16 + lo, lane);
        if (cbase < t.N && row < t.M) {
          if constexpr (kMax) p.part_m[ct * p.ldp + row] = mx[0];
          p.part_l[ct * p.ldp + row] = sm[0];
        }
      });
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
// Rows are handled one 32-row block (16 slots) at a time; its partials are
// reduced over the wave's columns by slot_reduce16.  A block's 32 features
// are one 128-byte line of a dW row: each block's dW values pass through 8
// KB of the wave's LDS ([64 output rows][32 features], 16-byte chunks
// XOR-swizzled by the row) and leave in whole lines, eight lanes per line
// (a lane's own four features would touch 32 lines per store), after the
// block's W loads have been consumed, so no store waits on a load.
template <typename T>
struct EpiWeightGrad {
  static constexpr bool kPersistent = true;  // launch_gemm runs it as one block per CU looping over the tiles
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
    constexpr int NB = Cfg::NB;
    const int lane = t.lane, lo = lane & 31, hw = lane >> 5;
    const int cbase = t.n0 + t.wave_n * Cfg::WN;
    const int64_t ct = cbase / Cfg::WN;
    const int rbase = t.m0 + t.wave_m * Cfg::WM + hw * 4;  // feature of the lane's slot 0
    const bool interior = t.m0 + Cfg::BM <= t.M && cbase + Cfg::WN <= t.N;
    constexpr int kStageOff = 8192;  // after the gain and bias
    static_assert(2 * Cfg::BM * 4 <= kStageOff && Cfg::WN == 64 &&
                      kStageOff + Cfg::THREADS / 64 * 8192 <= 2 * Cfg::STAGE_BYTES,
                  "8 KB of staging per wave");
    char *stage = t.smem + kStageOff + (t.wave_m * Cfg::WAVES_N + t.wave_n) * 8192;  // this wave's dW lines
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
      const T *wcol[NB];    // W[col][rbase]: group (I, Q) adds I*32 + Q*8
      static_for<NB>([&](auto j) EE_ALWAYS_INLINE {
        col[j] = t.col(j);
        cok[j] = kIn || col[j] < t.N;
        const int64_t o = static_cast<int64_t>(min(col[j], t.N - 1)) * p.ldw + rbase;
        wcol[j] = kW ? p.W + o : nullptr;
        gs[j] = kB ? p.gsum[min(col[j], t.N - 1)] : 0.0f;
      });
      // Offset of group (I, Q) from rbase, moved back into [0, M - 4] at the
      // problem's last rows (edge tiles only; such groups are not stored).
      auto goff = [&](int I, int Q) EE_ALWAYS_INLINE {
        const int o = I * 32 + Q * 8;
        return kIn ? o : min(o, t.M - 4 - rbase);
      };
      // W of one 32-row block, loaded as the block starts (the dW lines
      // leave through LDS afterwards, so no store waits on these loads).
      // fp32: four 16-byte loads per column, one per group of four features.
      // bf16: two 16-byte loads per column, eight features each: in load g
      // the half-waves take features 16 g + 8 hw .. + 7 of the block, and
      // one exchange between the half-waves (v_permlane32_swap) leaves each
      // lane its own four features of groups 2 g and 2 g + 1.
      Raw4<T> w[4][NB];
      auto load_w = [&](auto blk) EE_ALWAYS_INLINE {
        constexpr int I = decltype(blk)::value;
        if constexpr (kW && std::is_same<T, bf16_t>::value) {
          static_for<2>([&](auto g) EE_ALWAYS_INLINE {
            constexpr int G = decltype(g)::value;
            // wcol includes this lane's 4 hw; edge blocks clamp into [0, M - 8]
            const int o = kIn ? I * 32 + G * 16 + hw * 4 : min(I * 32 + G * 16 + hw * 4, t.M - 8 - rbase);
            static_for<NB>([&](auto j) EE_ALWAYS_INLINE {
              const u32x4_t v = *reinterpret_cast<const u32x4_t *>(wcol[j] + o);
              const auto s0 = __builtin_amdgcn_permlane32_swap(v[0], v[2], false, false);
              const auto s1 = __builtin_amdgcn_permlane32_swap(v[1], v[3], false, false);
              w[2 * G][j] = u32x2_t{s0[0], s1[0]};
              w[2 * G + 1][j] = u32x2_t{s0[1], s1[1]};
            });
          });
        } else if constexpr (kW) {
          static_for<4>([&](auto q) EE_ALWAYS_INLINE {
            const int o = goff(I, decltype(q)::value);
            static_for<NB>([&](auto j) EE_ALWAYS_INLINE { w[decltype(q)::value][j] = raw4(wcol[j] + o); });
          });
        }
      };
      static_for<Cfg::MB>([&](auto blk) EE_ALWAYS_INLINE {
        constexpr int I = decltype(blk)::value;
        __builtin_amdgcn_sched_barrier(0);
        float dg[16], db[16];
        {
          load_w(std::integral_constant<int, I>{});
          static_for<4>([&](auto q) EE_ALWAYS_INLINE {
            constexpr int Q = decltype(q)::value;
            const int o = goff(I, Q);
            const int lo4 = rbase - t.m0 + o;  // tile row of the group (o clamped at the problem's edge)
            const f32x4_t g4 = kG ? *reinterpret_cast<const f32x4_t *>(gl + lo4) : f32x4_t{1.0f, 1.0f, 1.0f, 1.0f};
            const f32x4_t b4 = kB ? *reinterpret_cast<const f32x4_t *>(gl + Cfg::BM + lo4) : f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
            f32x4_t sg = {0.0f, 0.0f, 0.0f, 0.0f}, sb = {0.0f, 0.0f, 0.0f, 0.0f};
            static_for<NB>([&](auto j) EE_ALWAYS_INLINE {
              const f32x4_t c = {acc[I][j][Q * 4], acc[I][j][Q * 4 + 1], acc[I][j][Q * 4 + 2], acc[I][j][Q * 4 + 3]};
              // output row fw = j * 32 + lane % 32 of the wave, features 8 Q + 4 hw + 0..3 of the block
              const int fw = decltype(j)::value * 32 + lo;
              *reinterpret_cast<f32x4_t *>(stage + fw * 128 + (((Q * 2 + hw) ^ (fw & 7)) << 4)) = c * g4;
              if constexpr (kW) {
                const f32x4_t wv = cvt4(w[Q][j]);
                if (cok[j]) {
                  sg += wv * c;
                  if constexpr (kB) sb += wv * gs[j];
                }
              }
            });
            static_for<4>([&](auto e) EE_ALWAYS_INLINE {
              constexpr int K = Q * 4 + decltype(e)::value;
              dg[K] = sg[decltype(e)::value];
              db[K] = sb[decltype(e)::value];
            });
          });
          // the block's lines: read back (this wave's own rows, so a
          // wave-scope fence suffices), add what accumulates, store
          __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
          __builtin_amdgcn_wave_barrier();
          __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
          const int fbase = t.m0 + t.wave_m * Cfg::WM + I * 32;  // the block's first feature
          const int fb = kIn ? fbase : min(fbase, t.M - 32);      // (M is a multiple of 32)
          static_for<8>([&](auto it) EE_ALWAYS_INLINE {
            // two rounds of four chunks per lane (registers)
            if constexpr (decltype(it)::value == 4) __builtin_amdgcn_sched_barrier(0);
            const int c = decltype(it)::value * 64 + lane;  // chunk: output row c / 8, features 4 (c % 8) ..
            const int fw = c >> 3, k = c & 7;
            f32x4_t v = *reinterpret_cast<const f32x4_t *>(stage + fw * 128 + ((k ^ (fw & 7)) << 4));
            const int colw = cbase + fw;
            float *dst = p.dW + static_cast<int64_t>(kIn ? colw : min(colw, t.N - 1)) * p.ldw + fb + k * 4;
            if constexpr (kAcc) v += raw4(dst);
            if constexpr (kB) {
              const f32x4_t bb = *reinterpret_cast<const f32x4_t *>(gl + Cfg::BM + (fb - t.m0) + k * 4);
              v += p.gsum[kIn ? colw : min(colw, t.N - 1)] * bb;
            }
            if (kIn || (colw < t.N && fbase < t.M)) store4(dst, v);
          });
          // the next block overwrites the staging rows
          __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
          __builtin_amdgcn_wave_barrier();
          __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        }
        if constexpr (kW) {
          slot_reduce16(dg, lane);
          if constexpr (kB) slot_reduce16(db, lane);
          const int row = t.m0 + t.wave_m * Cfg::WM + slot_row(I * 16 + (lo >> 1), lane);
          if (cbase < t.N && row < t.M && (lo & 1) == 0) {
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

// H_g and H_u of one token and feature side by side in one word (bf16) or
// two (fp32): what the SwiGLU backward loads per element.
template <typename T> struct GatePair;
template <> struct GatePair<bf16_t> {
  using type = uint32_t;
  __device__ __forceinline__ static type make(bf16_t g, bf16_t u) {
    return static_cast<uint32_t>(g) | (static_cast<uint32_t>(u) << 16);
  }
  __device__ __forceinline__ static float g(type v) { return __uint_as_float(v << 16); }
  __device__ __forceinline__ static float u(type v) { return __uint_as_float(v & 0xFFFF0000u); }
};
template <> struct GatePair<float> {
  typedef float type __attribute__((ext_vector_type(2)));
  __device__ __forceinline__ static type make(float g, float u) { return type{g, u}; }
  __device__ __forceinline__ static float g(type v) { return v[0]; }
  __device__ __forceinline__ static float u(type v) { return v[1]; }
};

// Gate and up projections as one product, with the SwiGLU product.  The B
// operand interleaves the rows of W_gate and W_up in blocks of 32
// (KMajorPairLoader; C has 2F columns for F features), so a lane's two
// column blocks hold H_g and H_u of the same tokens and feature
// f = n0 / 2 + wave_n * 32 + lane % 32.  Stores, token-major, the pair
// (H_g, H_u) at Hgu[n][f] and A = silu(H_g) * H_u at A[n][f], with H_g
// rounded to the element type before the SiLU (the value the backward
// reads); lanes 0-31 of each store cover 32 consecutive features of one
// token.
template <typename T>
struct EpiGateUp {
  static constexpr bool kPairB = true;
  using Pair = GatePair<T>;
  struct Params {
    typename Pair::type *Hgu;  // [M][F]
    T *A;                      // [M][F]
  };
  template <class Cfg>
  __device__ __forceinline__ static void apply(const Params &p, f32x16_t (&acc)[Cfg::MB][Cfg::NB], const TileCtx<Cfg> &t) {
    static_assert(Cfg::NB == 2 && Cfg::WN == 64, "one 32-column block of each matrix per wave");
    const int F = t.N / 2;
    const int f = t.n0 / 2 + t.wave_n * 32 + (t.lane & 31);
    if (f >= F) return;  // (no barrier follows)
    static_for<Cfg::MB>([&](auto i) EE_ALWAYS_INLINE {
      static_for<16>([&](auto v) EE_ALWAYS_INLINE {
        constexpr int I = decltype(i)::value, V = decltype(v)::value;
        const int row = t.row(I, V);
        if (row < t.M) {
          const int64_t o = static_cast<int64_t>(row) * F + f;
          const T hg = from_f32<T>(acc[I][0][V]);
          const float hu = acc[I][1][V];
          p.Hgu[o] = Pair::make(hg, from_f32<T>(hu));
          p.A[o] = from_f32<T>(silu_f(to_f32(hg)) * hu);
        }
      });
    });
  }
};

// Backward of the SwiGLU product (rows of C = dA = dY W_down are tokens,
// columns features i):
//   dH_g = dA * H_u * silu'(H_g),   dH_u = dA * silu(H_g),
// with (H_g, H_u) read token-major as EpiGateUp stores them (lanes 0-31 of
// each load cover 32 consecutive features of one token) and dH_g, dH_u
// stored transposed, [feature][ldt] with tokens contiguous: the K-major
// operands of the gate and up weight gradients.  Token columns M..ldt-1 are
// written as zeros.  The wave's 32-row blocks go in pairs (64 tokens = one
// 128-byte line of a bf16 feature row): both blocks' loads, then their
// results.  In bf16 the results pass through the wave's 16 KB of the tile's
// LDS ([output][64 features][64 tokens], 16-byte chunks XOR-swizzled by the
// feature), so that every global store writes whole lines, eight lanes per
// line; a lane's own four consecutive tokens (8 bytes) would touch 32 lines
// per store.  fp32 results (16 bytes per lane) are stored directly.
template <typename T>
struct EpiSwiGLUBwd {
  using Pair = GatePair<T>;
  struct Params {
    const typename Pair::type *Hgu;  // [M][ld]
    T *dHgT;                         // [N][ldt]
    T *dHuT;
    int64_t ld;
    int64_t ldt;                     // multiple of 64, >= M
  };
  template <class Cfg>
  __device__ __forceinline__ static void apply(const Params &p, f32x16_t (&acc)[Cfg::MB][Cfg::NB], const TileCtx<Cfg> &t) {
    constexpr int NB = Cfg::NB;
    constexpr bool kStage = std::is_same<T, bf16_t>::value;
    static_assert(Cfg::MB % 2 == 0, "blocks go in pairs");
    static_assert(!kStage || (Cfg::WN == 64 && Cfg::THREADS / 64 * 16384 <= 2 * Cfg::STAGE_BYTES),
                  "16 KB of staging per wave");
    const int wave = t.wave_m * Cfg::WAVES_N + t.wave_n;
    char *stage = t.smem + wave * 16384;
    if constexpr (kStage) __syncthreads();  // every wave is past its last fragment reads
    int col[NB];
    static_for<NB>([&](auto j) EE_ALWAYS_INLINE { col[j] = t.col(j); });
    static_for<Cfg::MB / 2>([&](auto pp) EE_ALWAYS_INLINE {
      constexpr int I0 = 2 * decltype(pp)::value;
      typename Pair::type pre[2][16][NB];
      static_for<2>([&](auto ii) EE_ALWAYS_INLINE {
        static_for<16>([&](auto v) EE_ALWAYS_INLINE {
          const int row = min(t.row(I0 + decltype(ii)::value, decltype(v)::value), t.M - 1);
          static_for<NB>([&](auto j) EE_ALWAYS_INLINE {
            pre[decltype(ii)::value][decltype(v)::value][j] =
                p.Hgu[static_cast<int64_t>(row) * p.ld + min(col[j], t.N - 1)];
          });
        });
      });
      static_for<2>([&](auto ii) EE_ALWAYS_INLINE {
        constexpr int I = I0 + decltype(ii)::value;
        static_for<4>([&](auto q) EE_ALWAYS_INLINE {
          constexpr int Q = decltype(q)::value;
          const int r0 = t.row(I, Q * 4);  // rows r0 .. r0 + 3
          static_for<NB>([&](auto j) EE_ALWAYS_INLINE {
            f32x4_t dg, du;
            static_for<4>([&](auto e) EE_ALWAYS_INLINE {
              constexpr int E = decltype(e)::value;
              const auto h = pre[decltype(ii)::value][Q * 4 + E][j];
              float sv, sg;
              silu_and_grad(Pair::g(h), sv, sg);
              const float da = acc[I][j][Q * 4 + E];
              const bool ok = r0 + E < t.M;
              dg[E] = ok ? da * Pair::u(h) * sg : 0.0f;
              du[E] = ok ? da * sv : 0.0f;
            });
            if constexpr (kStage) {
              // feature fw = j * 32 + lane % 32 of the wave, tokens 32 ii + 8 Q + 4 (lane / 32) + 0..3
              const int fw = j * 32 + (t.lane & 31);
              const int off = fw * 128 + (((decltype(ii)::value * 4 + Q) ^ (fw & 7)) << 4) + (t.lane >> 5) * 8;
              store4(reinterpret_cast<T *>(stage + off), dg);
              store4(reinterpret_cast<T *>(stage + 8192 + off), du);
            } else if (r0 < p.ldt && col[j] < t.N) {
              const int64_t o = static_cast<int64_t>(col[j]) * p.ldt + r0;
              store4(p.dHgT + o, dg);
              store4(p.dHuT + o, du);
            }
          });
        });
      });
      if constexpr (kStage) {
        // the rows read back are this wave's own: a wave-scope fence suffices
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        const int tok0 = t.m0 + t.wave_m * Cfg::WM + I0 * 32;  // first token of the pair
        static_for<2>([&](auto o) EE_ALWAYS_INLINE {
          T *out = decltype(o)::value == 0 ? p.dHgT : p.dHuT;
          static_for<8>([&](auto it) EE_ALWAYS_INLINE {
            const int c = decltype(it)::value * 64 + t.lane;  // chunk: feature c / 8, tokens 8 (c % 8) ..
            const int fw = c >> 3, k = c & 7;
            const u32x4_t v =
                *reinterpret_cast<const u32x4_t *>(stage + decltype(o)::value * 8192 + fw * 128 + ((k ^ (fw & 7)) << 4));
            const int f = t.n0 + t.wave_n * Cfg::WN + fw;
            const int tok = tok0 + k * 8;
            if (f < t.N && tok < p.ldt)
              *reinterpret_cast<u32x4_t *>(out + static_cast<int64_t>(f) * p.ldt + tok) = v;
          });
        });
        // the next pair overwrites the staging rows
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      }
    });
  }
};

}  // namespace ee
