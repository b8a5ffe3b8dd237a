// Decode-time exit head (Sec. 3 "Inference": greedy decoding with a
// confidence-based exit): a handful of rows through one exit, forward only.
//
// At decode the products are skinny, C[r][j] = sum_k W[r][k] Z[j][k] with
// a weight W of R rows and only B <= 32 token rows Z per pass, so they are
// bound by streaming W from HBM once.  A block owns 32 rows of W (64 for
// a wide W past 8 token rows, so that each token fragment serves two row
// groups and the token rows' share of the loads halves); each of its waves takes a share
// of K and reads its rows straight into MFMA A fragments (16 bytes of K per
// lane), 12 fragments per row group in flight per lane, with no LDS staging;
// the token rows come from L2 as B fragments (tokens past B re-read row B-1
// and their outputs are dropped).  The waves' partial sums meet in LDS in a
// fixed order and the first wave runs the epilogue.  Splitting K gives about
// 4000 waves at V = 32000, enough loads in flight on every CU.  bf16 uses
// v_mfma_f32_32x32x16_bf16, fp32 v_mfma_f32_32x32x2_f32 over the same
// 16-byte loads.
//
// Epilogues: store (gate projection), SwiGLU (up projection), residual
// (down projection) and, for the output matrix, per-wave softmax partials:
// for each token the maximum logit over the wave's rows, the lowest row
// reaching it and sum exp(S - max).  decide_kernel combines the partials
// of all waves into the greedy token, its probability and the exit flag.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "ee_device.h"
#include "launch.h"

namespace ee {

namespace {

constexpr int kDecRows = 32;    // rows of W per row group (one MFMA tile)
constexpr int kDecTokens = 32;  // token rows per pass (grid.y walks more)
// Waves per block (each a share of K): 4 when the rows give at least two
// blocks per CU of a 256-CU GPU, else 8 or 16, so that narrow products (the
// MLP's down projection: 5120 rows, K = 13824) still keep enough loads in
// flight.  A shape-only rule, so results do not depend on the device.
constexpr int kDecWavesMax = 16;
__host__ __device__ constexpr int dec_waves(int row_blocks) {
  return row_blocks >= 512 ? 4 : (row_blocks >= 256 ? 8 : 16);
}
constexpr int kDecGroup = 12;   // fragment loads per operand per lane in flight (8 and 16 measured slower)

template <typename T> struct DecFrag;
// bf16: a 16-byte load holds 8 values of K; one MFMA consumes 16 (two lane halves).
template <> struct DecFrag<bf16_t> {
  static constexpr int K_PER_LOAD = 16;  // values of K covered by one load across the wave
  __device__ __forceinline__ static void mma(const u32x4_t &a, const u32x4_t &b, f32x16_t &acc) {
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                  acc, 0, 0, 0);
  }
};
// fp32: a 16-byte load holds 4 values of K; four MFMAs of K = 2 (lane halves
// hold K offsets 0-3 and 4-7 of the same 8, in the same order for A and B).
template <> struct DecFrag<float> {
  static constexpr int K_PER_LOAD = 8;
  __device__ __forceinline__ static void mma(const u32x4_t &a, const u32x4_t &b, f32x16_t &acc) {
    static_for<4>([&](auto e) EE_ALWAYS_INLINE {
      constexpr int E = decltype(e)::value;
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a[E]), __uint_as_float(b[E]), acc, 0, 0, 0);
    });
  }
};

// acc[v] of lane l: row r0 + (v/4)*8 + (l/32)*4 + v%4, token j0 + l%32.
__device__ __forceinline__ int dec_row(int r0, int lane, int v) {
  return r0 + (v >> 2) * 8 + (lane >> 5) * 4 + (v & 3);
}

template <typename T, class Epi, int kDecWaves, int RG>
__global__ __launch_bounds__(64 * kDecWaves) void skinny_kernel(const T *__restrict__ W, int64_t ldw, int R,
                                                                const T *__restrict__ Z, int64_t ldz, int B, int K,
                                                                typename Epi::Params ep) {
  constexpr int KL = DecFrag<T>::K_PER_LOAD;
  constexpr int PER_LOAD = 16 / sizeof(T);  // elements of one 16-byte load
  __shared__ f32x16_t red[kDecWaves - 1][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r0 = blockIdx.x * kDecRows * RG, j0 = blockIdx.y * kDecTokens;
  const int zr = min(j0 + (lane & 31), B - 1);
  const int koff = (lane >> 5) * PER_LOAD;
  const char *wp[RG];
  static_for<RG>([&](auto g) EE_ALWAYS_INLINE {
    constexpr int G = decltype(g)::value;
    const int wr = min(r0 + G * kDecRows + (lane & 31), R - 1);
    wp[G] = reinterpret_cast<const char *>(W + static_cast<int64_t>(wr) * ldw + koff);
  });
  const char *zp = reinterpret_cast<const char *>(Z + static_cast<int64_t>(zr) * ldz + koff);
  f32x16_t acc[RG];
  static_for<RG>([&](auto g) EE_ALWAYS_INLINE {
    static_for<16>([&](auto v) EE_ALWAYS_INLINE { acc[decltype(g)::value][decltype(v)::value] = 0.0f; });
  });

  // This wave's share of K, in whole groups of 4 loads (K is a multiple of
  // 4 KL): groups [g0, g1) of the K / (4 KL) groups.  Each token fragment
  // serves the RG row groups of the block.
  constexpr int KG4 = 4 * KL;
  const int groups = K / KG4;
  const int g0 = wave * groups / kDecWaves, g1 = (wave + 1) * groups / kDecWaves;
  int k = g0 * KG4;
  const int kend = g1 * KG4;
  auto step = [&](auto nq) EE_ALWAYS_INLINE {
    constexpr int NQ = decltype(nq)::value;
    u32x4_t a[RG][NQ], b[NQ];
    static_for<NQ>([&](auto q) EE_ALWAYS_INLINE {
      constexpr int Q = decltype(q)::value;
      const int64_t off = (static_cast<int64_t>(k) + Q * KL) * sizeof(T);
      static_for<RG>([&](auto g) EE_ALWAYS_INLINE {
        a[decltype(g)::value][Q] = *reinterpret_cast<const u32x4_t *>(wp[decltype(g)::value] + off);
      });
      b[Q] = *reinterpret_cast<const u32x4_t *>(zp + off);
    });
    // Keep every load of the group ahead of the MFMAs: left alone, the
    // scheduler would trade loads in flight for registers.
    __builtin_amdgcn_sched_barrier(0);
    static_for<NQ>([&](auto q) EE_ALWAYS_INLINE {
      static_for<RG>([&](auto g) EE_ALWAYS_INLINE {
        DecFrag<T>::mma(a[decltype(g)::value][decltype(q)::value], b[decltype(q)::value], acc[decltype(g)::value]);
      });
    });
  };
  constexpr int KG = kDecGroup * KL;
  for (; k + KG <= kend; k += KG) step(std::integral_constant<int, kDecGroup>{});
  for (; k < kend; k += KG4) step(std::integral_constant<int, 4>{});
  // Per row group: partial sums of waves 1.. to LDS; wave 0 adds them in
  // order and finishes.
  static_for<RG>([&](auto g) EE_ALWAYS_INLINE {
    constexpr int G = decltype(g)::value;
    if (G > 0) __syncthreads();  // wave 0 has read the previous group
    if (wave > 0) red[wave - 1][lane] = acc[G];
    __syncthreads();
    if (wave == 0 && r0 + G * kDecRows < R) {  // a second group may lie past the last row
      f32x16_t c = acc[G];
      static_for<kDecWaves - 1>([&](auto w) EE_ALWAYS_INLINE { c += red[decltype(w)::value][lane]; });
      Epi::apply(ep, c, r0 + G * kDecRows, j0, lane, R, B);
    }
  });
}

// Four consecutive rows of one token as fp32 (bf16 or fp32 storage).
template <typename T> __device__ __forceinline__ f32x4_t dload4(const T *p);
template <> __device__ __forceinline__ f32x4_t dload4<float>(const float *p) {
  return *reinterpret_cast<const f32x4_t *>(p);
}
template <> __device__ __forceinline__ f32x4_t dload4<bf16_t>(const bf16_t *p) {
  const u32x2_t u = *reinterpret_cast<const u32x2_t *>(p);
  return f32x4_t{__uint_as_float(u[0] << 16), __uint_as_float(u[0] & 0xFFFF0000u), __uint_as_float(u[1] << 16),
                 __uint_as_float(u[1] & 0xFFFF0000u)};
}
template <typename T> __device__ __forceinline__ void dstore4(T *p, f32x4_t v);
template <> __device__ __forceinline__ void dstore4<float>(float *p, f32x4_t v) {
  *reinterpret_cast<f32x4_t *>(p) = v;
}
template <> __device__ __forceinline__ void dstore4<bf16_t>(bf16_t *p, f32x4_t v) {
  const u32x2_t u = {static_cast<uint32_t>(f32_to_bf16(v[0])) | (static_cast<uint32_t>(f32_to_bf16(v[1])) << 16),
                     static_cast<uint32_t>(f32_to_bf16(v[2])) | (static_cast<uint32_t>(f32_to_bf16(v[3])) << 16)};
  *reinterpret_cast<u32x2_t *>(p) = u;
}

// f(row0, token, vals) for each group of 4 consecutive rows of the lane
// (rows are feature indices, a multiple of 4 apart from the tile origin;
// R is a multiple of 64 for the MLP products that use this).
template <class F>
__device__ __forceinline__ void for_rows4(const f32x16_t &acc, int r0, int j0, int lane, int R, int B, F &&f) {
  const int j = j0 + (lane & 31);
  if (j >= B) return;
  static_for<4>([&](auto q) EE_ALWAYS_INLINE {
    constexpr int Q = decltype(q)::value;
    const int row0 = dec_row(r0, lane, 4 * Q);
    if (row0 < R) f(row0, j, f32x4_t{acc[4 * Q], acc[4 * Q + 1], acc[4 * Q + 2], acc[4 * Q + 3]});
  });
}

template <typename T>
struct DecStore {  // out[j][r] = C[r][j]
  struct Params {
    T *out;
    int64_t ld;
  };
  __device__ __forceinline__ static void apply(const Params &p, const f32x16_t &acc, int r0, int j0, int lane, int R,
                                               int B) {
    for_rows4(acc, r0, j0, lane, R, B, [&](int row0, int j, f32x4_t c) EE_ALWAYS_INLINE {
      dstore4<T>(p.out + static_cast<int64_t>(j) * p.ld + row0, c);
    });
  }
};

template <typename T>
struct DecSwiGLU {  // A[j][r] = silu(Hg[j][r]) * C[r][j]
  struct Params {
    const T *hg;
    T *act;
    int64_t ld;
  };
  __device__ __forceinline__ static void apply(const Params &p, const f32x16_t &acc, int r0, int j0, int lane, int R,
                                               int B) {
    for_rows4(acc, r0, j0, lane, R, B, [&](int row0, int j, f32x4_t hu) EE_ALWAYS_INLINE {
      const int64_t o = static_cast<int64_t>(j) * p.ld + row0;
      const f32x4_t hg = dload4<T>(p.hg + o);
      f32x4_t a;
      static_for<4>([&](auto e) EE_ALWAYS_INLINE {
        constexpr int E = decltype(e)::value;
        a[E] = silu_f(hg[E]) * hu[E];
      });
      dstore4<T>(p.act + o, a);
    });
  }
};

template <typename T>
struct DecResidual {  // Y[j][r] = X[j][r] + C[r][j]  (fp32 out)
  struct Params {
    const T *x;
    float *y;
    int64_t ld;
  };
  __device__ __forceinline__ static void apply(const Params &p, const f32x16_t &acc, int r0, int j0, int lane, int R,
                                               int B) {
    for_rows4(acc, r0, j0, lane, R, B, [&](int row0, int j, f32x4_t c) EE_ALWAYS_INLINE {
      const int64_t o = static_cast<int64_t>(j) * p.ld + row0;
      dstore4<float>(p.y + o, c + dload4<T>(p.x + o));
    });
  }
};

// Softmax partials of the output-matrix product over 32 rows (vocabulary
// ids), per token: m = max, arg = lowest id reaching m, l = sum exp(S - m).
// Stored at [32-row tile][token].
struct DecLogits {
  struct Params {
    float *part_m;
    float *part_l;
    int32_t *part_arg;
    int ld;  // tokens per partial row (B)
  };
  __device__ __forceinline__ static void apply(const Params &p, const f32x16_t &acc, int r0, int j0, int lane, int R,
                                               int B) {
    float m = -INFINITY;
    int arg = r0;  // a valid id even if no logit compares (NaN)
    static_for<16>([&](auto v) EE_ALWAYS_INLINE {
      constexpr int Vv = decltype(v)::value;
      const int row = dec_row(r0, lane, Vv);
      const float s = acc[Vv];
      if (row < R && (s > m || (s == m && row < arg))) {
        m = s;
        arg = row;
      }
    });
    const float om = __shfl_xor(m, 32);
    const int oa = __shfl_xor(arg, 32);
    if (om > m || (om == m && oa < arg)) {
      m = om;
      arg = oa;
    }
    float l = 0.0f;
    static_for<16>([&](auto v) EE_ALWAYS_INLINE {
      constexpr int Vv = decltype(v)::value;
      if (dec_row(r0, lane, Vv) < R) l += __expf(acc[Vv] - m);
    });
    l += __shfl_xor(l, 32);
    const int j = j0 + lane;
    if (lane < 32 && j < B) {
      const int64_t o = static_cast<int64_t>(r0 / kDecRows) * p.ld + j;
      p.part_m[o] = m;
      p.part_l[o] = l;
      p.part_arg[o] = arg;
    }
  }
};

// One block of 256 threads per token: combine the tiles' partials.  Each
// thread scans every 256th tile, then the waves combine by shuffles and the
// four waves through LDS (two barriers per reduction).
__device__ __forceinline__ void argmax_merge(float &m, int &t, float om, int ot) {
  // the larger maximum, the lower tile on a tie; a thread that saw no tile
  // (t < 0) takes any other, and a NaN never displaces a tile already seen
  if (ot >= 0 && (t < 0 || om > m || (om == m && ot < t))) {
    m = om;
    t = ot;
  }
}

__global__ __launch_bounds__(256) void decide_kernel(const float *part_m, const float *part_l,
                                                     const int32_t *part_arg, int tiles, int B, float threshold,
                                                     int32_t *token, float *confidence, int32_t *exit_flag) {
  __shared__ float sm[4];
  __shared__ int st[4];
  __shared__ float sl[4];
  const int j = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // max over tiles, and the lowest tile reaching it; the first tile a thread
  // sees is always taken, so the result is a valid tile even when no maximum
  // compares (NaN)
  float m = -INFINITY;
  int t_best = -1;
  for (int t = tid; t < tiles; t += 256) {
    const float v = part_m[static_cast<int64_t>(t) * B + j];
    if (t_best < 0 || v > m) {  // t increases, so the first tile reaching the maximum is kept
      m = v;
      t_best = t;
    }
  }
  for (int o = 1; o < 64; o <<= 1) argmax_merge(m, t_best, __shfl_xor(m, o), __shfl_xor(t_best, o));
  if (lane == 0) {
    sm[wave] = m;
    st[wave] = t_best;
  }
  __syncthreads();
  float mx = sm[0];
  int tb = st[0];
  for (int w = 1; w < 4; ++w) argmax_merge(mx, tb, sm[w], st[w]);
  float l = 0.0f;
  for (int t = tid; t < tiles; t += 256) {
    const int64_t o = static_cast<int64_t>(t) * B + j;
    l += part_l[o] * __expf(part_m[o] - mx);
  }
  l = warp_sum(l);
  if (lane == 0) sl[wave] = l;
  __syncthreads();
  if (tid == 0) {
    const float conf = 1.0f / ((sl[0] + sl[1]) + (sl[2] + sl[3]));
    token[j] = part_arg[static_cast<int64_t>(tb) * B + j];
    confidence[j] = conf;
    exit_flag[j] = conf > threshold ? 1 : 0;
  }
}

template <typename T, class Epi, int RG>
hipError_t launch_skinny_rg(const T *w, int64_t ldw, int R, const T *z, int64_t ldz, int B, int K,
                            const typename Epi::Params &ep, hipStream_t stream) {
  const int row_blocks = (R + kDecRows * RG - 1) / (kDecRows * RG);
  const dim3 grid(static_cast<unsigned>(row_blocks), static_cast<unsigned>((B + kDecTokens - 1) / kDecTokens));
  // 16 waves of 1024 threads leave 128 registers a lane: too few for two row groups
  const int waves = RG > 1 ? std::min(dec_waves(row_blocks), 8) : dec_waves(row_blocks);
  switch (waves) {
    case 4:
      hipLaunchKernelGGL((skinny_kernel<T, Epi, 4, RG>), grid, dim3(64 * 4), 0, stream, w, ldw, R, z, ldz, B, K, ep);
      break;
    case 8:
      hipLaunchKernelGGL((skinny_kernel<T, Epi, 8, RG>), grid, dim3(64 * 8), 0, stream, w, ldw, R, z, ldz, B, K, ep);
      break;
    default:
      if constexpr (RG == 1)
        hipLaunchKernelGGL((skinny_kernel<T, Epi, kDecWavesMax, RG>), grid, dim3(64 * kDecWavesMax), 0, stream, w, ldw,
                           R, z, ldz, B, K, ep);
  }
  return hipGetLastError();
}

// Past 8 token rows, a wide W (at least 12288 rows) is read by blocks of two
// 32-row groups per token fragment, halving the token rows' share of the
// loads (at 8 waves a block: measured 11% faster at 32 tokens for 13824 and
// 32000 rows; with 5120 rows the 80 blocks kept too few loads in flight).
template <typename T, class Epi>
hipError_t launch_skinny(const void *W, int64_t ldw, int R, const void *Z, int64_t ldz, int B, int K,
                         const typename Epi::Params &ep, hipStream_t stream) {
  if (R <= 0 || B <= 0) return hipSuccess;
  if (K % (4 * DecFrag<T>::K_PER_LOAD) != 0) return hipErrorInvalidValue;
  const T *w = static_cast<const T *>(W);
  const T *z = static_cast<const T *>(Z);
  if (B > 8 && R >= 12288) return launch_skinny_rg<T, Epi, 2>(w, ldw, R, z, ldz, B, K, ep, stream);
  return launch_skinny_rg<T, Epi, 1>(w, ldw, R, z, ldz, B, K, ep, stream);
}

}  // namespace

int decode_tiles(int rows) { return (rows + kDecRows - 1) / kDecRows; }

hipError_t decode_store(bool f32, const void *w, int rows, const void *z, int n, int k, void *out,
                        hipStream_t stream) {
  if (f32)
    return launch_skinny<float, DecStore<float>>(w, k, rows, z, k, n, k, {static_cast<float *>(out), rows}, stream);
  return launch_skinny<bf16_t, DecStore<bf16_t>>(w, k, rows, z, k, n, k, {static_cast<bf16_t *>(out), rows},
                                                 stream);
}

hipError_t decode_swiglu(bool f32, const void *w, int rows, const void *z, int n, int k, const void *hg,
                         void *act, hipStream_t stream) {
  if (f32)
    return launch_skinny<float, DecSwiGLU<float>>(
        w, k, rows, z, k, n, k, {static_cast<const float *>(hg), static_cast<float *>(act), rows}, stream);
  return launch_skinny<bf16_t, DecSwiGLU<bf16_t>>(
      w, k, rows, z, k, n, k, {static_cast<const bf16_t *>(hg), static_cast<bf16_t *>(act), rows}, stream);
}

hipError_t decode_residual(bool f32, const void *w, int rows, const void *z, int n, int k, const void *x,
                           float *y, hipStream_t stream) {
  if (f32)
    return launch_skinny<float, DecResidual<float>>(w, k, rows, z, k, n, k,
                                                    {static_cast<const float *>(x), y, rows}, stream);
  return launch_skinny<bf16_t, DecResidual<bf16_t>>(w, k, rows, z, k, n, k,
                                                    {static_cast<const bf16_t *>(x), y, rows}, stream);
}

hipError_t decode_logits(bool f32, const void *w_out, int vocab, const void *z, int n, int h, float *part_m,
                         float *part_l, int32_t *part_arg, hipStream_t stream) {
  const DecLogits::Params ep{part_m, part_l, part_arg, n};
  if (f32) return launch_skinny<float, DecLogits>(w_out, h, vocab, z, h, n, h, ep, stream);
  return launch_skinny<bf16_t, DecLogits>(w_out, h, vocab, z, h, n, h, ep, stream);
}

hipError_t decode_decide(const float *part_m, const float *part_l, const int32_t *part_arg, int tiles, int n,
                         float threshold, int32_t *token, float *confidence, int32_t *exit_flag,
                         hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(decide_kernel, dim3(static_cast<unsigned>(n)), dim3(256), 0, stream, part_m, part_l, part_arg,
                     tiles, n, threshold, token, confidence, exit_flag);
  return hipGetLastError();
}

}  // namespace ee
