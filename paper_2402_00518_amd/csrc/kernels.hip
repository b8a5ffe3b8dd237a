// Exit-head kernels for gfx950: RMSNorm forward/backward, the cross-entropy
// reduction and seed, the loss and gain-gradient reductions, and the GEMM
// instantiations with their fused epilogues.
#include <math.h>

#include <algorithm>
#include <functional>
#include <queue>
#include <type_traits>
#include <vector>

#include "epilogues.h"
#include "launch.h"

namespace ee {

// ------------------------------------------------------------ vector I/O
template <typename T, int N> __device__ __forceinline__ void load_f32(const T *p, float (&out)[N]);

template <int N> __device__ __forceinline__ void load_f32(const float *p, float (&out)[N]) {
  static_assert(N % 4 == 0, "");
#pragma unroll
  for (int c = 0; c < N / 4; ++c) {
    const f32x4_t v = reinterpret_cast<const f32x4_t *>(p)[c];
#pragma unroll
    for (int e = 0; e < 4; ++e) out[c * 4 + e] = v[e];
  }
}

template <int N> __device__ __forceinline__ void load_f32(const bf16_t *p, float (&out)[N]) {
  static_assert(N % 4 == 0, "");
  if constexpr (N % 8 == 0) {
#pragma unroll
    for (int c = 0; c < N / 8; ++c) {
      const u32x4_t w = reinterpret_cast<const u32x4_t *>(p)[c];
#pragma unroll
      for (int d = 0; d < 4; ++d) {
        out[c * 8 + 2 * d] = __uint_as_float(w[d] << 16);
        out[c * 8 + 2 * d + 1] = __uint_as_float(w[d] & 0xFFFF0000u);
      }
    }
  } else {
#pragma unroll
    for (int c = 0; c < N / 4; ++c) {
      const u32x2_t w = reinterpret_cast<const u32x2_t *>(p)[c];
#pragma unroll
      for (int d = 0; d < 2; ++d) {
        out[c * 4 + 2 * d] = __uint_as_float(w[d] << 16);
        out[c * 4 + 2 * d + 1] = __uint_as_float(w[d] & 0xFFFF0000u);
      }
    }
  }
}

template <int N> __device__ __forceinline__ void store_f32(float *p, const float (&in)[N]) {
#pragma unroll
  for (int c = 0; c < N / 4; ++c)
    reinterpret_cast<f32x4_t *>(p)[c] = f32x4_t{in[c * 4], in[c * 4 + 1], in[c * 4 + 2], in[c * 4 + 3]};
}

template <int N> __device__ __forceinline__ void store_f32(bf16_t *p, const float (&in)[N]) {
  static_assert(N % 8 == 0, "");
#pragma unroll
  for (int c = 0; c < N / 8; ++c) {
    u32x4_t w;
#pragma unroll
    for (int d = 0; d < 4; ++d)
      w[d] = static_cast<uint32_t>(f32_to_bf16(in[c * 8 + 2 * d])) |
             (static_cast<uint32_t>(f32_to_bf16(in[c * 8 + 2 * d + 1])) << 16);
    reinterpret_cast<u32x4_t *>(p)[c] = w;
  }
}

// ------------------------------------------------------- row statistics
// One wave per row.  RMSNorm: r = (mean x^2 + eps)^(-1/2).  LayerNorm (mu
// given): mu = mean x, then r = (mean (x - mu)^2 + eps)^(-1/2) from a second
// pass over the row (no cancellation from subtracting squared means).
template <typename Tin>
__global__ __launch_bounds__(256) void row_rms_kernel(const Tin *x, int64_t ldx, int n, int h, float eps,
                                                      float *r, float *mu, int *clear, int *clear_exit) {
  constexpr int V = 16 / sizeof(Tin);
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (blockIdx.x == 0 && threadIdx.x == 0) {  // a step's, or an exit's, first kernel
    if (clear != nullptr) *clear = 0;
    if (clear_exit != nullptr) *clear_exit = 0;
  }
  if (row >= n) return;
  const Tin *xr = x + static_cast<int64_t>(row) * ldx;
  float mean = 0.0f;
  if (mu != nullptr) {
    float t = 0.0f;
#pragma unroll 4
    for (int j = lane * V; j < h; j += kWave * V) {
      float v[V];
      load_f32<V>(xr + j, v);
#pragma unroll
      for (int e = 0; e < V; ++e) t += v[e];
    }
    mean = warp_sum(t) / static_cast<float>(h);
  }
  float s = 0.0f;
#pragma unroll 4
  for (int j = lane * V; j < h; j += kWave * V) {
    float v[V];
    load_f32<V>(xr + j, v);
#pragma unroll
    for (int e = 0; e < V; ++e) {
      const float c = v[e] - mean;
      s += c * c;
    }
  }
  s = warp_sum(s);
  if (lane == 0) {
    r[row] = 1.0f / sqrtf(s / static_cast<float>(h) + eps);
    if (mu != nullptr) mu[row] = mean;
  }
}

// RMSNorm statistics of the fp32 rows the split down projection leaves:
// outputs of tokens >= tok0 and features >= feat0 are held as SL partial
// sums zstride floats apart, which are first added up in slice order and
// the sum written over slice 0.  One wave per row; each lane rewrites only
// the elements it reads, and issues the loads of four 256-float groups
// before it adds and stores.
template <int SL>
__global__ __launch_bounds__(256) void row_rms_split_kernel(float *x, int n, int h, float eps, float *r, int tok0,
                                                            int feat0, int64_t zstride) {
  constexpr int U = 4, G = kWave * 4;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= n) return;
  float *xr = x + static_cast<int64_t>(row) * h;
  const int f0 = row >= tok0 ? feat0 : h;  // features from f0 on are split
  float s = 0.0f;
  for (int j0 = lane * 4; j0 < h; j0 += U * G) {
    f32x4_t v[U][SL];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = j0 + u * G;
      if (j < h) {
        v[u][0] = load4(xr + j);
        if (j >= f0) {
#pragma unroll
          for (int z = 1; z < SL; ++z) v[u][z] = load4(xr + z * zstride + j);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = j0 + u * G;
      if (j < h) {
        f32x4_t a = v[u][0];
        if (j >= f0) {
#pragma unroll
          for (int z = 1; z < SL; ++z) a += v[u][z];
          store4(xr + j, a);
        }
        s += a[0] * a[0] + a[1] * a[1] + a[2] * a[2] + a[3] * a[3];
      }
    }
  }
  s = warp_sum(s);
  if (lane == 0) r[row] = 1.0f / sqrtf(s / static_cast<float>(h) + eps);
}

// Statistics and application of the exit norm in one launch, one block per
// row, for the few rows of a decode call: z = (x - mu) r * gain (+ bias),
// mu = 0 unless `centre` (LayerNorm), r from the centred second moment.  The
// row is read again for each pass (from L1/L2).  h a multiple of 4.
template <typename Tin, typename T>
__global__ __launch_bounds__(256) void row_norm_kernel(const Tin *x, int h, float eps, const T *gain, const T *bias,
                                                       int centre, T *z) {
  __shared__ float red[4];
  const int tid = threadIdx.x;
  const Tin *xr = x + static_cast<int64_t>(blockIdx.x) * h;
  auto block_sum = [&](float v) {
    v = warp_sum(v);
    if ((tid & 63) == 0) red[tid >> 6] = v;
    __syncthreads();
    const float t = (red[0] + red[1]) + (red[2] + red[3]);
    __syncthreads();
    return t;
  };
  float mean = 0.0f;
  if (centre) {
    float t = 0.0f;
    for (int j = tid * 4; j < h; j += 1024) {
      float v[4];
      load_f32<4>(xr + j, v);
      t += (v[0] + v[1]) + (v[2] + v[3]);
    }
    mean = block_sum(t) / static_cast<float>(h);
  }
  float s = 0.0f;
  for (int j = tid * 4; j < h; j += 1024) {
    float v[4];
    load_f32<4>(xr + j, v);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float c = v[e] - mean;
      s += c * c;
    }
  }
  const float r = 1.0f / sqrtf(block_sum(s) / static_cast<float>(h) + eps);
  T *zr = z + static_cast<int64_t>(blockIdx.x) * h;
  for (int j = tid * 4; j < h; j += 1024) {
    float v[4], g[4], b[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    load_f32<4>(xr + j, v);
    load_f32<4>(gain + j, g);
    if (bias != nullptr) load_f32<4>(bias + j, b);
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = (v[e] - mean) * r * g[e] + b[e];
    store4(zr + j, f32x4_t{v[0], v[1], v[2], v[3]});
  }
}

// 64 tokens x 64 features per block.  Row-major outputs are written
// directly; the token-contiguous copy of x_hat goes through an LDS
// transpose so that both sides are coalesced.
template <typename Tin, typename T>
__global__ __launch_bounds__(256) void norm_apply_kernel(const Tin *x, int64_t ldx, const float *r,
                                                         const float *mu, const T *gain, const T *bias, int n,
                                                         int ldn, int h, T *z, T *x_hat, T *x_hat_t, int *clear,
                                                         int *clear_exit) {
  __shared__ float tile[64][65];
  if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) {  // a step's, or an exit's, first kernel
    if (clear != nullptr) *clear = 0;
    if (clear_exit != nullptr) *clear_exit = 0;
  }
  const int n0 = blockIdx.x * 64, j0 = blockIdx.y * 64;
  const int tid = threadIdx.x;
  const int tr = tid >> 2, tc = (tid & 3) * 16;
  const int row = n0 + tr;
  float v[16];
  if (row < n) {
    load_f32<16>(x + static_cast<int64_t>(row) * ldx + j0 + tc, v);
    const float rs = r != nullptr ? r[row] : 1.0f;
    const float m = mu != nullptr ? mu[row] : 0.0f;
#pragma unroll
    for (int e = 0; e < 16; ++e) v[e] = (v[e] - m) * rs;
    const int64_t o = static_cast<int64_t>(row) * h + j0 + tc;
    if (x_hat != nullptr) store_f32<16>(x_hat + o, v);
    if (z != nullptr) {
      float zz[16];
      if (gain != nullptr) {
        float g[16];
        load_f32<16>(gain + j0 + tc, g);
#pragma unroll
        for (int e = 0; e < 16; ++e) zz[e] = v[e] * g[e];
      } else {
#pragma unroll
        for (int e = 0; e < 16; ++e) zz[e] = v[e];
      }
      if (bias != nullptr) {
        float b[16];
        load_f32<16>(bias + j0 + tc, b);
#pragma unroll
        for (int e = 0; e < 16; ++e) zz[e] += b[e];
      }
      store_f32<16>(z + o, zz);
    }
  } else {
#pragma unroll
    for (int e = 0; e < 16; ++e) v[e] = 0.0f;
  }
  if (x_hat_t == nullptr) return;
#pragma unroll
  for (int e = 0; e < 16; ++e) tile[tr][tc + e] = v[e];
  __syncthreads();
  const int fr = tid >> 2, tk = (tid & 3) * 16;
  float o[16];
#pragma unroll
  for (int e = 0; e < 16; ++e) o[e] = tile[tk + e][fr];
  store_f32<16>(x_hat_t + static_cast<int64_t>(j0 + fr) * ldn + n0 + tk, o);
}

// Norm of the exit (or the MLP pre-norm) in one pass: the 8 rows of a
// block (one a wave) stay in LDS between their statistics and the two
// outputs, so x is read once instead of twice (row_rms_kernel, then
// norm_apply_kernel).  The per-lane order of the sums, the formulas and the
// roundings are those two kernels', so r, mu, z and x_hat_t come out the
// same.  Blocks of one XCD take consecutive row groups (the hardware gives
// block b to XCD b mod 8), so the 8-token pieces of each line of x_hat_t are
// written into one L2.  With rows of up to 8 KB two blocks share a CU (16
// rows were slower: one block a CU, no overlap of its load and store
// phases).
template <typename Tin> __device__ __forceinline__ void unpack16(const u32x4_t &w, float (&v)[16 / sizeof(Tin)]) {
  if constexpr (std::is_same<Tin, float>::value) {
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = __uint_as_float(w[e]);
  } else {
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      v[2 * d] = __uint_as_float(w[d] << 16);
      v[2 * d + 1] = __uint_as_float(w[d] & 0xFFFF0000u);
    }
  }
}

constexpr int kNormRows = 8;              // rows of a block, one a wave
constexpr int kNormRowsLds = 128 * 1024;  // at most, for the 8 rows of x

template <typename Tin, typename T>
__global__ __launch_bounds__(512) void norm_rows_kernel(const Tin *x, int64_t ldx, int n, int ldn, int h, float eps,
                                                        const T *gain, const T *bias, float *r, float *mu, T *z,
                                                        T *x_hat_t, int *clear, int *clear_exit) {
  constexpr int R = kNormRows;
  extern __shared__ __attribute__((aligned(16))) char rows_lds[];
  __shared__ float row_r[R], row_m[R];
  constexpr int V = 16 / sizeof(Tin);                // inputs per 16-byte chunk
  constexpr int CH = kNormRowsLds / R / 16 / kWave;  // chunks of a row per lane, at most
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (blockIdx.x == 0 && tid == 0) {  // a step's, or an exit's, first kernel
    if (clear != nullptr) *clear = 0;
    if (clear_exit != nullptr) *clear_exit = 0;
  }
  const int groups = ldn / R, per = groups / kNumXcd, rem = groups % kNumXcd;
  const int xcd = blockIdx.x % kNumXcd, idx = blockIdx.x / kNumXcd;
  const int t0 = (xcd < rem ? xcd * (per + 1) + idx : rem * (per + 1) + (xcd - rem) * per + idx) * R;
  Tin *lds = reinterpret_cast<Tin *>(rows_lds);

  // Statistics of row t0 + wave: every load of the row first, then it goes
  // to LDS and into the sums in row_rms_kernel's order.
  const int row = t0 + wave;
  float mean = 0.0f, rs = 0.0f;
  if (row < n) {
    const Tin *xr = x + static_cast<int64_t>(row) * ldx;
    Tin *lr = lds + wave * h;
    u32x4_t w[CH];
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      const int j = (lane + c * kWave) * V;
      if (j < h) w[c] = *reinterpret_cast<const u32x4_t *>(xr + j);
    }
    float t = 0.0f, s = 0.0f;
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      const int j = (lane + c * kWave) * V;
      if (j < h) {
        *reinterpret_cast<u32x4_t *>(lr + j) = w[c];
        float v[V];
        unpack16<Tin>(w[c], v);
        if (mu != nullptr) {
#pragma unroll
          for (int e = 0; e < V; ++e) t += v[e];
        } else {
#pragma unroll
          for (int e = 0; e < V; ++e) {
            const float d = v[e] - mean;
            s += d * d;
          }
        }
      }
    }
    if (mu != nullptr) {  // LayerNorm: centred second pass, from LDS
      mean = warp_sum(t) / static_cast<float>(h);
#pragma unroll
      for (int c = 0; c < CH; ++c) {
        const int j = (lane + c * kWave) * V;
        if (j < h) {
          float v[V];
          unpack16<Tin>(*reinterpret_cast<const u32x4_t *>(lr + j), v);
#pragma unroll
          for (int e = 0; e < V; ++e) {
            const float d = v[e] - mean;
            s += d * d;
          }
        }
      }
    }
    s = warp_sum(s);
    rs = 1.0f / sqrtf(s / static_cast<float>(h) + eps);
    if (lane == 0) {
      r[row] = rs;
      if (mu != nullptr) mu[row] = mean;
    }
  }
  if (lane == 0) {
    row_r[wave] = rs;
    row_m[wave] = mean;
  }
  __syncthreads();

  // z, row-major: a thread takes 8 features (gain and bias loaded once) in
  // every row, so each store of a wave is 1 KB of one row.
  for (int j = tid * 8; j < h; j += 512 * 8) {
    float g[8], b[8];
    load_f32<8>(gain + j, g);
    if (bias != nullptr) load_f32<8>(bias + j, b);
#pragma unroll
    for (int q = 0; q < R; ++q) {
      if (t0 + q >= n) break;
      float v[8], zz[8];
      load_f32<8>(lds + q * h + j, v);
      const float rq = row_r[q], m = row_m[q];
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = (v[e] - m) * rq;
#pragma unroll
      for (int e = 0; e < 8; ++e) zz[e] = v[e] * g[e];
      if (bias != nullptr) {
#pragma unroll
        for (int e = 0; e < 8; ++e) zz[e] += b[e];
      }
      store_f32<8>(z + static_cast<int64_t>(t0 + q) * h + j, zz);
    }
  }

  // x_hat_t, token-contiguous: two features a thread, the block's 8 tokens
  // each (zero past the last token, up to ldn).
  float rr[R], mm[R];
#pragma unroll
  for (int q = 0; q < R; ++q) {
    rr[q] = row_r[q];
    mm[q] = row_m[q];
  }
  for (int j = 2 * tid; j < h; j += 1024) {
    float o0[R], o1[R];
#pragma unroll
    for (int q = 0; q < R; ++q) {
      float a, b;
      if constexpr (std::is_same<Tin, float>::value) {
        const u32x2_t p = *reinterpret_cast<const u32x2_t *>(lds + q * h + j);
        a = __uint_as_float(p[0]);
        b = __uint_as_float(p[1]);
      } else {
        const uint32_t p = *reinterpret_cast<const uint32_t *>(lds + q * h + j);
        a = __uint_as_float(p << 16);
        b = __uint_as_float(p & 0xFFFF0000u);
      }
      const bool ok = t0 + q < n;
      o0[q] = ok ? (a - mm[q]) * rr[q] : 0.0f;
      o1[q] = ok ? (b - mm[q]) * rr[q] : 0.0f;
    }
    store_f32<R>(x_hat_t + static_cast<int64_t>(j) * ldn + t0, o0);
    store_f32<R>(x_hat_t + static_cast<int64_t>(j + 1) * ldn + t0, o1);
  }
}

// RMSNorm backward, one wave per row (see launch.h for the formula).
constexpr int kNormBwdMaxH = 16 * kWave * 8;  // 8192: at most 16 8-wide chunks per lane

// dZ arrives as partial sums zstride apart (split-K GEMM): ns slices at
// this position, added here in slice order.
__device__ __forceinline__ void load_dz8(const float *dz, int64_t o, int ns, int64_t zstride, float (&a)[8]) {
  load_f32<8>(dz + o, a);
  for (int z = 1; z < ns; ++z) {
    float t[8];
    load_f32<8>(dz + z * zstride + o, t);
#pragma unroll
    for (int e = 0; e < 8; ++e) a[e] += t[e];
  }
}

template <typename T, int CH>
__global__ __launch_bounds__(256) void norm_bwd_kernel(const float *dz, int splits, int64_t zstride, int tok0,
                                                       int feat0, const float *y, const float *r, const T *gain, int n,
                                                       int h, T *dy, const float *row_scale, const int *scale_off) {
  // One wave per row; the row's dZ * gain stays in registers (CH 8-wide
  // chunks per lane, h <= CH * 512) between the projection and the output,
  // so dZ's slices are read once; up to CH = 12 (h <= 6144) the row of Y
  // stays too (else it is read again, mostly from HBM: a row is 4h bytes).
  constexpr bool kKeepY = CH <= 12;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= n) return;
  const int64_t o = static_cast<int64_t>(row) * h;
  const float rr = r[row];
  // dZ's row as G W_out: with the unshifted logits the product was of P' and
  // G = diag(row_scale) P' (unless *scale_off is set)
  const float zs = row_scale != nullptr && *scale_off == 0 ? row_scale[row] : 1.0f;
  const int f0 = row >= tok0 ? feat0 : h;  // features from f0 on are split
  float dg[CH][8];
  float yk[kKeepY ? CH : 1][8];
  float s = 0.0f;
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    const int j = (c * kWave + lane) * 8;
    if (j < h) {
      float g[8], yy[8];
      load_dz8(dz, o + j, j >= f0 ? splits : 1, zstride, dg[c]);
      load_f32<8>(y + o + j, yy);
      load_f32<8>(gain + j, g);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        dg[c][e] *= g[e] * zs;
        s += dg[c][e] * yy[e] * rr;
        if constexpr (kKeepY) yk[c][e] = yy[e];
      }
    }
  }
  const float proj = warp_sum(s) / static_cast<float>(h);
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    const int j = (c * kWave + lane) * 8;
    if (j < h) {
      float yy[8], d[8];
      if constexpr (kKeepY) {
#pragma unroll
        for (int e = 0; e < 8; ++e) yy[e] = yk[c][e];
      } else {
        load_f32<8>(y + o + j, yy);
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) d[e] = rr * (dg[c][e] - yy[e] * rr * proj);
      store_f32<8>(dy + o + j, d);
    }
  }
}

// ---------------------------------------------------------- cross-entropy
// 32 tokens x 8 groups of vocab tiles per block: each thread merges the
// (max, sum-exp) partials of every 8th tile online, then the 8 groups are
// merged in a fixed order.
__device__ __forceinline__ void lse_merge(float &m, float &l, float m2, float l2) {
  const float mn = fmaxf(m, m2);
  l = l * expf(m - mn) + l2 * expf(m2 - mn);
  m = mn;
}

// 32 tokens per block: 8 threads of 4 consecutive tokens (16-byte loads) x 64
// groups of slices (slices g, g + 64, ... of group g, all loads in flight),
// merged through LDS in group order, so the result does not depend on timing.
// SHIFT0: the slices' sums are of exp(S) itself (EpiLogits with shift0), so
// LSE = log sum_s l_s (the maxima, read only for the confidence of dynamic
// token weights, may be absent).  Such a row passes the range check if
// |LSE| <= kUnshiftedLse: every logit is then at most 50 (P up to e^50) and
// the largest at least -50 - ln V (> -64 for V <= 2^20, far from bf16's
// e^-87), and coef = s_n e^-LSE, the scale of the operand it multiplies,
// within s_n e^(+-50); any row that fails sets *fallback, and the launches
// gated on it redo the exit's logits, reduce and seed in the shifted form.
// coef[n] = s_n exp(-LSE_n).
constexpr int kCeGroups = 64;
constexpr int kCeSlicesPerThread = 8;  // up to kCeGroups * 8 slices in one round of loads
constexpr float kUnshiftedLse = 50.0f;

template <bool SHIFT0>
__global__ __launch_bounds__(512) void ce_reduce_kernel(CeReduceArgs a) {
  __shared__ float sm_m[kCeGroups][32], sm_l[kCeGroups][32];
  if (a.run_if != nullptr && *a.run_if == 0) return;  // a gated rerun with nothing to redo
  const int tt = threadIdx.x & 7, g = threadIdx.x >> 3;
  const int n0 = blockIdx.x * 32 + tt * 4;  // < ldn: partials are padded to ldn tokens
  // Each thread: max over its slices, then the sum of l exp(m - max) (one
  // exponential per slice, no chain of merges).
  float m[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY}, l[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  const bool with_max = !SHIFT0 || a.dynamic_weights;  // the unshifted form's maxima exist only for those
  for (int t0 = g; t0 < a.tiles; t0 += kCeGroups * kCeSlicesPerThread) {
    f32x4_t pm[kCeSlicesPerThread], pl[kCeSlicesPerThread];
#pragma unroll
    for (int q = 0; q < kCeSlicesPerThread; ++q) {
      const int t = t0 + q * kCeGroups;
      const int64_t o = static_cast<int64_t>(min(t, a.tiles - 1)) * a.ldn + n0;
      pm[q] = with_max ? *reinterpret_cast<const f32x4_t *>(a.part_m + o) : f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
      pl[q] = *reinterpret_cast<const f32x4_t *>(a.part_l + o);
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float mx = -INFINITY;
#pragma unroll
      for (int q = 0; q < kCeSlicesPerThread; ++q)
        if (t0 + q * kCeGroups < a.tiles) mx = fmaxf(mx, pm[q][e]);
      float sl = 0.0f;
      if constexpr (SHIFT0) {
#pragma unroll
        for (int q = 0; q < kCeSlicesPerThread; ++q)
          if (t0 + q * kCeGroups < a.tiles) sl += pl[q][e];
        m[e] = fmaxf(m[e], mx);
        l[e] += sl;
      } else {
#pragma unroll
        for (int q = 0; q < kCeSlicesPerThread; ++q)
          if (t0 + q * kCeGroups < a.tiles && pl[q][e] > 0.0f) sl += pl[q][e] * fast_exp(pm[q][e] - mx);
        lse_merge(m[e], l[e], mx, sl);
      }
    }
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    sm_m[g][tt * 4 + e] = m[e];
    sm_l[g][tt * 4 + e] = l[e];
  }
  __syncthreads();
  // 16 threads per token combine the 64 groups (4 each, then a fixed
  // butterfly over the 16).
  const int tk = threadIdx.x >> 4, sub = threadIdx.x & 15, n = blockIdx.x * 32 + tk;
  float mm = -INFINITY;
#pragma unroll
  for (int q = 0; q < 4; ++q) mm = fmaxf(mm, sm_m[sub * 4 + q][tk]);
#pragma unroll
  for (int o = 8; o > 0; o >>= 1) mm = fmaxf(mm, __shfl_xor(mm, o, 16));
  float ll = 0.0f;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float lq = sm_l[sub * 4 + q][tk];
    if constexpr (SHIFT0)
      ll += lq;
    else if (lq > 0.0f)
      ll += lq * fast_exp(sm_m[sub * 4 + q][tk] - mm);
  }
#pragma unroll
  for (int o = 8; o > 0; o >>= 1) ll += __shfl_xor(ll, o, 16);
  if (sub == 0) {
    float contrib = 0.0f;
    if (n < a.n) {
      const float lse = SHIFT0 ? logf(ll) : mm + logf(ll);
      if (SHIFT0 && !(fabsf(lse) <= kUnshiftedLse)) *a.fallback = 1;  // NaN fails too
      const int y = a.targets[n];
      const bool ok = y >= 0 && y < a.vocab;
      if (!ok) *a.flag = 1;
      const float nll = ok ? lse - a.tgt[n] : NAN;
      float w = a.token_w != nullptr ? a.token_w[n] : 1.0f;
      if (a.dynamic_weights) w *= expf(mm - lse);  // detached confidence = max probability
      a.lse[n] = lse;
      const float sn = a.exit_weight * w / static_cast<float>(a.n);
      a.sn[n] = sn;
      if (SHIFT0) a.coef[n] = sn * expf(-lse);
      if (a.row_loss != nullptr) a.row_loss[n] = nll;
      contrib = w * nll;
    }
    sm_m[0][tk] = contrib;  // group 0's maxima were consumed above
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float total = 0.0f;
    for (int q = 0; q < 32; ++q) total += sm_m[0][q];
    a.block_sums[blockIdx.x] = total;
  }
}

// In-place seed: each thread owns 8 consecutive tokens of kSeedRows vocab
// rows, taken 16 at a time.  coef = s_n exp(m_tile - LSE_n) turns the stored
// exp(S - m_tile) into s_n softmax(S); the target entry loses s_n.  The
// coefficients are recomputed only where a group of 16 rows starts a new
// vocab tile (once per 64-row softmax slice).
constexpr int kSeedRows = 128;
// One block of the seed: vocab rows bx * kSeedRows .., tokens by * 2048 ..
template <typename T>
__device__ __forceinline__ void seed_block(int bx, int by, T *P, const float *part_m, const float *lse,
                                           const float *sn, const int32_t *targets, int n, int ldn, int vocab,
                                           int vtile, float *gsum_part, const float *coef = nullptr) {
  // coef != NULL: only the row sums of G = diag(coef) P (the unshifted
  // form's G, with P's target entries already shifted); P is not written.
  const bool sums_only = coef != nullptr;
  __shared__ float red[kSeedRows][4];
  const int c0 = by * 2048 + threadIdx.x * 8;
  if (gsum_part == nullptr && c0 >= ldn) return;
  const int vb = bx * kSeedRows;
  float cf[8], s[8], lz[8];
  int yy[8];
  bool ok[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int c = c0 + e;
    ok[e] = c < n;
    s[e] = ok[e] && !sums_only ? sn[c] : 0.0f;
    lz[e] = ok[e] && !sums_only ? lse[c] : 0.0f;
    yy[e] = ok[e] && !sums_only ? targets[c] : -1;
    if (sums_only) cf[e] = ok[e] ? coef[c] : 0.0f;
  }
  int tile = -1;
  const int cl = min(c0, ldn - 8);  // threads past ldn (kept for the row sums) re-read the last chunk
  constexpr int VEC = 8 * sizeof(T) / 16;  // 16-byte vectors per 8 values
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int b = 0; b < kSeedRows / 16; ++b) {
    const int v0 = vb + 16 * b;
    const int rows = min(16, vocab - v0);
    if (rows <= 0) break;  // uniform: past the vocabulary
    if (!sums_only && v0 / vtile != tile) {
      tile = v0 / vtile;
#pragma unroll
      for (int e = 0; e < 8; ++e)
        cf[e] = ok[e] ? s[e] * expf(part_m[static_cast<int64_t>(tile) * ldn + c0 + e] - lz[e]) : 0.0f;
    }
    // Issue every row's load before the first store (raw 16- or 32-byte
    // vectors; converted at use).
    u32x4_t raw[16][VEC];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const u32x4_t *src = reinterpret_cast<const u32x4_t *>(P + static_cast<int64_t>(v0 + min(r, rows - 1)) * ldn + cl);
#pragma unroll
      for (int q = 0; q < VEC; ++q) raw[r][q] = src[q];
    }
    float rsum[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      float p[8], g[8];
      load_f32<8>(reinterpret_cast<const T *>(raw[r]), p);
      rsum[r] = 0.0f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        g[e] = ok[e] ? p[e] * cf[e] - (yy[e] == v0 + r ? s[e] : 0.0f) : 0.0f;
        rsum[r] += g[e];
      }
      if (!sums_only && r < rows && c0 < ldn) store_f32<8>(P + static_cast<int64_t>(v0 + r) * ldn + c0, g);
    }
    // Row sums of G over this block's tokens (LayerNorm bias gradient):
    // fp32, fixed order.  A reduce-scatter over the wave leaves lane l with
    // row l % 16 after four halving exchanges (bits 3..0 of the lane) and
    // two full ones (16, 32): 17 shuffles instead of 16 wave sums; then the
    // 4 waves in order below.
    if (gsum_part != nullptr) {
      static_for<4>([&](auto st) EE_ALWAYS_INLINE {
        constexpr int S = decltype(st)::value, BIT = 3 - S, H = 8 >> S;
        const bool hi = (lane >> BIT) & 1;
        static_for<H>([&](auto kk) EE_ALWAYS_INLINE {
          constexpr int K = decltype(kk)::value;
          const float send = hi ? rsum[K] : rsum[K + H];
          const float keep = hi ? rsum[K + H] : rsum[K];
          rsum[K] = keep + __shfl_xor(send, 1 << BIT);
        });
      });
      rsum[0] += __shfl_xor(rsum[0], 16);
      rsum[0] += __shfl_xor(rsum[0], 32);
      if (lane < 16) red[16 * b + lane][wave] = rsum[0];
    }
  }
  if (gsum_part == nullptr) return;
  __syncthreads();
  const int rows_all = min(kSeedRows, vocab - vb);
  if (static_cast<int>(threadIdx.x) < rows_all)
    gsum_part[static_cast<int64_t>(by) * vocab + vb + threadIdx.x] =
        ((red[threadIdx.x][0] + red[threadIdx.x][1]) + red[threadIdx.x][2]) + red[threadIdx.x][3];
}

template <typename T>
__global__ __launch_bounds__(256) void seed_kernel(T *P, const float *part_m, const float *lse,
                                                   const float *sn, const int32_t *targets, int n,
                                                   int ldn, int vocab, int vtile, float *gsum_part) {
  seed_block<T>(blockIdx.x, blockIdx.y, P, part_m, lse, sn, targets, n, ldn, vocab, vtile, gsum_part);
}

// The exit's loss from the reduce's block sums (fp64, fixed order); every
// thread of a 256-thread block takes part.
__device__ __forceinline__ void final_loss_block(const float *bs, int nb, int n, float *loss, float *total, float w,
                                                 int first) {
  __shared__ double red[256];
  double s = 0.0;
  for (int i = threadIdx.x; i < nb; i += 256) s += bs[i];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const float L = static_cast<float>(red[0] / static_cast<double>(n));
    loss[0] = L;
    if (total != nullptr) total[0] = (first ? 0.0f : total[0]) + w * L;
  }
}

__global__ __launch_bounds__(256) void final_loss_kernel(const float *bs, int nb, int n, float *loss,
                                                         float *total, float w, int first) {
  final_loss_block(bs, nb, n, loss, total, w, first);
}

// 32 columns x 8 groups of tiles per block; groups merge in a fixed order.
// 32 columns per block: 8 threads of 4 consecutive columns x 32 groups of
// rows (rows g, g + 32, ... of group g, loads in flight in batches of 8),
// merged through LDS in group order.  Row strides that are multiples of 4
// (the gain gradients: h is a multiple of 64) take 16-byte loads; others
// (the vocabulary-wide row sums) take bounds-checked scalar loads.
constexpr int kGainGroups = 32;

template <bool VEC>
__device__ __forceinline__ f32x4_t sum_rows4(const float *p, int tiles, int h, int g, int j0) {
  f32x4_t s = {0.0f, 0.0f, 0.0f, 0.0f};
  if (j0 >= h) return s;
  for (int t0 = g; t0 < tiles; t0 += kGainGroups * 8) {
    f32x4_t v[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const float *row = p + static_cast<int64_t>(min(t0 + q * kGainGroups, tiles - 1)) * h;
      if constexpr (VEC) {
        v[q] = *reinterpret_cast<const f32x4_t *>(row + j0);
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) v[q][e] = j0 + e < h ? row[j0 + e] : 0.0f;
      }
    }
#pragma unroll
    for (int q = 0; q < 8; ++q)
      if (t0 + q * kGainGroups < tiles) s += v[q];
  }
  return s;
}

__global__ __launch_bounds__(256) void gain_reduce_kernel(const float *pa, int ta, const float *pb, int tb,
                                                          int h, float *out, int accumulate) {
  __shared__ float red[kGainGroups][32];
  const int tc = threadIdx.x & 7, g = threadIdx.x >> 3;
  const int j0 = blockIdx.x * 32 + tc * 4;
  f32x4_t s;
  with_flag(h % 4 == 0, [&](auto V_) EE_ALWAYS_INLINE {
    constexpr bool kVec = decltype(V_)::value;
    s = sum_rows4<kVec>(pa, ta, h, g, j0);
    if (pb != nullptr) s += sum_rows4<kVec>(pb, tb, h, g, j0);
  });
#pragma unroll
  for (int e = 0; e < 4; ++e) red[g][tc * 4 + e] = s[e];
  __syncthreads();
  if (threadIdx.x >= 32) return;
  const int c = threadIdx.x, j = blockIdx.x * 32 + c;
  if (j >= h) return;
  float total = red[0][c];
  for (int q = 1; q < kGainGroups; ++q) total += red[q][c];
  out[j] = accumulate ? out[j] + total : total;
}


// -------------------------------------------------------------- launchers
#define EE_DISPATCH(f32, ...)            \
  do {                                   \
    if (f32) {                           \
      using T = float;                   \
      __VA_ARGS__;                       \
    } else {                             \
      using T = bf16_t;                  \
      __VA_ARGS__;                       \
    }                                    \
  } while (0)

hipError_t launch_row_rms(bool x_f32, const void *x, int64_t ldx, int n, int h, float eps, float *r,
                          hipStream_t stream, float *mu, int *clear, int *clear_exit) {
  const dim3 grid(cdiv(n, 4));
  if (x_f32)
    hipLaunchKernelGGL(row_rms_kernel<float>, grid, dim3(256), 0, stream, static_cast<const float *>(x), ldx,
                       n, h, eps, r, mu, clear, clear_exit);
  else
    hipLaunchKernelGGL(row_rms_kernel<bf16_t>, grid, dim3(256), 0, stream, static_cast<const bf16_t *>(x),
                       ldx, n, h, eps, r, mu, clear, clear_exit);
  return hipGetLastError();
}

hipError_t launch_row_rms_split(float *x, int n, int h, float eps, float *r, SplitTail sp, hipStream_t stream) {
  if (sp.splits <= 1) return launch_row_rms(true, x, h, n, h, eps, r, stream);
  if (h % 4 != 0 || sp.tok0 < 0 || sp.tok0 > n || sp.feat0 < 0 || sp.feat0 > h) return hipErrorInvalidValue;
  const dim3 grid(cdiv(n, 4));
  const int64_t zs = static_cast<int64_t>(n) * h;
  switch (sp.splits) {
    case 2:
      hipLaunchKernelGGL(row_rms_split_kernel<2>, grid, dim3(256), 0, stream, x, n, h, eps, r, sp.tok0, sp.feat0, zs);
      break;
    case 3:
      hipLaunchKernelGGL(row_rms_split_kernel<3>, grid, dim3(256), 0, stream, x, n, h, eps, r, sp.tok0, sp.feat0, zs);
      break;
    case 4:
      hipLaunchKernelGGL(row_rms_split_kernel<4>, grid, dim3(256), 0, stream, x, n, h, eps, r, sp.tok0, sp.feat0, zs);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_row_norm(bool x_f32, bool f32, const void *x, int n, int h, float eps, const void *gain,
                           const void *bias, bool centre, void *z, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  if (h % 4 != 0 || gain == nullptr) return hipErrorInvalidValue;
  const dim3 grid(static_cast<unsigned>(n));
  const int c = centre ? 1 : 0;
  EE_DISPATCH(f32, {
    const T *g = static_cast<const T *>(gain), *b = static_cast<const T *>(bias);
    if (x_f32)
      hipLaunchKernelGGL((row_norm_kernel<float, T>), grid, dim3(256), 0, stream, static_cast<const float *>(x), h, eps,
                         g, b, c, static_cast<T *>(z));
    else
      hipLaunchKernelGGL((row_norm_kernel<bf16_t, T>), grid, dim3(256), 0, stream, static_cast<const bf16_t *>(x), h,
                         eps, g, b, c, static_cast<T *>(z));
  });
  return hipGetLastError();
}

hipError_t launch_norm_apply(bool x_f32, bool f32, const void *x, int64_t ldx, const float *r,
                             const void *gain, int n, int ldn, int h, void *z, void *x_hat, void *x_hat_t,
                             hipStream_t stream, const float *mu, const void *bias, int *clear, int *clear_exit) {
  const dim3 grid(cdiv(ldn, 64), h / 64);
  EE_DISPATCH(f32, {
    if (x_f32)
      hipLaunchKernelGGL((norm_apply_kernel<float, T>), grid, dim3(256), 0, stream,
                         static_cast<const float *>(x), ldx, r, mu, static_cast<const T *>(gain),
                         static_cast<const T *>(bias), n, ldn, h, static_cast<T *>(z), static_cast<T *>(x_hat),
                         static_cast<T *>(x_hat_t), clear, clear_exit);
    else
      hipLaunchKernelGGL((norm_apply_kernel<bf16_t, T>), grid, dim3(256), 0, stream,
                         static_cast<const bf16_t *>(x), ldx, r, mu, static_cast<const T *>(gain),
                         static_cast<const T *>(bias), n, ldn, h, static_cast<T *>(z), static_cast<T *>(x_hat),
                         static_cast<T *>(x_hat_t), clear, clear_exit);
  });
  return hipGetLastError();
}

bool norm_rows(int h, bool x_f32) { return kNormRows * h * (x_f32 ? 4 : 2) <= kNormRowsLds; }

hipError_t launch_norm_rows(bool f32, const void *x, int64_t ldx, int n, int ldn, int h, float eps, const void *gain,
                            const void *bias, float *r, float *mu, void *z, void *x_hat_t, hipStream_t stream,
                            int *clear, int *clear_exit) {
  if (!norm_rows(h, f32) || h % 64 != 0 || ldn % 64 != 0 || n > ldn || gain == nullptr || z == nullptr ||
      x_hat_t == nullptr)
    return hipErrorInvalidValue;
  const int lds = kNormRows * h * (f32 ? 4 : 2);
  hipError_t e = hipSuccess;
  EE_DISPATCH(f32, {
    const auto k = norm_rows_kernel<T, T>;
    e = hipFuncSetAttribute(reinterpret_cast<const void *>(k), hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e == hipSuccess) {
      hipLaunchKernelGGL(k, dim3(ldn / kNormRows), dim3(512), lds, stream, static_cast<const T *>(x), ldx, n, ldn, h,
                         eps, static_cast<const T *>(gain), static_cast<const T *>(bias), r, mu, static_cast<T *>(z),
                         static_cast<T *>(x_hat_t), clear, clear_exit);
      e = hipGetLastError();
    }
  });
  return e;
}

hipError_t launch_ce_reduce(const CeReduceArgs &a, hipStream_t stream) {
  if (a.shift0)
    hipLaunchKernelGGL(ce_reduce_kernel<true>, dim3(cdiv(a.n, 32)), dim3(512), 0, stream, a);
  else
    hipLaunchKernelGGL(ce_reduce_kernel<false>, dim3(cdiv(a.n, 32)), dim3(512), 0, stream, a);
  return hipGetLastError();
}

int seed_chunks(int ldn) { return cdiv(ldn, 2048); }

hipError_t launch_seed(bool f32, void *P, const float *part_m, const float *lse, const float *sn,
                       const int32_t *targets, int n, int ldn, int vocab, int vtile, hipStream_t stream,
                       float *gsum_part) {
  const dim3 grid(cdiv(vocab, kSeedRows), seed_chunks(ldn));
  EE_DISPATCH(f32, hipLaunchKernelGGL(seed_kernel<T>, grid, dim3(256), 0, stream, static_cast<T *>(P), part_m,
                                      lse, sn, targets, n, ldn, vocab, vtile, gsum_part));
  return hipGetLastError();
}

// The unshifted form's counterpart of the seed: G = diag(coef) P' with
// P' = P except at each token's target, P'[y_n][n] = P[y_n][n] - exp(LSE_n)
// (then coef_n P' = s_n (p - 1) there), so instead of rewriting P the
// per-token factor goes into the other operand of the weight gradient:
// x_hat_t[j][n] *= coef_n (token columns n..ldn-1 stay zero).  One block:
// tokens bx * 2048 .., feature rows by * 8 .. + 7, each thread 8 tokens of
// the 8 rows (all loads first); a thread of the row bands by < 8 also fixes
// the target of its token c0 + by (h >= 64), one each.
template <typename T>
__device__ __forceinline__ void scale_block(int bx, int by, T *x_hat_t, T *P, const float *coef, const float *lse,
                                            const int32_t *targets, int n, int ldn, int vocab) {
  const int c0 = bx * 2048 + threadIdx.x * 8;
  if (c0 >= ldn) return;
  float cf[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) cf[e] = c0 + e < n ? coef[c0 + e] : 0.0f;
  float v[8][8];
#pragma unroll
  for (int r = 0; r < 8; ++r) load_f32<8>(x_hat_t + static_cast<int64_t>(by * 8 + r) * ldn + c0, v[r]);
#pragma unroll
  for (int r = 0; r < 8; ++r) {
#pragma unroll
    for (int e = 0; e < 8; ++e) v[r][e] *= cf[e];
    store_f32<8>(x_hat_t + static_cast<int64_t>(by * 8 + r) * ldn + c0, v[r]);
  }
  const int c = c0 + by;
  if (by < 8 && c < n) {
    const int y = targets[c];
    if (y >= 0 && y < vocab) {
      T *q = P + static_cast<int64_t>(y) * ldn + c;
      *q = from_f32<T>(to_f32(*q) - expf(lse[c]));
    }
  }
}

// After the unshifted reduce: the seed if *fallback is set (the shifted
// form was redone), else the operand scale.  One grid for either job (a
// block past the job's blocks does nothing); block 0 first turns the
// reduce's block sums into the exit's loss (FinalLoss: as
// launch_final_loss).
struct FinalLoss {
  const float *block_sums;
  int blocks;
  float *loss;
  float *total;
  float w;
  int first;
};

template <typename T>
__global__ __launch_bounds__(256) void seed_or_scale_kernel(T *P, T *x_hat_t, const float *part_m, const float *lse,
                                                            const float *sn, const float *coef,
                                                            const int32_t *targets, int n, int ldn, int h, int vocab,
                                                            int vtile, const int *fallback, float *gsum_part,
                                                            FinalLoss fl) {
  const int b = blockIdx.x;
  if (b == 0) final_loss_block(fl.block_sums, fl.blocks, n, fl.loss, fl.total, fl.w, fl.first);
  if (*fallback != 0) {
    const int sx = cdiv(vocab, kSeedRows), sy = cdiv(ldn, 2048);  // seed_chunks(ldn)
    if (b < sx * sy) seed_block<T>(b % sx, b / sx, P, part_m, lse, sn, targets, n, ldn, vocab, vtile, gsum_part);
  } else {
    const int cx = cdiv(ldn, 2048), cy = h / 8;
    if (b < cx * cy) scale_block<T>(b % cx, b / cx, x_hat_t, P, coef, lse, targets, n, ldn, vocab);
  }
}

hipError_t launch_seed_or_scale(bool f32, void *P, void *x_hat_t, const float *part_m, const float *lse,
                                const float *sn, const float *coef, const int32_t *targets, int n, int ldn, int h,
                                int vocab, int vtile, const int *fallback, const float *block_sums, int loss_blocks,
                                float *loss, float *total, float w, int first, hipStream_t stream,
                                float *gsum_part) {
  if (n <= 0) return hipSuccess;
  if (h % 8 != 0 || h < 64 || ldn % 8 != 0 || fallback == nullptr) return hipErrorInvalidValue;
  const int64_t blocks = std::max<int64_t>(static_cast<int64_t>(cdiv(vocab, kSeedRows)) * seed_chunks(ldn),
                                           static_cast<int64_t>(cdiv(ldn, 2048)) * (h / 8));
  if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
  EE_DISPATCH(f32, hipLaunchKernelGGL(seed_or_scale_kernel<T>, dim3(static_cast<unsigned>(blocks)), dim3(256), 0,
                                      stream, static_cast<T *>(P), static_cast<T *>(x_hat_t), part_m, lse, sn, coef,
                                      targets, n, ldn, h, vocab, vtile, fallback, gsum_part,
                                      FinalLoss{block_sums, loss_blocks, loss, total, w, first}));
  return hipGetLastError();
}

// Row sums of G = diag(coef) P' per 2048-token chunk (the seed's partials),
// for the bias gradient of an exit in the unshifted form, after the operand
// scale has shifted P's target entries; nothing if the exit fell back to
// the shifted form, whose seed wrote them.
template <typename T>
__global__ __launch_bounds__(256) void gsum_unshifted_kernel(const T *P, const float *coef, int n, int ldn, int vocab,
                                                             const int *fallback, float *gsum_part) {
  if (*fallback != 0) return;  // the same word for every thread
  seed_block<T>(blockIdx.x, blockIdx.y, const_cast<T *>(P), nullptr, nullptr, nullptr, nullptr, n, ldn, vocab, 1,
                gsum_part, coef);
}

hipError_t launch_gsum_unshifted(bool f32, const void *P, const float *coef, int n, int ldn, int vocab,
                                 const int *fallback, float *gsum_part, hipStream_t stream) {
  if (n <= 0 || vocab <= 0) return hipSuccess;
  if (ldn % 8 != 0 || coef == nullptr || fallback == nullptr || gsum_part == nullptr) return hipErrorInvalidValue;
  const dim3 grid(cdiv(vocab, kSeedRows), seed_chunks(ldn));
  EE_DISPATCH(f32, hipLaunchKernelGGL(gsum_unshifted_kernel<T>, grid, dim3(256), 0, stream, static_cast<const T *>(P),
                                      coef, n, ldn, vocab, fallback, gsum_part));
  return hipGetLastError();
}

hipError_t launch_final_loss(const float *block_sums, int blocks, int n, float *loss, float *total, float w,
                             int first, hipStream_t stream) {
  hipLaunchKernelGGL(final_loss_kernel, dim3(1), dim3(256), 0, stream, block_sums, blocks, n, loss, total, w,
                     first);
  return hipGetLastError();
}

hipError_t launch_gain_reduce(const float *part_a, int tiles_a, const float *part_b, int tiles_b, int h,
                              float *out, int accumulate, hipStream_t stream) {
  hipLaunchKernelGGL(gain_reduce_kernel, dim3(cdiv(h, 32)), dim3(256), 0, stream, part_a, tiles_a, part_b,
                     tiles_b, h, out, accumulate);
  return hipGetLastError();
}

hipError_t launch_norm_bwd(bool f32, const float *dz, const float *y, const float *r, const void *gain, int n,
                           int h, void *dy, hipStream_t stream, SplitTail sp, const float *row_scale,
                           const int *scale_off) {
  if (row_scale != nullptr && scale_off == nullptr) return hipErrorInvalidValue;
  if (h > kNormBwdMaxH) return hipErrorInvalidValue;
  const int splits = sp.splits > 1 ? sp.splits : 1;
  const int t0 = splits > 1 ? sp.tok0 : n, f0 = splits > 1 ? sp.feat0 : h;
  if (t0 < 0 || t0 > n || f0 < 0 || f0 > h) return hipErrorInvalidValue;
  const int64_t zs = static_cast<int64_t>(n) * h;
  const dim3 grid(cdiv(n, 4));
  EE_DISPATCH(f32, {
    const T *g = static_cast<const T *>(gain);
    T *d = static_cast<T *>(dy);
    if (h <= 2048)
      hipLaunchKernelGGL((norm_bwd_kernel<T, 4>), grid, dim3(256), 0, stream, dz, splits, zs, t0, f0, y, r, g, n, h, d, row_scale, scale_off);
    else if (h <= 4096)
      hipLaunchKernelGGL((norm_bwd_kernel<T, 8>), grid, dim3(256), 0, stream, dz, splits, zs, t0, f0, y, r, g, n, h, d, row_scale, scale_off);
    else if (h <= 6144)
      hipLaunchKernelGGL((norm_bwd_kernel<T, 12>), grid, dim3(256), 0, stream, dz, splits, zs, t0, f0, y, r, g, n, h, d, row_scale, scale_off);
    else
      hipLaunchKernelGGL((norm_bwd_kernel<T, 16>), grid, dim3(256), 0, stream, dz, splits, zs, t0, f0, y, r, g, n, h, d, row_scale, scale_off);
  });
  return hipGetLastError();
}


// ------------------------------------------------------------------ GEMMs
// bf16 GEMMs take the 256 x 256 tile (either operand K-major or MN-major),
// fp32 GEMMs the 128 x 128 tile.
template <typename T, bool AK, bool BKM, class Epi>
hipError_t run_gemm(Operand A, Operand B, GemmShape s, const typename Epi::Params &ep, hipStream_t stream) {
  if constexpr (std::is_same<T, bf16_t>::value)
    return launch_gemm<T, AK, BKM, Epi, CfgBig>(A, B, s, ep, stream);
  else
    return launch_gemm<T, AK, BKM, Epi, CfgSmall>(A, B, s, ep, stream);
}

template <typename T, bool AK1, bool BKM1, class Epi1, bool AK2, bool BKM2, class Epi2>
hipError_t run_gemm_pair(Operand A1, Operand B1, GemmShape s1, const typename Epi1::Params &ep1, Operand A2,
                         Operand B2, GemmShape s2, const typename Epi2::Params &ep2, hipStream_t stream) {
  if constexpr (std::is_same<T, bf16_t>::value)
    return launch_gemm_pair<T, AK1, BKM1, Epi1, AK2, BKM2, Epi2, CfgBig>(A1, B1, s1, ep1, A2, B2, s2, ep2, stream);
  else
    return launch_gemm_pair<T, AK1, BKM1, Epi1, AK2, BKM2, Epi2, CfgSmall>(A1, B1, s1, ep1, A2, B2, s2, ep2, stream);
}

int gemm_part_cols(bool f32) { return f32 ? CfgSmall::WN : CfgBig::WN; }

hipError_t gemm_logits(bool f32, const void *w_out, const void *z, int vocab, int n, int h, void *P, int ldn,
                       float *part_m, float *part_l, float *tgt, const int32_t *targets, hipStream_t stream,
                       int shift0, const int *run_if) {
  EE_DISPATCH(f32, {
    typename EpiLogits<T>::Params ep{static_cast<T *>(P), ldn, part_m, part_l, tgt, targets, shift0};
    const Operand A{z, h}, B{w_out, h};
    const GemmShape sh{n, vocab, h};
    if (run_if != nullptr) {
      if constexpr (std::is_same<T, bf16_t>::value)
        return launch_gemm_gated<T, true, true, EpiLogits<T>, CfgBig>(A, B, sh, ep, run_if, stream);
      else
        return launch_gemm_gated<T, true, true, EpiLogits<T>, CfgSmall>(A, B, sh, ep, run_if, stream);
    }
    return run_gemm<T, true, true, EpiLogits<T>>(A, B, sh, ep, stream);
  });
  return hipSuccess;
}

hipError_t gemm_weight_grad_kk(bool f32, const void *g_t, const void *xhat_t, int m, int h, int ldn,
                               const void *gain, const void *w, float *dw, float *part, int accumulate,
                               hipStream_t stream, const float *gsum, const void *bias, float *part_b) {
  EE_DISPATCH(f32, {
    typename EpiWeightGrad<T>::Params ep{dw,   h,         static_cast<const T *>(gain), static_cast<const T *>(w),
                                         part, accumulate, gsum, static_cast<const T *>(bias), part_b};
    return run_gemm<T, true, true, EpiWeightGrad<T>>(Operand{xhat_t, ldn}, Operand{g_t, ldn},
                                                        GemmShape{h, m, ldn}, ep, stream);
  });
  return hipSuccess;
}

hipError_t gemm_weight_grad_kk_pair(bool f32, const void *g1_t, const void *g2_t, const void *xhat_t, int m, int h,
                                    int ldn, const void *gain, const void *w1, const void *w2, float *dw1, float *dw2,
                                    float *part1, float *part2, int accumulate, hipStream_t stream) {
  EE_DISPATCH(f32, {
    const T *gn = static_cast<const T *>(gain);
    typename EpiWeightGrad<T>::Params e1{dw1, h, gn, static_cast<const T *>(w1), part1, accumulate};
    typename EpiWeightGrad<T>::Params e2{dw2, h, gn, static_cast<const T *>(w2), part2, accumulate};
    return run_gemm_pair<T, true, true, EpiWeightGrad<T>, true, true, EpiWeightGrad<T>>(
        Operand{xhat_t, ldn}, Operand{g1_t, ldn}, GemmShape{h, m, ldn}, e1, Operand{xhat_t, ldn},
        Operand{g2_t, ldn}, GemmShape{h, m, ldn}, e2, stream);
  });
  return hipSuccess;
}

hipError_t gemm_gate_up_swiglu(bool f32, const void *u, const void *w_gate, const void *w_up, int n, int inter,
                               int h, void *hgu, void *act, hipStream_t stream) {
  EE_DISPATCH(f32, {
    typename EpiGateUp<T>::Params ep{static_cast<typename GatePair<T>::type *>(hgu), static_cast<T *>(act)};
    const int64_t pair = static_cast<const char *>(w_up) - static_cast<const char *>(w_gate);
    return run_gemm<T, true, true, EpiGateUp<T>>(Operand{u, h}, Operand{w_gate, h, pair},
                                                    GemmShape{n, 2 * inter, h}, ep, stream);
  });
  return hipSuccess;
}

hipError_t gemm_down_residual(bool f32, const void *act, const void *w_down, const void *x, int n, int h,
                              int inter, float *y, hipStream_t stream, SplitTail sp) {
  EE_DISPATCH(f32, {
    const T *xt = static_cast<const T *>(x), *at = static_cast<const T *>(act), *wd = static_cast<const T *>(w_down);
    // Tiles: tokens as rows, features as columns.  Split region: tokens
    // [t0, n) x features [f0, h).  The rest takes all of K: tokens [0, t0)
    // (f0 == 0) or features [0, f0) (t0 == 0).
    const bool split = sp.splits > 1;
    const int t0 = split ? sp.tok0 : n, f0 = split ? sp.feat0 : 0;
    if (t0 < 0 || t0 > n || f0 < 0 || f0 > h || (t0 > 0 && f0 > 0)) return hipErrorInvalidValue;
    const int m1 = t0 > 0 ? t0 : n, n1 = t0 > 0 ? h : f0;
    const int64_t o = static_cast<int64_t>(t0) * h + f0;
    typename EpiResidual<T>::Params e1{y, xt, h, 0};
    typename EpiResidual<T>::Params e2{y + o, xt + o, h, static_cast<int64_t>(n) * h};
    GemmShape s2{n - t0, h - f0, inter};
    if (split) {
      s2.kchunk = split_kchunk(inter, sp.splits);
      if (cdiv(inter, s2.kchunk) != sp.splits) return hipErrorInvalidValue;  // Y holds sp.splits slices
    }
    return run_gemm_pair<T, true, true, EpiResidual<T>, true, true, EpiResidual<T>>(
        Operand{at, inter}, Operand{wd, inter}, GemmShape{m1, n1, inter}, e1,
        Operand{at + static_cast<int64_t>(t0) * inter, inter}, Operand{wd + static_cast<int64_t>(f0) * inter, inter},
        s2, e2, stream);
  });
  return hipSuccess;
}

namespace {

constexpr int kCus = 256;           // compute units the launch shapes are planned for
constexpr double kEpilogueK = 1024;  // prologue and epilogue of a 256 x 256 tile, in K values of its main loop
constexpr double kBytesPerK = 1.2e5;  // HBM bytes moved while a CU runs one such K value

// Duration, in K values, of `full` whole-K tiles followed by `parts` blocks
// of kchunk K values each, dispatched in order to the first free of kCus
// compute units.
double launch_span(int64_t full, int64_t parts, int K, int kchunk) {
  const double D = K + kEpilogueK, d = kchunk + kEpilogueK;
  const int64_t rest = full % kCus;
  std::priority_queue<double, std::vector<double>, std::greater<double>> q;
  double end = rest > 0 ? D : 0.0;
  for (int i = 0; i < kCus; ++i) q.push(i < rest ? D : 0.0);
  for (int64_t p = 0; p < parts; ++p) {
    const double t = q.top() + d;
    q.pop();
    q.push(t);
    end = std::max(end, t);
  }
  return static_cast<double>(full / kCus) * D + end;
}

}  // namespace

int split_kchunk(int K, int splits) { return cdiv(cdiv(K, splits), 64) * 64; }

SplitTail split_tail(bool f32, int n, int h, int K) {
  SplitTail best{n, 0, 1};
  if (f32 || n <= 0) return best;
  // the last few shapes asked for (a layout asks for two per call)
  struct Memo {
    int n = -1, h = -1, K = -1;
    SplitTail sp{0, 0, 1};
  };
  static thread_local Memo memo[4];
  static thread_local int next = 0;
  for (const Memo &m : memo)
    if (m.n == n && m.h == h && m.K == K) return m.sp;
  const int tm = cdiv(h, CfgBig::BM), tn = cdiv(n, CfgBig::BN);
  const int64_t tiles = static_cast<int64_t>(tm) * tn;
  if (tiles < 4 * kCus) {
    const int64_t rounds = tiles / kCus;
    double best_span = 0.9 * launch_span(tiles, 0, K, K);
    for (int s = 2; s <= 4; s *= 2) {
      if (K / s < 4 * 64) break;
      const int kc = split_kchunk(K, s), slices = cdiv(K, kc);
      // Split the last c token blocks (dim 0) or feature blocks (dim 1):
      // all of them, or the fewest that leave the whole-K tiles one or two
      // rounds short of the current count.
      for (int dim = 0; dim < 2; ++dim) {
        const int blocks = dim == 0 ? tn : tm, across = dim == 0 ? tm : tn;
        int cand[3] = {blocks, 0, 0};
        for (int r = 0; r < 2; ++r)
          if (rounds - r >= 0) cand[r + 1] = static_cast<int>((tiles - (rounds - r) * kCus + across - 1) / across);
        for (int c : cand) {
          if (c < 1 || c > blocks) continue;
          const SplitTail sp = dim == 0 ? SplitTail{(tn - c) * CfgBig::BN, 0, slices}
                                        : SplitTail{0, (tm - c) * CfgBig::BM, slices};
          // extra HBM traffic: slices 1.. written and read back, their sum written
          const double outs = static_cast<double>(n - sp.tok0) * (h - sp.feat0);
          const double extra = outs * 4 * (2 * (slices - 1) + 1) / kBytesPerK;
          const double span = launch_span(static_cast<int64_t>(blocks - c) * across,
                                          static_cast<int64_t>(c) * across * slices, K, kc) + extra;
          if (span < best_span) {
            best_span = span;
            best = sp;
          }
        }
      }
    }
  }
  memo[next] = Memo{n, h, K, best};
  next = (next + 1) % 4;
  return best;
}

hipError_t gemm_dz(bool f32, const void *g_t, const void *w_out, int n, int ldn, int h, int vocab, float *dz,
                   hipStream_t stream, SplitTail sp) {
  EE_DISPATCH(f32, {
    const T *gt = static_cast<const T *>(g_t), *wo = static_cast<const T *>(w_out);
    // Tiles: tokens (padded to ldn; rows past n are not stored) as rows,
    // features as columns, both operands read MN-major.  Split region:
    // tokens [t0, n) x features [f0, h); the rest takes all of K: tokens
    // [0, t0) (f0 == 0) or features [0, f0) (t0 == 0).
    if (sp.splits <= 1) {
      typename EpiStoreF32<T>::Params ep{dz, h, n, 0, 0};
      return run_gemm<T, false, false, EpiStoreF32<T>>(Operand{gt, ldn}, Operand{wo, h}, GemmShape{ldn, h, vocab}, ep,
                                                        stream);
    }
    const int t0 = sp.tok0, f0 = sp.feat0;
    if (t0 < 0 || t0 > n || t0 % 64 != 0 || f0 < 0 || f0 > h || (t0 > 0 && f0 > 0)) return hipErrorInvalidValue;
    const int m1 = t0 > 0 ? t0 : ldn, n1 = t0 > 0 ? h : f0;
    typename EpiStoreF32<T>::Params e1{dz, h, t0 > 0 ? t0 : n, 0, 0};
    typename EpiStoreF32<T>::Params e2{dz + static_cast<int64_t>(t0) * h + f0, h, n - t0, 0,
                                       static_cast<int64_t>(n) * h};
    GemmShape s2{ldn - t0, h - f0, vocab};
    s2.kchunk = split_kchunk(vocab, sp.splits);
    if (cdiv(vocab, s2.kchunk) != sp.splits) return hipErrorInvalidValue;  // dZ holds sp.splits slices
    return run_gemm_pair<T, false, false, EpiStoreF32<T>, false, false, EpiStoreF32<T>>(
        Operand{gt, ldn}, Operand{wo, h}, GemmShape{m1, n1, vocab}, e1, Operand{gt + t0, ldn}, Operand{wo + f0, h}, s2,
        e2, stream);
  });
  return hipSuccess;
}

hipError_t gemm_da_swiglu_dw_down(bool f32, const void *dy, const void *w_down, int n, int inter, int h,
                                 const void *hgu, void *dhg_t, void *dhu_t, int ldn, const void *act, float *dwd,
                                 int accumulate, hipStream_t stream) {
  EE_DISPATCH(f32, {
    typename EpiSwiGLUBwd<T>::Params e1{static_cast<const typename GatePair<T>::type *>(hgu),
                                        static_cast<T *>(dhg_t), static_cast<T *>(dhu_t), inter, ldn};
    typename EpiStoreF32<T>::Params e2{dwd, inter, h, accumulate};
    return run_gemm_pair<T, true, false, EpiSwiGLUBwd<T>, false, false, EpiStoreF32<T>>(
        Operand{dy, h}, Operand{w_down, inter}, GemmShape{n, inter, h}, e1, Operand{dy, h}, Operand{act, inter},
        GemmShape{h, inter, n}, e2, stream);
  });
  return hipSuccess;
}

}  // namespace ee
