// Tiled MFMA GEMM for gfx950 with fused epilogues.
//
//   C[m][n] = sum_k A(m, k) * B(n, k)
//
// Each operand is either K-major (element (r, k) at ptr[r*ld + k], K
// contiguous) or MN-major (element (r, k) at ptr[k*ld + r], rows
// contiguous).  Tiles are staged through LDS in one canonical K-contiguous
// layout, so the MFMA fragment reads are the same for both: an MN-major
// operand is transposed in registers (4 k-rows x one 16-byte column group
// per thread) on its way into LDS.
//
// Work split: 256 threads = 4 waves of 64 lanes arranged 2 x 2 over a
// 128 x 128 output tile; each wave owns 64 x 64 = 2 x 2 blocks of
// 32 x 32 MFMA accumulators.  Each LDS tile row holds 128 bytes of K
// (64 bf16 or 32 fp32 values), XOR-swizzled in 16-byte chunks so that the
// 8 rows a quarter-wave reads hit distinct banks.  Two LDS stages; the
// next stage's global loads are in flight while the current one feeds the
// matrix cores.
//
// bf16 operands use v_mfma_f32_32x32x16_bf16, fp32 operands
// v_mfma_f32_32x32x2_f32; both accumulate in fp32.
#pragma once

#include "ee_device.h"

namespace ee {

struct Operand {
  const void *ptr;
  int64_t ld;  // elements between consecutive rows of the stored matrix
};

struct GemmShape {
  int M, N, K;
};

constexpr int kGemmThreads = 256;
constexpr int kBM = 128;
constexpr int kBN = 128;
constexpr int kRowBytes = 128;
constexpr int kStageBytes = (kBM + kBN) * kRowBytes;  // A tile then B tile

template <typename T> struct Elem;
template <> struct Elem<bf16_t> {
  static constexpr int CH = 8;  // elements per 16-byte chunk
};
template <> struct Elem<float> {
  static constexpr int CH = 4;
};

__host__ __device__ constexpr int cdiv(int64_t a, int64_t b) { return static_cast<int>((a + b - 1) / b); }

// Byte offset of 16-byte chunk `ch` (0..7) of LDS tile row `row`.
__device__ __forceinline__ int lds_off(int row, int ch) {
  return row * kRowBytes + ((ch ^ (row & 7)) << 4);
}

// ---------------------------------------------------------------- loaders
// K-major tile: 128 rows x 8 chunks = 1024 16-byte loads, 4 per thread.
template <typename T>
struct KMajorLoader {
  static constexpr int CH = Elem<T>::CH;
  u32x4_t reg[4];

  __device__ __forceinline__ void load(const T *base, int64_t ld, int row0, int rows, int k0,
                                       int K, int tid) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = tid + i * kGemmThreads;
      const int r = c >> 3, ch = c & 7;
      const int gr = row0 + r, gk = k0 + ch * CH;
      if (gr < rows && gk < K)
        reg[i] = *reinterpret_cast<const u32x4_t *>(base + static_cast<int64_t>(gr) * ld + gk);
      else
        reg[i] = u32x4_t{0, 0, 0, 0};
    }
  }
  __device__ __forceinline__ void store(char *lds, int tid) const {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = tid + i * kGemmThreads;
      *reinterpret_cast<u32x4_t *>(lds + lds_off(c >> 3, c & 7)) = reg[i];
    }
  }
};

// MN-major tile: BK k-rows x 128 contiguous rows of the operand.  Each
// thread loads 4 consecutive k-rows of one 16-byte column group and writes
// them transposed (k contiguous) into LDS.
template <typename T> struct MNMajorLoader;

template <> struct MNMajorLoader<bf16_t> {
  u32x4_t reg[4];  // reg[r] = 8 values of k-row r, columns mb*8 .. mb*8+7

  __device__ __forceinline__ void load(const bf16_t *base, int64_t ld, int row0, int rows,
                                       int k0, int K, int tid) {
    const int kb = tid >> 4, mb = tid & 15;
    const int m = row0 + mb * 8;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int k = k0 + kb * 4 + r;
      if (k < K && m < rows)
        reg[r] = *reinterpret_cast<const u32x4_t *>(base + static_cast<int64_t>(k) * ld + m);
      else
        reg[r] = u32x4_t{0, 0, 0, 0};
    }
  }
  __device__ __forceinline__ void store(char *lds, int tid) const {
    const int kb = tid >> 4, mb = tid & 15;
    const int ch = kb >> 1, half = (kb & 1) * 8;
#pragma unroll
    for (int j = 0; j < 4; ++j) {  // dword j holds columns 2j (low) and 2j+1 (high)
      const uint32_t a0 = reg[0][j], a1 = reg[1][j], a2 = reg[2][j], a3 = reg[3][j];
      const u32x2_t lo = {(a0 & 0xFFFFu) | (a1 << 16), (a2 & 0xFFFFu) | (a3 << 16)};
      const u32x2_t hi = {(a0 >> 16) | (a1 & 0xFFFF0000u), (a2 >> 16) | (a3 & 0xFFFF0000u)};
      const int row = mb * 8 + 2 * j;
      *reinterpret_cast<u32x2_t *>(lds + lds_off(row, ch) + half) = lo;
      *reinterpret_cast<u32x2_t *>(lds + lds_off(row + 1, ch) + half) = hi;
    }
  }
};

template <> struct MNMajorLoader<float> {
  u32x4_t reg[4];  // reg[r] = 4 values of k-row r, columns mb*4 .. mb*4+3

  __device__ __forceinline__ void load(const float *base, int64_t ld, int row0, int rows,
                                       int k0, int K, int tid) {
    const int kb = tid >> 5, mb = tid & 31;
    const int m = row0 + mb * 4;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int k = k0 + kb * 4 + r;
      if (k < K && m < rows)
        reg[r] = *reinterpret_cast<const u32x4_t *>(base + static_cast<int64_t>(k) * ld + m);
      else
        reg[r] = u32x4_t{0, 0, 0, 0};
    }
  }
  __device__ __forceinline__ void store(char *lds, int tid) const {
    const int kb = tid >> 5, mb = tid & 31;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const u32x4_t v = {reg[0][j], reg[1][j], reg[2][j], reg[3][j]};
      *reinterpret_cast<u32x4_t *>(lds + lds_off(mb * 4 + j, kb)) = v;
    }
  }
};

template <typename T, bool KMajor> struct LoaderSel {
  using type = KMajorLoader<T>;
};
template <typename T> struct LoaderSel<T, false> {
  using type = MNMajorLoader<T>;
};

// ------------------------------------------------------------ MFMA step
// One LDS stage (BK of K) of the wave's 2 x 2 block of 32 x 32 outputs.
template <typename T> struct MfmaStage;

template <> struct MfmaStage<bf16_t> {
  __device__ __forceinline__ static void run(const char *a_lds, const char *b_lds, int a_row0,
                                             int b_row0, int lane, f32x16_t (&acc)[2][2]) {
    const int r = lane & 31, half = lane >> 5;
#pragma unroll
    for (int s = 0; s < 4; ++s) {  // 4 x 16 = 64 = BK
      const int ch = s * 2 + half;
      bf16x8_t a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        a[i] = *reinterpret_cast<const bf16x8_t *>(a_lds + lds_off(a_row0 + i * 32 + r, ch));
        b[i] = *reinterpret_cast<const bf16x8_t *>(b_lds + lds_off(b_row0 + i * 32 + r, ch));
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  }
};

template <> struct MfmaStage<float> {
  __device__ __forceinline__ static void run(const char *a_lds, const char *b_lds, int a_row0,
                                             int b_row0, int lane, f32x16_t (&acc)[2][2]) {
    const int r = lane & 31, half = lane >> 5;
#pragma unroll
    for (int s = 0; s < 2; ++s) {  // 2 x 16 = 32 = BK
      f32x4_t a[2][2], b[2][2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          const int ch = s * 4 + half * 2 + c;
          a[i][c] = *reinterpret_cast<const f32x4_t *>(a_lds + lds_off(a_row0 + i * 32 + r, ch));
          b[i][c] = *reinterpret_cast<const f32x4_t *>(b_lds + lds_off(b_row0 + i * 32 + r, ch));
        }
#pragma unroll
      for (int e = 0; e < 8; ++e)
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i][e >> 2][e & 3], b[j][e >> 2][e & 3],
                                                              acc[i][j], 0, 0, 0);
    }
  }
};

// Position of accumulator element (i, j, v) of a lane:
//   row = m0 + wave_m*64 + i*32 + (v/4)*8 + (lane/32)*4 + v%4
//   col = n0 + wave_n*64 + j*32 + lane%32
struct TileCtx {
  int M, N;            // problem bounds of C
  int m0, n0;          // tile origin
  int tile_m, tile_n;  // tile indices
  int wave_m, wave_n, lane;
  char *smem;          // >= 64 KB of LDS, free for the epilogue

  __device__ __forceinline__ int row(int i, int v) const {
    return m0 + wave_m * 64 + i * 32 + (v >> 2) * 8 + (lane >> 5) * 4 + (v & 3);
  }
  __device__ __forceinline__ int col(int j) const { return n0 + wave_n * 64 + j * 32 + (lane & 31); }
  // column index inside the tile
  __device__ __forceinline__ int tcol(int j) const { return wave_n * 64 + j * 32 + (lane & 31); }
};

// Column reduction of per-lane partial values over the tile's 128 rows:
// lanes l and l+32 hold the same column, and the two wave rows meet in LDS.
// `part[j]` is the lane's partial for its column j; returns the tile total.
template <bool IsMax>
__device__ __forceinline__ void tile_col_reduce(const TileCtx &t, float (&part)[2]) {
  float *red = reinterpret_cast<float *>(t.smem);
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const float o = __shfl_xor(part[j], 32);
    part[j] = IsMax ? fmaxf(part[j], o) : part[j] + o;
  }
  if (t.lane < 32) {
#pragma unroll
    for (int j = 0; j < 2; ++j) red[t.wave_m * kBN + t.tcol(j)] = part[j];
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const float a = red[t.tcol(j)], b = red[kBN + t.tcol(j)];
    part[j] = IsMax ? fmaxf(a, b) : a + b;
  }
  __syncthreads();
}

// ----------------------------------------------------------------- kernel
template <typename T, bool AK, bool BKM, class Epi>
__global__ __launch_bounds__(kGemmThreads, 2) void gemm_kernel(Operand A, Operand B, GemmShape s,
                                                                typename Epi::Params ep) {
  __shared__ __attribute__((aligned(16))) char smem[2 * kStageBytes];
  constexpr int BK = 8 * Elem<T>::CH;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wave_m = wave >> 1, wave_n = wave & 1;
  const int tiles_n = cdiv(s.N, kBN);
  const int tile_m = blockIdx.x / tiles_n, tile_n = blockIdx.x % tiles_n;
  const int m0 = tile_m * kBM, n0 = tile_n * kBN;
  const T *a_ptr = static_cast<const T *>(A.ptr);
  const T *b_ptr = static_cast<const T *>(B.ptr);

  typename LoaderSel<T, AK>::type la;
  typename LoaderSel<T, BKM>::type lb;
  f32x16_t acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

  const int nk = cdiv(s.K, BK);
  la.load(a_ptr, A.ld, m0, s.M, 0, s.K, tid);
  lb.load(b_ptr, B.ld, n0, s.N, 0, s.K, tid);
  la.store(smem, tid);
  lb.store(smem + kBM * kRowBytes, tid);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const bool more = kt + 1 < nk;
    if (more) {
      la.load(a_ptr, A.ld, m0, s.M, (kt + 1) * BK, s.K, tid);
      lb.load(b_ptr, B.ld, n0, s.N, (kt + 1) * BK, s.K, tid);
    }
    const char *stage = smem + (kt & 1) * kStageBytes;
    MfmaStage<T>::run(stage, stage + kBM * kRowBytes, wave_m * 64, wave_n * 64, lane, acc);
    if (more) {
      char *next = smem + ((kt + 1) & 1) * kStageBytes;
      la.store(next, tid);
      lb.store(next + kBM * kRowBytes, tid);
    }
    __syncthreads();
  }

  TileCtx t{s.M, s.N, m0, n0, tile_m, tile_n, wave_m, wave_n, lane, smem};
  Epi::apply(ep, acc, t);
}

template <typename T, bool AK, bool BKM, class Epi>
hipError_t launch_gemm(Operand A, Operand B, GemmShape s, const typename Epi::Params &ep,
                       hipStream_t stream) {
  const int64_t blocks = static_cast<int64_t>(cdiv(s.M, kBM)) * cdiv(s.N, kBN);
  if (blocks <= 0) return hipSuccess;
  hipLaunchKernelGGL((gemm_kernel<T, AK, BKM, Epi>), dim3(static_cast<unsigned>(blocks)),
                     dim3(kGemmThreads), 0, stream, A, B, s, ep);
  return hipGetLastError();
}

}  // namespace ee
