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
// A tile configuration fixes the output tile (BM x BN) and the part of it
// each wave64 owns (WM x WN = MB x NB blocks of 32 x 32 accumulators).  Each
// LDS tile row holds 128 bytes of K (64 bf16 or 32 fp32 values),
// XOR-swizzled in 16-byte chunks so that fragment reads are free of bank
// conflicts (see lds_off).  Two LDS stages; the next stage's global loads are in
// flight (in registers) while the current stage feeds the matrix cores.
//
// Blocks are ordered for the L2 of each XCD: the hardware hands block b to
// XCD b % 8, so consecutive logical tiles are given to the same XCD, and
// logical tiles walk GROUP_M tile rows at a time (the concurrent tiles of an
// XCD then share a few A and B panels).
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

constexpr int kRowBytes = 128;
constexpr int kNumXcd = 8;
constexpr int kGroupM = 4;

template <int BM_, int BN_, int WM_, int WN_, int MIN_BLOCKS_, int PGR_>
struct TileCfg {
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_;
  static constexpr int MIN_BLOCKS = MIN_BLOCKS_;  // workgroups per CU the registers must allow
  static constexpr int PGR = PGR_;                // stages of global loads in flight (register sets)
  static constexpr int WAVES_M = BM / WM, WAVES_N = BN / WN;
  static constexpr int THREADS = WAVES_M * WAVES_N * 64;
  static constexpr int MB = WM / 32, NB = WN / 32;
  static constexpr int STAGE_BYTES = (BM + BN) * kRowBytes;
};
// 128 x 128 tile, 64 x 64 per wave: any operand layout, bf16 or fp32.
using CfgSmall = TileCfg<128, 128, 64, 64, 2, 1>;
// 256 x 256 tile, 8 waves of 128 x 64 (two waves per SIMD): K-major bf16
// operands.  1.5x the MFMA work per byte read from LDS of the small tile,
// and a second wave per SIMD to issue while the other waits.
using CfgBig8 = TileCfg<256, 256, 128, 64, 1, 1>;
// 256 x 256 tile, 4 waves of 128 x 128 with two stages of global loads in
// flight: twice the MFMA work per LDS byte of the small tile, and enough
// loads outstanding to cover the latency of L2 misses.
using CfgBig4 = TileCfg<256, 256, 128, 128, 1, 1>;
#ifndef EE_BIG_CFG
#define EE_BIG_CFG CfgBig8
#endif
using CfgBig = EE_BIG_CFG;

template <typename T> struct Elem;
template <> struct Elem<bf16_t> {
  static constexpr int CH = 8;  // elements per 16-byte chunk
};
template <> struct Elem<float> {
  static constexpr int CH = 4;
};

__host__ __device__ constexpr int cdiv(int64_t a, int64_t b) { return static_cast<int>((a + b - 1) / b); }

// Byte offset of 16-byte chunk `ch` (0..7) of LDS tile row `row`.  A
// ds_read_b128 is served 16 lanes at a time from 256 bytes of banks, i.e.
// two 128-byte tile rows; the 16 lanes of a fragment read read 16
// consecutive rows at one logical chunk, so within every aligned group of 16
// rows, rows of equal parity must land on distinct chunks: the XOR key's
// bits come from row / 2.  That key repeats every 16 rows, so a lane's
// fragment rows 32 apart share one swizzle and their addresses differ by a
// constant.  Tiles written by the MN-major bf16 loader, whose lanes write
// rows 8 apart, fold row / 16 into the key as well (WIDE), which spreads
// those writes over all chunks.
template <bool WIDE>
__device__ __forceinline__ int lds_key(int row) {
  return WIDE ? ((row >> 1) ^ (row >> 4)) & 7 : (row >> 1) & 7;
}
template <bool WIDE = false>
__device__ __forceinline__ int lds_off(int row, int ch) {
  return row * kRowBytes + ((ch ^ lds_key<WIDE>(row)) << 4);
}

// ---------------------------------------------------------------- loaders
// K-major tile: ROWS rows x 8 chunks of 16 bytes.  Each thread's byte
// offsets inside the tile's row panel are computed once (32-bit: a panel
// spans at most ROWS x 32768 x 4 bytes); per stage only the uniform panel
// base moves, so every load is a scalar base plus a per-thread offset.
template <typename T, int ROWS, int THREADS, int GROUPS>
struct KMajorLoader {
  static constexpr int CH = Elem<T>::CH;
  static constexpr int PER = ROWS * 8 / THREADS;  // 16-byte loads per thread per stage
  static constexpr int PG = PER / GROUPS;         // loads per group
  static_assert(PER % GROUPS == 0, "stage loads must split evenly over the substeps");
  u32x4_t reg[PER];
  uint32_t off[PER];

  // Rows past the operand's end are clamped to its last row: they only feed
  // output rows or columns that the epilogues never store.
  __device__ __forceinline__ void init(int64_t ld, int row0, int rows, int /*K*/, int tid) {
    static_for<PER>([&](auto i) EE_ALWAYS_INLINE {
      const int c = tid + i * THREADS;
      const int r = min(row0 + (c >> 3), rows - 1) - row0;
      off[i] = static_cast<uint32_t>((static_cast<int64_t>(r) * ld + (c & 7) * CH) * sizeof(T));
    });
  }
  // Group g of the stage starting at K offset k0 (a multiple of the stage
  // depth; K itself is one too, checked by the launcher): no load is
  // predicated, since predicated loads would split the code into blocks
  // across which the compiler can only wait for every outstanding load.
  template <int G>
  __device__ __forceinline__ void load(const T *base, int64_t ld, int row0, int k0) {
    const char *panel = reinterpret_cast<const char *>(base + static_cast<int64_t>(row0) * ld + k0);
    static_for<PG>([&](auto q) EE_ALWAYS_INLINE {
      constexpr int i = G * PG + decltype(q)::value;
      reg[i] = *reinterpret_cast<const u32x4_t *>(panel + off[i]);
    });
  }
  template <int G>
  __device__ __forceinline__ void store(char *lds, int tid) const {
    static_for<PG>([&](auto q) EE_ALWAYS_INLINE {
      constexpr int i = G * PG + decltype(q)::value;
      const int c = tid + i * THREADS;
      *reinterpret_cast<u32x4_t *>(lds + lds_off(c >> 3, c & 7)) = reg[i];
    });
  }
};

// MN-major tile: BK k-rows x ROWS contiguous operand rows, written
// transposed (k contiguous) into LDS.
template <typename T, int ROWS, int THREADS> struct MNMajorLoader;

// Adapter giving the fp32 MN-major loader the grouped interface: the whole
// stage is loaded and stored by group 0.
template <typename T, int ROWS, int THREADS, int GROUPS>
struct MNMajorLoaderGrouped : MNMajorLoader<T, ROWS, THREADS> {
  int rows_, K_, tid_;
  __device__ __forceinline__ void init(int64_t, int, int rows, int K, int tid) {
    rows_ = rows;
    K_ = K;
    tid_ = tid;
  }
  template <int G>
  __device__ __forceinline__ void load(const T *base, int64_t ld, int row0, int k0) {
    if constexpr (G == 0) MNMajorLoader<T, ROWS, THREADS>::load(base, ld, row0, rows_, k0, K_, tid_);
  }
  template <int G>
  __device__ __forceinline__ void store(char *lds, int tid) const {
    if constexpr (G == 0) MNMajorLoader<T, ROWS, THREADS>::store(lds, tid);
  }
};

// bf16, 64 k-rows x ROWS operand rows per stage, in blocks of 4 k-rows x 8
// operand rows (one 16-byte load per k-row), one block per thread.  Inside
// a wave, lane bits 0-2 pick 8 consecutive column groups (128 contiguous
// bytes of one k-row per load) and bits 3-5 pick the k-block, so each load
// instruction reads whole 128-byte lines.  A block becomes 8 LDS rows of 4 k
// values (8 bytes); each ds_write_b64 writes the even rows of half the lanes
// and the odd rows of the other half, which with the WIDE lds_key reaches
// every bank.
// The byte shuffles are v_perm_b32, whose per-lane selector also makes that
// even/odd choice.  The whole stage is loaded and written in the first
// substep: the writes need all four k-rows of a block, and loading them at
// once gives each a full stage of latency.
// K-rows past the end re-read the last k-row; with ZERO_TAIL they are
// written to LDS as zeros.  One operand of a product zeroed is enough, so
// only the A side pays for it.
template <int ROWS, int THREADS, int GROUPS, bool ZERO_TAIL>
struct MNMajorLoaderB16 {
  static constexpr int MBW = ROWS / 64;  // 8-block column groups per tile
  static_assert(16 * ROWS / 8 == THREADS, "one 4 x 8 block per thread");
  u32x4_t reg[4];   // k-rows 0..3 of the block
  uint32_t goff;    // byte offset of the block's first k-row in a stage's panel
  int kr0;          // first k-row of the block inside the stage
  int lim;          // last valid k-row of the block (relative), as of the last load
  int K_;
  int lbase;        // LDS byte offset of the block's first row (with the even/odd choice)
  int c0;           // logical chunk XOR the rows' swizzle key (before the row pair index)
  uint32_t sel_first;  // v_perm_b32 selector of the row written first
  int dsec;             // byte distance from the first row written to the second

  __device__ __forceinline__ void init(int64_t ld, int row0, int rows, int K, int tid) {
    const int lane = tid & 63, wb = tid >> 6;
    const int mb = (lane & 7) + 8 * (wb % MBW);
    const int kb = (lane >> 3) + 8 * (wb / MBW);
    const int mcol = min(row0 + mb * 8, rows - 8) - row0;  // rows is a multiple of 8
    kr0 = kb * 4;
    goff = static_cast<uint32_t>((static_cast<int64_t>(kr0) * ld + mcol) * 2);
    K_ = K;
    lim = 3;
    const int sw = (lane >> 5) & 1;  // this lane writes the odd row of each pair first
    // rows mb*8 + 2j + {0, 1} share lds_key = K0 ^ j (j < 4)
    const int key0 = ((4 * (mb & 1)) ^ ((mb >> 1) & 7)) & 7;
    c0 = (kb >> 1) ^ key0;
    lbase = mb * 8 * kRowBytes + sw * kRowBytes + (kb & 1) * 8;
    // v_perm_b32(x = k-row pair high, y = k-row pair low): even operand row
    // takes the low 16 bits of both, odd operand row the high 16 bits.
    sel_first = sw ? 0x07060302u : 0x05040100u;
    dsec = sw ? -kRowBytes : kRowBytes;
  }
  template <int G>
  __device__ __forceinline__ void load(const bf16_t *base, int64_t ld, int row0, int k0) {
    if constexpr (G == 0) {
      const char *panel = reinterpret_cast<const char *>(base + static_cast<int64_t>(k0) * ld + row0);
      const int l = min(3, K_ - 1 - k0 - kr0);  // k-rows past K re-read the last one
      // l < 0 when the whole block lies past K: the (negative) row offset
      // then points back at k-row K - 1, and goff + offset stays >= 0.
      const int ld2 = static_cast<int>(ld * 2);  // < 2^23, checked by the launcher
      static_for<4>([&](auto r) EE_ALWAYS_INLINE {
        const int rr = min(static_cast<int>(decltype(r)::value), l);
        reg[r] = *reinterpret_cast<const u32x4_t *>(panel + (goff + static_cast<uint32_t>(__mul24(rr, ld2))));
      });
      if constexpr (ZERO_TAIL) lim = l;
    }
  }
  template <int G>
  __device__ __forceinline__ void store(char *lds, int) const {
    if constexpr (G == 0) {
      u32x4_t a[4];
      static_for<4>([&](auto r) EE_ALWAYS_INLINE {
        constexpr int R = decltype(r)::value;
        if constexpr (ZERO_TAIL) {
          const bool ok = R <= lim;
          static_for<4>([&](auto j) EE_ALWAYS_INLINE { a[R][decltype(j)::value] = ok ? reg[R][decltype(j)::value] : 0u; });
        } else {
          a[R] = reg[R];
        }
      });
      static_for<4>([&](auto jj) EE_ALWAYS_INLINE {
        constexpr int j = decltype(jj)::value;
        // dword j of a k-row holds operand rows 2j (low half) and 2j+1 (high half)
        const uint32_t sel_second = sel_first ^ 0x02020202u;  // the other half of each dword
        const u32x2_t first = {__builtin_amdgcn_perm(a[1][j], a[0][j], sel_first),
                               __builtin_amdgcn_perm(a[3][j], a[2][j], sel_first)};
        const u32x2_t second = {__builtin_amdgcn_perm(a[1][j], a[0][j], sel_second),
                                __builtin_amdgcn_perm(a[3][j], a[2][j], sel_second)};
        const int off = lbase + j * 2 * kRowBytes + ((c0 ^ j) << 4);
        *reinterpret_cast<u32x2_t *>(lds + off) = first;
        *reinterpret_cast<u32x2_t *>(lds + off + dsec) = second;
      });
    }
  }
};

template <int ROWS, int THREADS> struct MNMajorLoader<float, ROWS, THREADS> {
  static constexpr int GROUPS = ROWS / 4;
  static constexpr int PER = (32 / 4) * GROUPS / THREADS;
  u32x4_t reg[PER][4];  // reg[p][r] = 4 values of k-row r

  __device__ __forceinline__ void load(const float *base, int64_t ld, int row0, int rows,
                                       int k0, int K, int tid) {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int b = tid + p * THREADS;
      const int kb = b / GROUPS, mb = b % GROUPS;
      const int m = min(row0 + mb * 4, rows - 4);  // rows is a multiple of 4
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int k = k0 + kb * 4 + r;
        const u32x4_t v = *reinterpret_cast<const u32x4_t *>(base + static_cast<int64_t>(min(k, K - 1)) * ld + m);
        reg[p][r] = k < K ? v : u32x4_t{0, 0, 0, 0};
      }
    }
  }
  __device__ __forceinline__ void store(char *lds, int tid) const {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int b = tid + p * THREADS;
      const int kb = b / GROUPS, mb = b % GROUPS;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const u32x4_t v = {reg[p][0][j], reg[p][1][j], reg[p][2][j], reg[p][3][j]};
        *reinterpret_cast<u32x4_t *>(lds + lds_off(mb * 4 + j, kb)) = v;
      }
    }
  }
};

template <typename T, bool KMajor, int ROWS, int THREADS, int GROUPS, bool ZERO_TAIL> struct LoaderSel {
  using type = KMajorLoader<T, ROWS, THREADS, GROUPS>;
};
template <int ROWS, int THREADS, int GROUPS, bool ZERO_TAIL> struct LoaderSel<float, false, ROWS, THREADS, GROUPS, ZERO_TAIL> {
  using type = MNMajorLoaderGrouped<float, ROWS, THREADS, GROUPS>;
};
template <int ROWS, int THREADS, int GROUPS, bool ZERO_TAIL> struct LoaderSel<bf16_t, false, ROWS, THREADS, GROUPS, ZERO_TAIL> {
  using type = MNMajorLoaderB16<ROWS, THREADS, GROUPS, ZERO_TAIL>;
};


// ------------------------------------------------------------ MFMA step
// Fragments of one K substep (16 values of K) for the wave's MB x NB blocks
// of 32 x 32, read from one LDS stage, and the MFMAs that consume them.
template <typename T, class Cfg, bool A_WIDE, bool B_WIDE> struct Frags;

template <class Cfg, bool A_WIDE, bool B_WIDE> struct Frags<bf16_t, Cfg, A_WIDE, B_WIDE> {
  static constexpr int MB = Cfg::MB, NB = Cfg::NB;
  static constexpr int SUBSTEPS = 4;  // 4 x 16 = 64 values of K per stage
  static constexpr int MMAS = MB * NB;  // MFMAs per substep
  bf16x8_t a[MB], b[NB];

  __device__ __forceinline__ void load(const char *a_lds, const char *b_lds, int a_row0, int b_row0,
                                       int lane, int s) {
    const int r = lane & 31, ch = s * 2 + (lane >> 5);
    static_for<MB>([&](auto i) EE_ALWAYS_INLINE {
      a[i] = *reinterpret_cast<const bf16x8_t *>(a_lds + lds_off<A_WIDE>(a_row0 + i * 32 + r, ch));
    });
    static_for<NB>([&](auto j) EE_ALWAYS_INLINE {
      b[j] = *reinterpret_cast<const bf16x8_t *>(b_lds + lds_off<B_WIDE>(b_row0 + j * 32 + r, ch));
    });
  }
  __device__ __forceinline__ void mma(f32x16_t (&acc)[MB][NB]) const {
    static_for<MB>([&](auto i) EE_ALWAYS_INLINE {
      static_for<NB>([&](auto j) EE_ALWAYS_INLINE {
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
      });
    });
  }
};

template <class Cfg, bool A_WIDE, bool B_WIDE> struct Frags<float, Cfg, A_WIDE, B_WIDE> {
  static_assert(!A_WIDE && !B_WIDE, "fp32 tiles use the narrow swizzle");
  static constexpr int MB = Cfg::MB, NB = Cfg::NB;
  static constexpr int SUBSTEPS = 2;  // 2 x 16 = 32 values of K per stage
  static constexpr int MMAS = 8 * MB * NB;  // MFMAs per substep
  f32x4_t a[MB][2], b[NB][2];

  __device__ __forceinline__ void load(const char *a_lds, const char *b_lds, int a_row0, int b_row0,
                                       int lane, int s) {
    const int r = lane & 31, half = lane >> 5;
    static_for<2>([&](auto c) EE_ALWAYS_INLINE {
      const int ch = s * 4 + half * 2 + c;
      static_for<MB>([&](auto i) EE_ALWAYS_INLINE {
        a[i][c] = *reinterpret_cast<const f32x4_t *>(a_lds + lds_off(a_row0 + i * 32 + r, ch));
      });
      static_for<NB>([&](auto j) EE_ALWAYS_INLINE {
        b[j][c] = *reinterpret_cast<const f32x4_t *>(b_lds + lds_off(b_row0 + j * 32 + r, ch));
      });
    });
  }
  __device__ __forceinline__ void mma(f32x16_t (&acc)[MB][NB]) const {
    static_for<8>([&](auto e) EE_ALWAYS_INLINE {
      static_for<MB>([&](auto i) EE_ALWAYS_INLINE {
        static_for<NB>([&](auto j) EE_ALWAYS_INLINE {
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i][e / 4][decltype(e)::value % 4],
                                                            b[j][e / 4][decltype(e)::value % 4], acc[i][j],
                                                            0, 0, 0);
        });
      });
    });
  }
};

// Position of accumulator element (i, j, v) of a lane:
//   row = m0 + wave_m*WM + i*32 + (v/4)*8 + (lane/32)*4 + v%4
//   col = n0 + wave_n*WN + j*32 + lane%32
template <class Cfg>
struct TileCtx {
  static constexpr int MB = Cfg::MB, NB = Cfg::NB;
  int M, N;            // problem bounds of C
  int m0, n0;          // tile origin
  int tile_m, tile_n;  // tile indices
  int wave_m, wave_n, lane;
  char *smem;          // LDS free for the epilogue (>= WAVES_M * BN floats)

  __device__ __forceinline__ int row(int i, int v) const {
    return m0 + wave_m * Cfg::WM + i * 32 + (v >> 2) * 8 + (lane >> 5) * 4 + (v & 3);
  }
  __device__ __forceinline__ int col(int j) const { return n0 + tcol(j); }
  // column index inside the tile
  __device__ __forceinline__ int tcol(int j) const { return wave_n * Cfg::WN + j * 32 + (lane & 31); }
};

// Column reduction of per-lane partial values over the tile's BM rows: lanes
// l and l+32 hold the same column, and the wave rows meet in LDS.  `part[j]`
// is the lane's partial for its column j; on return it holds the tile total.
template <bool IsMax, class Cfg>
__device__ __forceinline__ void tile_col_reduce(const TileCtx<Cfg> &t, float (&part)[Cfg::NB]) {
  float *red = reinterpret_cast<float *>(t.smem);
  static_for<Cfg::NB>([&](auto j) EE_ALWAYS_INLINE {
    const float o = __shfl_xor(part[j], 32);
    part[j] = IsMax ? fmaxf(part[j], o) : part[j] + o;
  });
  if (t.lane < 32) static_for<Cfg::NB>([&](auto j) EE_ALWAYS_INLINE { red[t.wave_m * Cfg::BN + t.tcol(j)] = part[j]; });
  __syncthreads();
  static_for<Cfg::NB>([&](auto j) EE_ALWAYS_INLINE {
    float a = red[t.tcol(j)];
    static_for<Cfg::WAVES_M - 1>([&](auto w) EE_ALWAYS_INLINE {
      const float b = red[(w + 1) * Cfg::BN + t.tcol(j)];
      a = IsMax ? fmaxf(a, b) : a + b;
    });
    part[j] = a;
  });
  __syncthreads();
}

// Logical tile of this block (XCD-aware, GROUP_M-grouped order).
__device__ __forceinline__ void tile_of_block(int tiles_m, int tiles_n, int &tile_m, int &tile_n) {
  const int nblk = gridDim.x, b = blockIdx.x;
  const int per = nblk / kNumXcd, rem = nblk % kNumXcd;
  const int xcd = b % kNumXcd, idx = b / kNumXcd;
  const int logical = xcd < rem ? xcd * (per + 1) + idx : rem * (per + 1) + (xcd - rem) * per + idx;
  const int in_group = kGroupM * tiles_n;
  const int first_m = (logical / in_group) * kGroupM;
  const int gm = min(tiles_m - first_m, kGroupM);
  const int r = logical % in_group;
  tile_m = first_m + r % gm;
  tile_n = r / gm;
}

// ----------------------------------------------------------------- kernel
template <typename T, bool AK, bool BKM, class Epi, class Cfg>
__global__ __launch_bounds__(Cfg::THREADS, Cfg::MIN_BLOCKS) void gemm_kernel(Operand A, Operand B, GemmShape s,
                                                                typename Epi::Params ep) {
  __shared__ __attribute__((aligned(16))) char smem[2 * Cfg::STAGE_BYTES];
  constexpr int BK = 8 * Elem<T>::CH;
  constexpr int MB = Cfg::MB, NB = Cfg::NB;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wave_m = wave / Cfg::WAVES_N, wave_n = wave % Cfg::WAVES_N;
  const int tiles_m = cdiv(s.M, Cfg::BM), tiles_n = cdiv(s.N, Cfg::BN);
  int tile_m, tile_n;
  tile_of_block(tiles_m, tiles_n, tile_m, tile_n);
  const int m0 = tile_m * Cfg::BM, n0 = tile_n * Cfg::BN;
  const T *a_ptr = static_cast<const T *>(A.ptr);
  const T *b_ptr = static_cast<const T *>(B.ptr);

  constexpr bool kB16 = std::is_same<T, bf16_t>::value;
  using F = Frags<T, Cfg, kB16 && !AK, kB16 && !BKM>;
  constexpr int SUB = F::SUBSTEPS;
  typename LoaderSel<T, AK, Cfg::BM, Cfg::THREADS, SUB, true>::type la;
  typename LoaderSel<T, BKM, Cfg::BN, Cfg::THREADS, SUB, false>::type lb;
  la.init(A.ld, m0, s.M, s.K, tid);
  lb.init(B.ld, n0, s.N, s.K, tid);
  f32x16_t acc[MB][NB];
  static_for<MB>([&](auto i) EE_ALWAYS_INLINE {
    static_for<NB>([&](auto j) EE_ALWAYS_INLINE {
      static_for<16>([&](auto v) EE_ALWAYS_INLINE { acc[i][j][decltype(v)::value] = 0.0f; });
    });
  });

  // Software pipeline over K stages (BK values of K each).  Registers hold
  // stage kt + 1 while stage kt is consumed from LDS.  Each of the stage's
  // substeps (16 values of K) interleaves, MFMA by MFMA:
  //   * the fragment reads of the next substep,
  //   * its share of the LDS writes of stage kt + 1 (the other buffer),
  //   * its share of the global loads of stage kt + 2 into the registers
  //     those writes just drained.
  // A wave issues in order, so bursts of memory instructions would hold up
  // its MFMAs; spread out, they issue while the matrix core is busy.  The
  // writes of stage kt + 1 are finished by the second-to-last substep; the
  // barrier follows it, and the last substep then reads the first fragments
  // of stage kt + 1 while its own MFMAs run, so no stage starts by waiting
  // for LDS.  The code of a stage has no branches (loads past the last
  // stage re-read it), so the scheduler sees each stage as one region.
  constexpr int B_OFF = Cfg::BM * kRowBytes;
  const int nk = cdiv(s.K, BK);
  const int a_row0 = wave_m * Cfg::WM, b_row0 = wave_n * Cfg::WN;
  static_for<SUB>([&](auto g) EE_ALWAYS_INLINE {
    la.template load<decltype(g)::value>(a_ptr, A.ld, m0, 0);
    lb.template load<decltype(g)::value>(b_ptr, B.ld, n0, 0);
  });
  static_for<SUB>([&](auto g) EE_ALWAYS_INLINE {
    la.template store<decltype(g)::value>(smem, tid);
    lb.template store<decltype(g)::value>(smem + B_OFF, tid);
  });
  const int k1 = min(1, nk - 1) * BK;
  static_for<SUB>([&](auto g) EE_ALWAYS_INLINE {
    la.template load<decltype(g)::value>(a_ptr, A.ld, m0, k1);
    lb.template load<decltype(g)::value>(b_ptr, B.ld, n0, k1);
  });
  __syncthreads();
  F f0, f1;
  f0.load(smem, smem + B_OFF, a_row0, b_row0, lane, 0);
  for (int kt = 0; kt < nk; ++kt) {
    const char *cur = smem + (kt & 1) * Cfg::STAGE_BYTES;
    char *next = smem + ((kt + 1) & 1) * Cfg::STAGE_BYTES;
    const int k2 = min(kt + 2, nk - 1) * BK;
    static_for<SUB>([&](auto st) EE_ALWAYS_INLINE {
      constexpr int sub = decltype(st)::value;
      F &now = (sub % 2 == 0) ? f0 : f1;
      F &later = (sub % 2 == 0) ? f1 : f0;
      if constexpr (sub + 1 < SUB)
        later.load(cur, cur + B_OFF, a_row0, b_row0, lane, sub + 1);
      else
        later.load(next, next + B_OFF, a_row0, b_row0, lane, 0);  // next stage, published by the barrier
      if constexpr (sub < SUB - 2) {
        la.template store<sub>(next, tid);
        lb.template store<sub>(next + B_OFF, tid);
        la.template load<sub>(a_ptr, A.ld, m0, k2);
        lb.template load<sub>(b_ptr, B.ld, n0, k2);
      } else if constexpr (sub == SUB - 2) {
        static_for<2>([&](auto gg) EE_ALWAYS_INLINE {
          constexpr int g = SUB - 2 + decltype(gg)::value;
          la.template store<g>(next, tid);
          lb.template store<g>(next + B_OFF, tid);
          la.template load<g>(a_ptr, A.ld, m0, k2);
          lb.template load<g>(b_ptr, B.ld, n0, k2);
        });
      }
      now.mma(acc);
      static_for<F::MMAS>([&](auto) EE_ALWAYS_INLINE {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
        __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);  // DS write
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // VMEM read
      });
      if constexpr (sub == SUB - 2) __syncthreads();
    });
  }

  TileCtx<Cfg> t{s.M, s.N, m0, n0, tile_m, tile_n, wave_m, wave_n, lane, smem};
  Epi::template apply<Cfg>(ep, acc, t);
}

template <typename T, bool AK, bool BKM, class Epi, class Cfg>
hipError_t launch_gemm(Operand A, Operand B, GemmShape s, const typename Epi::Params &ep,
                       hipStream_t stream) {
  const int64_t blocks = static_cast<int64_t>(cdiv(s.M, Cfg::BM)) * cdiv(s.N, Cfg::BN);
  if (blocks <= 0) return hipSuccess;
  constexpr int BK = 8 * Elem<T>::CH;
  if (((AK || BKM) && s.K % BK != 0) || (!AK && s.M % 8 != 0) || (!BKM && s.N % 8 != 0))
    return hipErrorInvalidValue;  // shapes the loaders do not handle
  if ((!AK && A.ld >= (int64_t{1} << 22)) || (!BKM && B.ld >= (int64_t{1} << 22)))
    return hipErrorInvalidValue;  // MN-major loaders keep signed 24-bit k-row strides
  hipLaunchKernelGGL((gemm_kernel<T, AK, BKM, Epi, Cfg>), dim3(static_cast<unsigned>(blocks)),
                     dim3(Cfg::THREADS), 0, stream, A, B, s, ep);
  return hipGetLastError();
}

}  // namespace ee
