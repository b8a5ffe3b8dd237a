// Tiled MFMA GEMM for gfx950 with fused epilogues.
//
//   C[m][n] = sum_k A(m, k) * B(n, k)
//
// Each operand is either K-major (element (r, k) at ptr[r*ld + k], K
// contiguous) or MN-major (element (r, k) at ptr[k*ld + r], rows
// contiguous).  K-major tiles sit in LDS as rows of K; bf16 MN-major tiles
// are copied as they are (k-rows) and transposed by the fragment reads
// themselves (ds_read_b64_tr_b16), so neither side spends ALU work on the
// layout.  (fp32 MN-major operands, used only by the fp32 path, are
// transposed in registers on their way into LDS.)
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

#include <algorithm>

#include "ee_device.h"

namespace ee {

struct Operand {
  const void *ptr;
  int64_t ld;         // elements between consecutive rows of the stored matrix
  int64_t pair = 0;   // interleaved pair (KMajorPairLoader): bytes from the first matrix to the second
};

struct GemmShape {
  int M, N, K;
  int kchunk = 0;  // split-K: blockIdx.z covers K values [z kchunk, (z + 1) kchunk); 0 = all of K
};

constexpr int kRowBytes = 128;
constexpr int kNumXcd = 8;
constexpr int kGroupM = 4;
constexpr int kLoopBlocks = 256;  // grid of the looping kernels: one block per CU of a 256-CU GPU (a multiple of kNumXcd)

template <int BM_, int BN_, int WM_, int WN_, int MIN_BLOCKS_>
struct TileCfg {
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_;
  static constexpr int MIN_BLOCKS = MIN_BLOCKS_;  // workgroups per CU the registers must allow
  static constexpr int WAVES_M = BM / WM, WAVES_N = BN / WN;
  static constexpr int THREADS = WAVES_M * WAVES_N * 64;
  static constexpr int MB = WM / 32, NB = WN / 32;
  static constexpr int STAGE_BYTES = (BM + BN) * kRowBytes;
};
// 128 x 128 tile, 64 x 64 per wave: any operand layout, bf16 or fp32.
using CfgSmall = TileCfg<128, 128, 64, 64, 2>;
// 256 x 256 tile, 8 waves of 128 x 64 (two waves per SIMD): every bf16 GEMM.
// 1.5x the MFMA work per byte read from LDS of the small tile, and a second
// wave per SIMD to issue while the other waits.
using CfgBig = TileCfg<256, 256, 128, 64, 1>;

template <typename T> struct Elem;
template <> struct Elem<bf16_t> {
  static constexpr int CH = 8;  // elements per 16-byte chunk
};
template <> struct Elem<float> {
  static constexpr int CH = 4;
};

__host__ __device__ constexpr int cdiv(int64_t a, int64_t b) { return static_cast<int>((a + b - 1) / b); }

// Byte offset of 16-byte chunk `ch` (0..7) of K-major LDS tile row `row`.
// A ds_read_b128 is served 16 lanes at a time from 256 bytes of banks, i.e.
// two 128-byte tile rows; the 16 lanes of a fragment read read 16
// consecutive rows at one logical chunk, so within every aligned group of 16
// rows, rows of equal parity must land on distinct chunks: the XOR key is
// (row / 2) mod 8.  It repeats every 16 rows, so a lane's fragment rows 32
// apart share one swizzle and their addresses differ by a constant.
__device__ __forceinline__ int lds_off(int row, int ch) {
  return row * kRowBytes + ((ch ^ ((row >> 1) & 7)) << 4);
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

// K-major tile whose rows come from two matrices of equal shape, F rows
// each (F a multiple of 32), interleaved in blocks of 32: tile-space row r
// is row (r / 64) * 32 + r % 32 of the first matrix when (r / 32) is even,
// of the second when it is odd.  A wave whose columns are 64 tile rows wide
// then holds both matrices' products for the same 32 rows in its two
// 32-column blocks (the gate and up projections of one set of features).
// Tile rows past 2F are clamped to the last row of the second matrix.
template <typename T, int ROWS, int THREADS, int GROUPS>
struct KMajorPairLoader {
  static constexpr int CH = Elem<T>::CH;
  static constexpr int PER = ROWS * 8 / THREADS;
  static constexpr int PG = PER / GROUPS;
  static_assert(PER % GROUPS == 0, "stage loads must split evenly over the substeps");
  static_assert(ROWS % 64 == 0, "the tile must hold whole 64-row pairs");
  u32x4_t reg[PER];
  int64_t off[PER];  // bytes from the first matrix's row row0 / 2

  // row0: the tile's first tile-space row (a multiple of 64); rows: 2F.
  __device__ __forceinline__ void init(int64_t ld, int row0, int rows, int64_t pair, int tid) {
    static_for<PER>([&](auto i) EE_ALWAYS_INLINE {
      const int c = tid + i * THREADS;
      const int r = min(row0 + (c >> 3), rows - 1);   // tile-space row
      const int f = (r >> 6) * 32 + (r & 31) - row0 / 2;  // row of its matrix, from row0 / 2
      off[i] = (static_cast<int64_t>(f) * ld + (c & 7) * CH) * static_cast<int64_t>(sizeof(T)) +
               (((r >> 5) & 1) ? pair : 0);
    });
  }
  template <int G>
  __device__ __forceinline__ void load(const T *base, int64_t ld, int row0, int k0) {
    const char *panel = reinterpret_cast<const char *>(base + static_cast<int64_t>(row0 / 2) * ld + k0);
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

// Epilogues that take the B operand as an interleaved pair declare
// kPairB = true.
template <class E, class = void> struct EpiPairB : std::false_type {};
template <class E> struct EpiPairB<E, std::void_t<decltype(E::kPairB)>> : std::bool_constant<E::kPairB> {};
// Epilogues whose GEMMs run as one block per CU looping over the tiles.
template <class E, class = void> struct EpiPersistent : std::false_type {};
template <class E>
struct EpiPersistent<E, std::void_t<decltype(E::kPersistent)>> : std::bool_constant<E::kPersistent> {};

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

// bf16 MN-major tile, stored in LDS as it is in memory: 64 k-rows of ROWS
// operand rows (2 ROWS bytes each), 16-byte chunks XOR-swizzled by
// 4 (k mod 4) (see mn_off).  The transpose happens in the fragment reads
// (ds_read_b64_tr_b16, see Frags), so the copy is a plain one: each thread
// moves PER 16-byte chunks, one per substep group, consecutive threads
// along a k-row (whole 128-byte lines per load).  K-rows past the end
// re-read the last k-row; with ZERO_TAIL they are written as zeros.  One
// operand of a product zeroed is enough, so only the A side pays for it.
template <int ROWS>
__device__ __forceinline__ int mn_off(int k, int m) {
  return k * (2 * ROWS) + (((m >> 3) ^ (4 * (k & 3))) << 4) + (m & 7) * 2;
}

template <int ROWS, int THREADS, int GROUPS, bool ZERO_TAIL>
struct MNMajorLoaderB16 {
  static constexpr int CHUNKS = ROWS / 8;               // 16-byte chunks per k-row
  static constexpr int PER = 64 * CHUNKS / THREADS;     // chunks per thread per stage
  static constexpr int PG = PER / GROUPS;
  static_assert(PER % GROUPS == 0 && CHUNKS >= 16, "stage chunks must split evenly; swizzle needs 16 chunks");
  u32x4_t reg[PER];
  uint32_t moff[PER];   // byte offset of the chunk's operand row within a k-row (clamped)
  int kr[PER];          // k-row of the chunk inside the stage
  int loff[PER];        // LDS byte offset of the chunk
  int K_;
  int lim;              // K - 1 - k0 of the last load (k-rows beyond it are past K)

  __device__ __forceinline__ void init(int64_t, int row0, int rows, int K, int tid) {
    K_ = K;
    lim = 63;
    static_for<PER>([&](auto i) EE_ALWAYS_INLINE {
      const int c = tid + decltype(i)::value * THREADS;
      const int k = c / CHUNKS, ch = c % CHUNKS;
      const int m = min(row0 + ch * 8, rows - 8) - row0;  // rows is a multiple of 8
      kr[i] = k;
      moff[i] = static_cast<uint32_t>(m * 2);
      loff[i] = k * (2 * ROWS) + ((ch ^ (4 * (k & 3))) << 4);
    });
  }
  template <int G>
  __device__ __forceinline__ void load(const bf16_t *base, int64_t ld, int row0, int k0) {
    const char *panel = reinterpret_cast<const char *>(base + static_cast<int64_t>(k0) * ld + row0);
    const int l = K_ - 1 - k0;
    const int ld2 = static_cast<int>(ld * 2);  // < 2^23, checked by the launcher
    static_for<PG>([&](auto q) EE_ALWAYS_INLINE {
      constexpr int i = G * PG + decltype(q)::value;
      const int k = min(kr[i], l);
      reg[i] = *reinterpret_cast<const u32x4_t *>(panel + (moff[i] + static_cast<uint32_t>(__mul24(k, ld2))));
    });
    if constexpr (ZERO_TAIL && G == GROUPS - 1) lim = l;
  }
  template <int G>
  __device__ __forceinline__ void store(char *lds, int) const {
    static_for<PG>([&](auto q) EE_ALWAYS_INLINE {
      constexpr int i = G * PG + decltype(q)::value;
      u32x4_t v = reg[i];
      if constexpr (ZERO_TAIL) {
        const bool ok = kr[i] <= lim;
        static_for<4>([&](auto j) EE_ALWAYS_INLINE { v[decltype(j)::value] = ok ? v[decltype(j)::value] : 0u; });
      }
      *reinterpret_cast<u32x4_t *>(lds + loff[i]) = v;
    });
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
template <typename T, class Cfg, bool A_MN, bool B_MN> struct Frags;

typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4_t lds_s16x4_t;

// Lane base offsets of the MFMA fragment reads of one operand of a wave:
// `blocks` blocks of 32 rows from row0.  K-major tiles: row (row0 + 32 b +
// lane % 32), logical chunk (lane / 32) (the substep adds 2 chunks).
// MN-major tiles (k-rows of ROWS operand rows): ds_read_b64_tr_b16 gives
// lane 4a + b of each 16-lane group element b of the 8-byte chunks that
// lanes a, a + 4, a + 8, a + 12 of the group address.  Lane j of group g
// therefore addresses k-row 8 (g / 2) + j / 4 (+ 4 for the second read,
// + 16 per substep) at operand rows m0 + 16 (g % 2) + 4 (j % 4) .. + 3, and
// receives rows m0 + 16 (g % 2) + j at four consecutive k: with the second
// read, the 8 values of K that the MFMA expects of lane (row = lane % 32,
// k = 8 (lane / 32) + e).  K offsets that are multiples of 4 keep the
// swizzle (4 (k mod 4)), so they go into the instruction offset.
template <bool MN, int ROWS>
__device__ __forceinline__ int frag_base(int row0, int lane) {
  if constexpr (MN) {
    const int g = lane >> 4, j = lane & 15;
    return mn_off<ROWS>(8 * (g >> 1) + (j >> 2), row0 + 16 * (g & 1) + 4 * (j & 3));
  } else {
    return 0;  // unused: K-major reads compute lds_off directly
  }
}

template <class Cfg, bool A_MN, bool B_MN> struct Frags<bf16_t, Cfg, A_MN, B_MN> {
  static constexpr int MB = Cfg::MB, NB = Cfg::NB;
  static constexpr int SUBSTEPS = 4;  // 4 x 16 = 64 values of K per stage
  static constexpr int MMAS = MB * NB;  // MFMAs per substep
  bf16x8_t a[MB], b[NB];

  // One operand's fragments of substep s.  `base` = frag_base of each block
  // (MN-major tiles), or the tile's first row (K-major tiles).
  template <bool MN, int ROWS, int NBLK>
  __device__ __forceinline__ static void read(bf16x8_t (&f)[NBLK], const char *lds, const int (&base)[NBLK],
                                              int row0, int lane, int s) {
    if constexpr (MN) {
      static_for<NBLK>([&](auto i) EE_ALWAYS_INLINE {
        const char *p = lds + base[i] + 16 * s * (2 * ROWS);
        const s16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t *)(p));
        const s16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t *)(p + 4 * (2 * ROWS)));
        const s16x4_t both[2] = {lo, hi};
        f[i] = __builtin_bit_cast(bf16x8_t, both);
      });
    } else {
      const int r = lane & 31, ch = s * 2 + (lane >> 5);
      static_for<NBLK>([&](auto i) EE_ALWAYS_INLINE {
        f[i] = *reinterpret_cast<const bf16x8_t *>(lds + lds_off(row0 + i * 32 + r, ch));
      });
    }
  }
  __device__ __forceinline__ void load(const char *a_lds, const char *b_lds, const int (&a_base)[MB],
                                       const int (&b_base)[NB], int a_row0, int b_row0, int lane, int s) {
    read<A_MN, Cfg::BM>(a, a_lds, a_base, a_row0, lane, s);
    read<B_MN, Cfg::BN>(b, b_lds, b_base, b_row0, lane, s);
  }
  __device__ __forceinline__ void mma(f32x16_t (&acc)[MB][NB]) const {
    static_for<MB>([&](auto i) EE_ALWAYS_INLINE {
      static_for<NB>([&](auto j) EE_ALWAYS_INLINE {
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
      });
    });
  }
};

template <class Cfg, bool A_MN, bool B_MN> struct Frags<float, Cfg, A_MN, B_MN> {
  // fp32 MN-major operands are transposed in registers on their way into
  // LDS, so both fp32 operands are read K-major here.
  static constexpr int MB = Cfg::MB, NB = Cfg::NB;
  static constexpr int SUBSTEPS = 2;  // 2 x 16 = 32 values of K per stage
  static constexpr int MMAS = 8 * MB * NB;  // MFMAs per substep
  f32x4_t a[MB][2], b[NB][2];

  __device__ __forceinline__ void load(const char *a_lds, const char *b_lds, const int (&)[MB], const int (&)[NB],
                                       int a_row0, int b_row0, int lane, int s) {
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
  char *smem;          // the tile's LDS (two stages), free for the epilogue after a barrier
  int kz = 0;          // split-K slice of this block (epilogues that support splits offset by it)

  __device__ __forceinline__ int row(int i, int v) const {
    return m0 + wave_m * Cfg::WM + i * 32 + (v >> 2) * 8 + (lane >> 5) * 4 + (v & 3);
  }
  __device__ __forceinline__ int col(int j) const { return n0 + tcol(j); }
  // column index inside the tile
  __device__ __forceinline__ int tcol(int j) const { return wave_n * Cfg::WN + j * 32 + (lane & 31); }
};

// Logical tile of this block (XCD-aware, grouped order).  Blocks that run
// together on one XCD take consecutive logical tiles; the logical order
// walks groups of kGroupM tiles along the dimension with more tiles, sweeping
// the other dimension inside a group, so the operand with more panels is
// streamed once while the few panels of the other stay cache-resident.
__device__ __forceinline__ void tile_of_block(int b, int nblk, int tiles_m, int tiles_n, int &tile_m, int &tile_n) {
  const int per = nblk / kNumXcd, rem = nblk % kNumXcd;
  const int xcd = b % kNumXcd, idx = b / kNumXcd;
  const int logical = xcd < rem ? xcd * (per + 1) + idx : rem * (per + 1) + (xcd - rem) * per + idx;
  const bool swap = tiles_n > tiles_m;
  const int ta = swap ? tiles_n : tiles_m, tb = swap ? tiles_m : tiles_n;  // grouped, swept
  const int in_group = kGroupM * tb;
  const int first = (logical / in_group) * kGroupM;
  const int g = min(ta - first, kGroupM);
  const int r = logical % in_group;
  const int a = first + r % g, c = r / g;
  tile_m = swap ? c : a;
  tile_n = swap ? a : c;
}

// ----------------------------------------------------------------- kernel
// Block b of nblk (b mod 8 = the XCD it runs on) of one GEMM problem, split-K
// slice kz: main loop and epilogue of its tile.  LOOP: the caller loops over
// tiles; the thread index is then opaque to the compiler, so that no address
// it derives is hoisted out of the loop and kept live through the epilogue
// (which spilled registers).
template <typename T, bool AK, bool BKM, class Epi, class Cfg, bool LOOP = false>
__device__ __forceinline__ void gemm_block(const Operand &A, const Operand &B, const GemmShape &s,
                                           const typename Epi::Params &ep, int b, int nblk, int kz, char *smem) {
  constexpr int BK = 8 * Elem<T>::CH;
  constexpr int MB = Cfg::MB, NB = Cfg::NB;
  int tid_v = threadIdx.x;
  if constexpr (LOOP) asm volatile("" : "+v"(tid_v));
  const int tid = tid_v, lane = tid & 63, wave = tid >> 6;
  const int wave_m = wave / Cfg::WAVES_N, wave_n = wave % Cfg::WAVES_N;
  const int tiles_m = cdiv(s.M, Cfg::BM), tiles_n = cdiv(s.N, Cfg::BN);
  int tile_m, tile_n;
  tile_of_block(b, nblk, tiles_m, tiles_n, tile_m, tile_n);
  const int m0 = tile_m * Cfg::BM, n0 = tile_n * Cfg::BN;
  const T *a_ptr = static_cast<const T *>(A.ptr);
  const T *b_ptr = static_cast<const T *>(B.ptr);

  constexpr bool kB16 = std::is_same<T, bf16_t>::value;
  constexpr bool kAMN = kB16 && !AK, kBMN = kB16 && !BKM;  // read with the LDS transpose
  using F = Frags<T, Cfg, kAMN, kBMN>;
  constexpr int SUB = F::SUBSTEPS;
  constexpr bool kPair = EpiPairB<Epi>::value;
  static_assert(!kPair || BKM, "an interleaved pair is read K-major");
  typename LoaderSel<T, AK, Cfg::BM, Cfg::THREADS, SUB, true>::type la;
  std::conditional_t<kPair, KMajorPairLoader<T, Cfg::BN, Cfg::THREADS, SUB>,
                     typename LoaderSel<T, BKM, Cfg::BN, Cfg::THREADS, SUB, false>::type>
      lb;
  la.init(A.ld, m0, s.M, s.K, tid);
  if constexpr (kPair)
    lb.init(B.ld, n0, s.N, B.pair, tid);
  else
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
  const int kbeg = s.kchunk > 0 ? kz * s.kchunk : 0;
  const int kend = s.kchunk > 0 ? min(s.K, kbeg + s.kchunk) : s.K;
  const int nk = cdiv(kend - kbeg, BK);
  const int a_row0 = wave_m * Cfg::WM, b_row0 = wave_n * Cfg::WN;
  static_for<SUB>([&](auto g) EE_ALWAYS_INLINE {
    la.template load<decltype(g)::value>(a_ptr, A.ld, m0, kbeg);
    lb.template load<decltype(g)::value>(b_ptr, B.ld, n0, kbeg);
  });
  static_for<SUB>([&](auto g) EE_ALWAYS_INLINE {
    la.template store<decltype(g)::value>(smem, tid);
    lb.template store<decltype(g)::value>(smem + B_OFF, tid);
  });
  const int k1 = kbeg + min(1, nk - 1) * BK;
  static_for<SUB>([&](auto g) EE_ALWAYS_INLINE {
    la.template load<decltype(g)::value>(a_ptr, A.ld, m0, k1);
    lb.template load<decltype(g)::value>(b_ptr, B.ld, n0, k1);
  });
  __syncthreads();
  int a_base[MB], b_base[NB];
  static_for<MB>([&](auto i) EE_ALWAYS_INLINE { a_base[i] = frag_base<kAMN, Cfg::BM>(a_row0 + 32 * i, lane); });
  static_for<NB>([&](auto j) EE_ALWAYS_INLINE { b_base[j] = frag_base<kBMN, Cfg::BN>(b_row0 + 32 * j, lane); });
  F f0, f1;
  f0.load(smem, smem + B_OFF, a_base, b_base, a_row0, b_row0, lane, 0);
  for (int kt = 0; kt < nk; ++kt) {
    const char *cur = smem + (kt & 1) * Cfg::STAGE_BYTES;
    char *next = smem + ((kt + 1) & 1) * Cfg::STAGE_BYTES;
    const int k2 = kbeg + min(kt + 2, nk - 1) * BK;
    static_for<SUB>([&](auto st) EE_ALWAYS_INLINE {
      constexpr int sub = decltype(st)::value;
      F &now = (sub % 2 == 0) ? f0 : f1;
      F &later = (sub % 2 == 0) ? f1 : f0;
      if constexpr (sub + 1 < SUB)
        later.load(cur, cur + B_OFF, a_base, b_base, a_row0, b_row0, lane, sub + 1);
      else
        later.load(next, next + B_OFF, a_base, b_base, a_row0, b_row0, lane, 0);  // next stage, published by the barrier
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

  TileCtx<Cfg> t{s.M, s.N, m0, n0, tile_m, tile_n, wave_m, wave_n, lane, smem, kz};
  Epi::template apply<Cfg>(ep, acc, t);
}

template <typename T, bool AK, bool BKM, class Epi, class Cfg>
__global__ __launch_bounds__(Cfg::THREADS, Cfg::MIN_BLOCKS) void gemm_kernel(Operand A, Operand B, GemmShape s,
                                                                typename Epi::Params ep) {
  __shared__ __attribute__((aligned(16))) char smem[2 * Cfg::STAGE_BYTES];
  gemm_block<T, AK, BKM, Epi, Cfg>(A, B, s, ep, blockIdx.x, gridDim.x, blockIdx.z, smem);
}

// The same product for a launch that usually has nothing to do: it runs
// only if *run_if is non-zero (a flag an earlier kernel of the stream set),
// one block per CU looping over the tiles.  The grid is a multiple of the
// XCD count, so tile t still runs on XCD t mod 8 and keeps its place in the
// XCD-aware order; when the flag is clear the launch costs one round of
// blocks that read it and return.
template <typename T, bool AK, bool BKM, class Epi, class Cfg>
__global__ __launch_bounds__(Cfg::THREADS, Cfg::MIN_BLOCKS) void gemm_gated_kernel(Operand A, Operand B, GemmShape s,
                                                                      typename Epi::Params ep, const int *run_if) {
  __shared__ __attribute__((aligned(16))) char smem[2 * Cfg::STAGE_BYTES];
  if (*run_if == 0) return;  // the same word for every thread
  const int tiles = cdiv(s.M, Cfg::BM) * cdiv(s.N, Cfg::BN);
  for (int t = blockIdx.x; t < tiles; t += gridDim.x) {
    gemm_block<T, AK, BKM, Epi, Cfg, true>(A, B, s, ep, t, tiles, 0, smem);
    __syncthreads();  // the next tile's first stage overwrites what the epilogue used
  }
}

// One block per CU looping over the tiles, tile t on block t mod gridDim.x
// (a multiple of 8, so on XCD t mod 8 as in the one-block-per-tile launch):
// a CU starts its next tile's loads right after the epilogue's barrier,
// without waiting for a new block to be dispatched (measured at 2.6 us
// between one weight-gradient tile's end and the next one's start on the
// freed CU).
template <typename T, bool AK, bool BKM, class Epi, class Cfg>
__global__ __launch_bounds__(Cfg::THREADS, Cfg::MIN_BLOCKS) void gemm_persistent_kernel(Operand A, Operand B,
                                                                           GemmShape s,
                                                                           typename Epi::Params ep) {
  __shared__ __attribute__((aligned(16))) char smem[2 * Cfg::STAGE_BYTES];
  const int tiles = cdiv(s.M, Cfg::BM) * cdiv(s.N, Cfg::BN);
  for (int t = blockIdx.x; t < tiles; t += gridDim.x) {
    gemm_block<T, AK, BKM, Epi, Cfg, true>(A, B, s, ep, t, tiles, 0, smem);
    __syncthreads();  // the next tile's first stage overwrites what the epilogue used
  }
}

// Two independent problems in one grid: blocks [0, blocks1) take problem 1,
// blocks [base2, gridDim.x) problem 2, where base2 = blocks1 rounded up to a
// multiple of 8 (the blocks in between do nothing), so that both keep the
// XCD-aware tile order.  The hardware dispatches blocks in order, so the
// problems share the GPU only where the first one's last round of tiles
// leaves CUs idle.  Problem 2 may be split along K (s2.kchunk > 0): its
// blocks then run slice by slice, each slice over all of its tiles.
template <typename T, bool AK1, bool BKM1, class Epi1, bool AK2, bool BKM2, class Epi2, class Cfg>
__global__ __launch_bounds__(Cfg::THREADS, Cfg::MIN_BLOCKS) void gemm_pair_kernel(
    Operand A1, Operand B1, GemmShape s1, typename Epi1::Params ep1, Operand A2, Operand B2, GemmShape s2,
    typename Epi2::Params ep2, int blocks1, int base2) {
  __shared__ __attribute__((aligned(16))) char smem[2 * Cfg::STAGE_BYTES];
  const int b = blockIdx.x;
  if (b < blocks1)
    gemm_block<T, AK1, BKM1, Epi1, Cfg>(A1, B1, s1, ep1, b, blocks1, 0, smem);
  else if (b >= base2) {
    const int tiles2 = cdiv(s2.M, Cfg::BM) * cdiv(s2.N, Cfg::BN), b2 = b - base2;
    gemm_block<T, AK2, BKM2, Epi2, Cfg>(A2, B2, s2, ep2, b2 % tiles2, tiles2, b2 / tiles2, smem);
  }
}

// The pair as one block per CU looping over the same block order (logical
// block t on block t mod gridDim.x, a multiple of 8), for two
// weight-gradient products.
template <typename T, bool AK1, bool BKM1, class Epi1, bool AK2, bool BKM2, class Epi2, class Cfg>
__global__ __launch_bounds__(Cfg::THREADS, Cfg::MIN_BLOCKS) void gemm_pair_persistent_kernel(
    Operand A1, Operand B1, GemmShape s1, typename Epi1::Params ep1, Operand A2, Operand B2, GemmShape s2,
    typename Epi2::Params ep2, int blocks1, int base2, int total) {
  __shared__ __attribute__((aligned(16))) char smem[2 * Cfg::STAGE_BYTES];
  const int tiles2 = cdiv(s2.M, Cfg::BM) * cdiv(s2.N, Cfg::BN);
  for (int t = blockIdx.x; t < total; t += gridDim.x) {
    if (t < blocks1) {
      gemm_block<T, AK1, BKM1, Epi1, Cfg, true>(A1, B1, s1, ep1, t, blocks1, 0, smem);
    } else if (t >= base2) {
      const int b2 = t - base2;
      gemm_block<T, AK2, BKM2, Epi2, Cfg, true>(A2, B2, s2, ep2, b2 % tiles2, tiles2, b2 / tiles2, smem);
    }
    __syncthreads();  // the next tile's first stage overwrites what the epilogue used
  }
}

// Shapes the loaders handle.
template <typename T, bool AK, bool BKM>
bool gemm_shape_ok(const Operand &A, const Operand &B, const GemmShape &s) {
  constexpr int BK = 8 * Elem<T>::CH;
  if (((AK || BKM) && s.K % BK != 0) || (!AK && s.M % 8 != 0) || (!BKM && s.N % 8 != 0)) return false;
  // MN-major loaders keep signed 24-bit k-row strides
  return !((!AK && A.ld >= (int64_t{1} << 22)) || (!BKM && B.ld >= (int64_t{1} << 22)));
}

template <typename T, bool AK, bool BKM, class Epi, class Cfg>
hipError_t launch_gemm(Operand A, Operand B, GemmShape s, const typename Epi::Params &ep,
                       hipStream_t stream) {
  const int64_t blocks = static_cast<int64_t>(cdiv(s.M, Cfg::BM)) * cdiv(s.N, Cfg::BN);
  if (blocks <= 0) return hipSuccess;
  constexpr int BK = 8 * Elem<T>::CH;
  if (!gemm_shape_ok<T, AK, BKM>(A, B, s)) return hipErrorInvalidValue;
  int splits = 1;
  if (s.kchunk > 0) {
    if (s.kchunk % BK != 0) return hipErrorInvalidValue;  // slices start on stage boundaries
    splits = cdiv(s.K, s.kchunk);
  }
  if constexpr (EpiPersistent<Epi>::value && std::is_same<T, bf16_t>::value) {
    if (splits == 1 && blocks > 2 * kLoopBlocks) {
      hipLaunchKernelGGL((gemm_persistent_kernel<T, AK, BKM, Epi, Cfg>), dim3(kLoopBlocks), dim3(Cfg::THREADS), 0,
                         stream, A, B, s, ep);
      return hipGetLastError();
    }
  }
  hipLaunchKernelGGL((gemm_kernel<T, AK, BKM, Epi, Cfg>), dim3(static_cast<unsigned>(blocks), 1, splits),
                     dim3(Cfg::THREADS), 0, stream, A, B, s, ep);
  return hipGetLastError();
}

constexpr int kGatedBlocks = kLoopBlocks;

template <typename T, bool AK, bool BKM, class Epi, class Cfg>
hipError_t launch_gemm_gated(Operand A, Operand B, GemmShape s, const typename Epi::Params &ep, const int *run_if,
                             hipStream_t stream) {
  const int64_t tiles = static_cast<int64_t>(cdiv(s.M, Cfg::BM)) * cdiv(s.N, Cfg::BN);
  if (tiles <= 0) return hipSuccess;
  if (s.kchunk != 0 || run_if == nullptr || !gemm_shape_ok<T, AK, BKM>(A, B, s)) return hipErrorInvalidValue;
  const int64_t blocks = std::min<int64_t>(kGatedBlocks, (tiles + kNumXcd - 1) / kNumXcd * kNumXcd);
  hipLaunchKernelGGL((gemm_gated_kernel<T, AK, BKM, Epi, Cfg>), dim3(static_cast<unsigned>(blocks)),
                     dim3(Cfg::THREADS), 0, stream, A, B, s, ep, run_if);
  return hipGetLastError();
}

template <typename T, bool AK1, bool BKM1, class Epi1, bool AK2, bool BKM2, class Epi2, class Cfg>
hipError_t launch_gemm_pair(Operand A1, Operand B1, GemmShape s1, const typename Epi1::Params &ep1, Operand A2,
                            Operand B2, GemmShape s2, const typename Epi2::Params &ep2, hipStream_t stream) {
  const int64_t b1 = static_cast<int64_t>(cdiv(s1.M, Cfg::BM)) * cdiv(s1.N, Cfg::BN);
  const int64_t b2 = static_cast<int64_t>(cdiv(s2.M, Cfg::BM)) * cdiv(s2.N, Cfg::BN);
  constexpr int BK = 8 * Elem<T>::CH;
  if (s1.kchunk != 0) return hipErrorInvalidValue;
  if (b1 <= 0) return launch_gemm<T, AK2, BKM2, Epi2, Cfg>(A2, B2, s2, ep2, stream);
  if (b2 <= 0) return launch_gemm<T, AK1, BKM1, Epi1, Cfg>(A1, B1, s1, ep1, stream);
  if (!gemm_shape_ok<T, AK1, BKM1>(A1, B1, s1) || !gemm_shape_ok<T, AK2, BKM2>(A2, B2, s2))
    return hipErrorInvalidValue;
  int64_t splits2 = 1;
  if (s2.kchunk > 0) {
    if (s2.kchunk % BK != 0) return hipErrorInvalidValue;
    splits2 = cdiv(s2.K, s2.kchunk);
  }
  const int64_t base2 = (b1 + kNumXcd - 1) / kNumXcd * kNumXcd;
  if constexpr (EpiPersistent<Epi1>::value && EpiPersistent<Epi2>::value && std::is_same<T, bf16_t>::value) {
    if (base2 + b2 * splits2 > 2 * kLoopBlocks) {
      hipLaunchKernelGGL((gemm_pair_persistent_kernel<T, AK1, BKM1, Epi1, AK2, BKM2, Epi2, Cfg>), dim3(kLoopBlocks),
                         dim3(Cfg::THREADS), 0, stream, A1, B1, s1, ep1, A2, B2, s2, ep2, static_cast<int>(b1),
                         static_cast<int>(base2), static_cast<int>(base2 + b2 * splits2));
      return hipGetLastError();
    }
  }
  hipLaunchKernelGGL((gemm_pair_kernel<T, AK1, BKM1, Epi1, AK2, BKM2, Epi2, Cfg>),
                     dim3(static_cast<unsigned>(base2 + b2 * splits2)), dim3(Cfg::THREADS), 0, stream, A1, B1, s1, ep1, A2,
                     B2, s2, ep2, static_cast<int>(b1), static_cast<int>(base2));
  return hipGetLastError();
}

}  // namespace ee
