// The bfloat16 MFMA GEMM main loop, shared by the plain GEMM and the fused
// LM-head kernels (which only differ in what they do with the accumulators).
//
// Tiles of 256x256x64 on 8 waves (128x64 per wave, 4x2 v_mfma_f32_32x32x16_bf16
// tiles), LDS double-buffered.  Operands are copied into LDS in their memory
// order: a K-major one as [row][k], an M/N-major one as [k][row], whose MFMA
// fragments come out of LDS already transposed through ds_read_tr16_b64.
#pragma once
#include "common.h"

namespace aj {
namespace gemm_core {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

// Tile rows per group of the tile walk: the 32 tiles an XCD runs at once then
// cover 4 rows x 8 columns of tiles (12 operand panels shared through its L2;
// measured 1-3 % faster than 8 x 4 on the long-reduction layouts, 16 x 2 and
// 2 x 16 slower).
constexpr int kGroupM = 4;
constexpr int kXcds = 8;

struct TileIdx { int tm, tn; };

AJ_DEV TileIdx tile_of(int wg, int nwg, int tiles_m, int tiles_n) {
  const int per = nwg / kXcds, rem = nwg % kXcds;
  const int xcd = wg % kXcds, idx = wg / kXcds;
  const int t = xcd * per + (xcd < rem ? xcd : rem) + idx;
  // a skinny product runs whole tile rows (or columns) side by side, so that
  // each operand tile is fetched once for all the tiles that share it
  if (tiles_n <= 16) return {t / tiles_n, t % tiles_n};
  if (tiles_m <= 16) return {t % tiles_m, t / tiles_m};
  const int span = kGroupM * tiles_n;
  const int first_m = (t / span) * kGroupM;
  const int gm = min(tiles_m - first_m, kGroupM);
  const int r = t % span;
  return {first_m + r % gm, r / gm};
}


template <int BM_, int BN_, int BK_, int WM_, int WN_>
struct MfmaCfg {
  static constexpr int BM = BM_, BN = BN_, BK = BK_, WM = WM_, WN = WN_;
  static constexpr int NT = WM * WN * 64;
  static constexpr int WTM = BM / WM, WTN = BN / WN;
  static constexpr int TM = WTM / 32, TN = WTN / 32;
  static_assert(WTM % 32 == 0 && WTN % 32 == 0 && BK % 16 == 0, "tile shape");
};

// One operand tile of 256 rows (M or N) x 64 k, bfloat16, in LDS (32 KB), filled
// by asynchronous direct-to-LDS global loads: a wave instruction moves 64 x 16
// bytes and lane l's 16 bytes land at dst + 16*l, so the layout is chosen
// through each lane's global address.  16-byte chunks are XOR-swizzled so that
// the MFMA fragment reads hit all 64 banks:
//   K-major operand (rows r, k contiguous): [256][64], chunk c of row r at
//     r*128 + 16*(c ^ ((r >> 1) & 7))       (ds_read_b128 fragments)
//   M/N-major operand (k rows, r contiguous): [64][256], chunk c of k row k at
//     k*512 + 16*(c ^ (4 * (k & 3)))         (ds_read_tr16_b64 fragments)
// Rows past the operand's end read row `rows - 1` (their products land in
// output rows / columns that are never stored); k past K reads zeros.
__device__ __attribute__((aligned(16))) const uint32_t kZero16[4] = {0, 0, 0, 0};

AJ_DEV uint32_t lds_addr(const void *p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void *)p;
}

template <int NT, bool KMAJOR>
struct Tile {
  static constexpr int R = 256, BK = 64;
  static constexpr int kHalfs = R * BK;              // bf16 elements per stage
  static constexpr int kInstr = R * BK * 2 / 1024 / (NT / 64);   // wave instructions per stage

  AJ_DEV static void load(uint16_t *lds, const bf16_t *X, int64_t ld, int r0, int rows, int k0,
                          int K) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int q = 0; q < kInstr; ++q) {
      const int blk = wave * kInstr + q;             // 1 KB block of the tile
      const void *src;
      if (KMAJOR) {
        const int r = blk * 8 + (lane >> 3);
        const int c = (lane & 7) ^ ((r >> 1) & 7);
        const int k = k0 + 8 * c;
        const int rr = min(r0 + r, rows - 1);
        src = k < K ? (const void *)(X + (int64_t)rr * ld + k) : (const void *)kZero16;
      } else {
        const int kr = blk * 2 + (lane >> 5);
        const int c = (lane & 31) ^ (4 * (kr & 3));
        const int k = k0 + kr;
        const int rr = min(r0 + 8 * c, rows - 8);
        src = k < K ? (const void *)(X + (int64_t)k * ld + rr) : (const void *)kZero16;
      }
      __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void *)(lds + blk * 512),
                                       16, 0, 0);
    }
  }

  // MFMA 32x32x16 operand of rows [rb, rb+32), k [kk, kk+16): lane l gets row
  // rb + l%32 and k = kk + 8*(l/32) + 0..7.  The reads are issued as inline
  // assembly: the compiler cannot tell them apart from the LDS writes of the
  // in-flight direct-to-LDS copies and would otherwise wait for those copies
  // before every read; the caller waits for the reads itself (frag_wait).
  AJ_DEV static bf16x8_t frag(const uint16_t *lds, int rb, int kk) {
    const int lane = threadIdx.x & 63;
    bf16x8_t v;
    if (KMAJOR) {
      const int m = rb + (lane & 31);
      const int c = (kk >> 3) + (lane >> 5);
      const uint32_t a = lds_addr(lds + m * 64 + 8 * (c ^ ((m >> 1) & 7)));
      asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(a) : "memory");
      return v;
    }
    // ds_read_b64_tr_b16: in each 16-lane group, lane j receives element j%4
    // of the 4-element run addressed by lane 4e + j/4 (e = 0..3).  Source lane
    // s points at k row k0 + s/4, columns mb + 4*(s%4)..+3, so lane j
    // receives row mb + j at k0..k0+3; a second read gives k0+4..k0+7.
    const int g = lane >> 4, s = lane & 15;
    const int k = kk + 8 * (g >> 1) + (s >> 2);
    const int col = rb + 16 * (g & 1) + 4 * (s & 3);
    const int c = (col >> 3) ^ (4 * (k & 3));          // (k + 4) & 3 == k & 3
    const uint32_t a = lds_addr(lds + k * 256 + 8 * c + (col & 7));
    u32x2_t lo, hi;
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(lo) : "v"(a) : "memory");
    asm volatile("ds_read_b64_tr_b16 %0, %1 offset:2048" : "=v"(hi) : "v"(a) : "memory");
    return __builtin_bit_cast(bf16x8_t, u32x4_t{lo[0], lo[1], hi[0], hi[1]});
  }
};

// Waits for every LDS read in flight; the fragments pass through empty
// statements after the wait so that no MFMA consuming them is scheduled
// above it.
template <int TM, int TN>
AJ_DEV void frag_wait(bf16x8_t (&a)[TM], bf16x8_t (&b)[TN]) {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
  for (int i = 0; i < TM; ++i) asm volatile("" : "+v"(a[i]));
#pragma unroll
  for (int j = 0; j < TN; ++j) asm volatile("" : "+v"(b[j]));
}

// The plain GEMM: 8 waves as 2 x 4, each 128 rows x 64 columns.
using Cfg = MfmaCfg<256, 256, 64, 2, 4>;
// The LM-head kernels: 8 waves as 4 x 2, each 64 rows x 128 columns, so that a
// lane holds 4 columns of each of its rows for the per-row epilogue reductions.
using CfgWide = MfmaCfg<256, 256, 64, 4, 2>;

template <bool A_K, bool B_K, typename C = Cfg>
struct Smem {
  uint16_t a[2][256 * 64];
  uint16_t b[2][256 * 64];
};

AJ_DEV void wait_lds_dma() { __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// acc[i][j] (lane's share of the wave's block) = sum over k in [kbeg, kend)
// of A(m, k) B(n, k) for the 256x256 tile at (m0, n0) (added to acc instead
// when zero is false: a second reduction segment).  The next k-step's
// loads stream into the other LDS buffer while this one is consumed; the
// fragments of the next 16-wide k slice are read while the current one's
// MFMAs issue.
template <bool A_K, bool B_K, typename C = Cfg>
AJ_DEV void mainloop(f32x16_t (&acc)[C::TM][C::TN], const bf16_t *A, int64_t lda,
                     const bf16_t *B, int64_t ldb, int M, int N, int m0, int n0, int kbeg,
                     int kend, Smem<A_K, B_K, C> &sm, bool zero = true) {
  static_assert(C::BM == 256 && C::BN == 256 && C::BK == 64 && C::NT == 512, "tile");
  using TA = Tile<C::NT, A_K>;
  using TB = Tile<C::NT, B_K>;
  constexpr int BK = C::BK;
  const int nk = kend > kbeg ? (kend - kbeg + BK - 1) / BK : 0;
  const int wave = threadIdx.x >> 6;
  const int wm = wave / C::WN, wn = wave % C::WN;
  if (zero)
#pragma unroll
    for (int i = 0; i < C::TM; ++i)
#pragma unroll
      for (int j = 0; j < C::TN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  if (nk > 0) {
    TA::load(sm.a[0], A, lda, m0, M, kbeg, kend);
    TB::load(sm.b[0], B, ldb, n0, N, kbeg, kend);
  }
  wait_lds_dma();
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) {
      TA::load(sm.a[buf ^ 1], A, lda, m0, M, kbeg + (kt + 1) * BK, kend);
      TB::load(sm.b[buf ^ 1], B, ldb, n0, N, kbeg + (kt + 1) * BK, kend);
    }
    bf16x8_t af[2][C::TM], bfr[2][C::TN];
#pragma unroll
    for (int i = 0; i < C::TM; ++i) af[0][i] = TA::frag(sm.a[buf], wm * C::WTM + i * 32, 0);
#pragma unroll
    for (int j = 0; j < C::TN; ++j) bfr[0][j] = TB::frag(sm.b[buf], wn * C::WTN + j * 32, 0);
#pragma unroll
    for (int s = 0; s < BK / 16; ++s) {
      const int cur = s & 1;
      frag_wait(af[cur], bfr[cur]);
      if (s + 1 < BK / 16) {
#pragma unroll
        for (int i = 0; i < C::TM; ++i)
          af[cur ^ 1][i] = TA::frag(sm.a[buf], wm * C::WTM + i * 32, 16 * (s + 1));
#pragma unroll
        for (int j = 0; j < C::TN; ++j)
          bfr[cur ^ 1][j] = TB::frag(sm.b[buf], wn * C::WTN + j * 32, 16 * (s + 1));
      }
#pragma unroll
      for (int i = 0; i < C::TM; ++i)
#pragma unroll
        for (int j = 0; j < C::TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[cur][i], bfr[cur][j], acc[i][j],
                                                              0, 0, 0);
    }
    wait_lds_dma();
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Four waves, one per SIMD, as 2 x 2, each 128x128 (4x4 MFMA tiles, 256
// float32 accumulators per lane, held in AGPRs).  Against 8 waves of 128x64
// this halves the LDS fragment traffic per MFMA; with a single wave per SIMD
// nothing else hides latency, so the k loop (mainloop4s below) is issued in a
// fixed order.  Used for long reductions, where its heavier per-tile prologue
// and epilogue are amortised.
using Cfg4 = MfmaCfg<256, 256, 64, 2, 2>;

// Row / column of accumulator element r of tile (i, j) for this lane: the
// lane holds column lane%32 and rows 8*(r/4) + 4*(lane/32) + r%4 of each 32x32.
template <typename C = Cfg>
AJ_DEV int acc_row(int wm, int i, int r, int lane) {
  return wm * C::WTM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
}
template <typename C = Cfg>
AJ_DEV int acc_col(int wn, int j, int lane) { return wn * C::WTN + j * 32 + (lane & 31); }

// ---------------------------------------------------------------------------
// The 4-wave tile with 32-wide k-steps in four LDS stages (4 x 2 x 16 KB, the
// same 128 KB): the copies of a k-step are issued three k-steps before its
// products, and the end of a k-step waits only for the copies of the next
// one (the vector-memory counter lets the two younger steps' copies stay in
// flight), so a copy has three k-steps of matrix work to land instead of one.
// Layouts as above with 32 k: a K-major row is 64 bytes (4 chunks), chunk c
// of row r at r*64 + 16*(c ^ ((r >> 2) & 3)) -- the 16 rows of one read pass
// hit each of the 64 banks once; an M/N-major operand keeps [k][256] rows.
template <bool KMAJOR, int NW = 4>
struct Tile32 {
  static constexpr int BK = 32;
  static constexpr int kHalfs = 256 * BK;
  static constexpr int kInstr = 256 * BK * 2 / 1024 / NW;   // copies per wave (NW waves)

  AJ_DEV static int swz(int r) { return (r >> 2) & 3; }

  // bounded copy of the k-step at k0 (rows past the end repeat the last row,
  // k past K reads zeros)
  AJ_DEV static void load(uint16_t *lds, const bf16_t *X, int64_t ld, int r0, int rows, int k0,
                          int K) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int q = 0; q < kInstr; ++q) {
      const int blk = wave * kInstr + q;
      const void *src;
      if (KMAJOR) {
        const int r = blk * 16 + (lane >> 2);
        const int c = (lane & 3) ^ swz(r);
        const int k = k0 + 8 * c;
        const int rr = min(r0 + r, rows - 1);
        src = k < K ? (const void *)(X + (int64_t)rr * ld + k) : (const void *)kZero16;
      } else {
        const int kr = blk * 2 + (lane >> 5);
        const int c = (lane & 31) ^ (4 * (kr & 3));
        const int k = k0 + kr;
        const int rr = min(r0 + 8 * c, rows - 8);
        src = k < K ? (const void *)(X + (int64_t)k * ld + rr) : (const void *)kZero16;
      }
      __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void *)(lds + blk * 512),
                                       16, 0, 0);
    }
  }

  // MFMA operand of rows [rb, rb+32), k [kk, kk+16), as Tile::frag
  AJ_DEV static bf16x8_t frag(const uint16_t *lds, int rb, int kk) {
    const int lane = threadIdx.x & 63;
    bf16x8_t v;
    if (KMAJOR) {
      const int m = rb + (lane & 31);
      const int c = (kk >> 3) + (lane >> 5);
      const uint32_t a = lds_addr(lds + m * 32 + 8 * (c ^ swz(m)));
      asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(a) : "memory");
      return v;
    }
    const int g = lane >> 4, s = lane & 15;
    const int k = kk + 8 * (g >> 1) + (s >> 2);
    const int col = rb + 16 * (g & 1) + 4 * (s & 3);
    const int c = (col >> 3) ^ (4 * (k & 3));
    const uint32_t a = lds_addr(lds + k * 256 + 8 * c + (col & 7));
    u32x2_t lo, hi;
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(lo) : "v"(a) : "memory");
    asm volatile("ds_read_b64_tr_b16 %0, %1 offset:2048" : "=v"(hi) : "v"(a) : "memory");
    return __builtin_bit_cast(bf16x8_t, u32x4_t{lo[0], lo[1], hi[0], hi[1]});
  }
};

// Loop-invariant per-lane offsets of the copies of a whole 32-wide k-step.
template <bool KMAJOR, int NW = 4>
struct Copier32 {
  static constexpr int kInstr = Tile32<KMAJOR, NW>::kInstr;
  uint32_t off[kInstr];
  int64_t step;

  AJ_DEV void init(int64_t ld, int r0, int rows) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int q = 0; q < kInstr; ++q) {
      const int blk = wave * kInstr + q;
      if (KMAJOR) {
        const int r = blk * 16 + (lane >> 2);
        const int c = (lane & 3) ^ Tile32<true>::swz(r);
        const int rr = min(r0 + r, rows - 1) - r0;
        off[q] = (uint32_t)(((int64_t)rr * ld + 8 * c) * 2);
      } else {
        const int kr = blk * 2 + (lane >> 5);
        const int c = (lane & 31) ^ (4 * (kr & 3));
        const int rr = min(r0 + 8 * c, rows - 8) - r0;
        off[q] = (uint32_t)(((int64_t)kr * ld + rr) * 2);
      }
    }
    step = KMAJOR ? 32 : 32 * ld;
  }
  AJ_DEV void issue_one(int q, uint16_t *lds, const bf16_t *tile) const {
    const int wave = threadIdx.x >> 6;
    __builtin_amdgcn_global_load_lds(
        reinterpret_cast<const char *>(tile) + off[q],
        (__attribute__((address_space(3))) void *)(lds + (wave * kInstr + q) * 512), 16, 0, 0);
  }
};

// S stages of a 32-wide k-step (16 KB per operand each): four fill the
// common 128 KB, five the whole 160 KB of a gfx950 CU.
template <bool A_K, bool B_K, int S = 4>
struct Smem4s {
  static constexpr int kStages = S;
  uint16_t a[S][256 * 32];
  uint16_t b[S][256 * 32];
};

// A workgroup barrier without the memory fence of __syncthreads: that fence
// waits for every outstanding vector-memory operation, the direct-to-LDS
// copies still meant to fly included.  Visibility of the copies and reads that
// must be complete is ensured by explicit vmcnt / lgkmcnt waits before it; the
// empty asm statements keep the compiler from moving memory operations across.
AJ_DEV void bar_nofence() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Waits until at most n k-steps' copies (PER per wave each, n <= 3) are
// still in flight.
template <int PER>
AJ_DEV void wait_steps(int n) {
  static_assert(PER == 4 || PER == 8, "copies per wave and k-step");
  switch (n * PER) {
    case 24: __asm__ volatile("s_waitcnt vmcnt(24)" ::: "memory"); break;
    case 16: __asm__ volatile("s_waitcnt vmcnt(16)" ::: "memory"); break;
    case 12: __asm__ volatile("s_waitcnt vmcnt(12)" ::: "memory"); break;
    case 8: __asm__ volatile("s_waitcnt vmcnt(8)" ::: "memory"); break;
    case 4: __asm__ volatile("s_waitcnt vmcnt(4)" ::: "memory"); break;
    default: __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory"); break;
  }
}
AJ_DEV void wait_copies(int n) { wait_steps<8>(n); }

// Fragment reads of one 16-wide slice, issued one after each of the last 8
// MFMAs of the slice before, in the order B0 A0 B1 B2 B3 A1 A2 A3, so that
// each MFMA of the slice waits only for the reads it consumes (the MFMAs run
// A-major: t uses A[t/4], B[t%4]).  LDS reads complete in order, so the wait
// before MFMA t is "at most n reads in flight" with n the LDS instructions
// issued after the last one it needs (an M/N-major fragment is two reads).
template <bool A_K, bool B_K>
struct ReadPlan {
  static constexpr int nA = A_K ? 1 : 2, nB = B_K ? 1 : 2;
  static constexpr int kTotal = 4 * nA + 4 * nB;
  AJ_DEV static constexpr bool is_b(int q) { return q == 0 || (q >= 2 && q <= 4); }
  AJ_DEV static constexpr int index(int q) { return q <= 1 ? 0 : q <= 4 ? q - 1 : q - 4; }
  // LDS instructions issued by reads 0..q-1
  AJ_DEV static constexpr int issued(int q) {
    int n = 0;
    for (int i = 0; i < q; ++i) n += is_b(i) ? nB : nA;
    return n;
  }
  // LDS instructions allowed in flight before MFMA t (-1: no wait): the
  // slice's own reads after the last one MFMA t needs, plus the next slice's
  // reads already issued (one after each MFMA from the 8th on) when kRead
  AJ_DEV static constexpr int wait_before(int t, bool kRead) {
    const int last = t == 0 ? 1 : t <= 3 ? t + 1 : t == 4 ? 5 : t == 8 ? 6 : t == 12 ? 7 : -1;
    if (last < 0) return -1;
    const int next = kRead && t > 8 ? issued(t - 8) : 0;
    return kTotal - issued(last + 1) + next;
  }
};

AJ_DEV void lgkm_wait(int n) {
  switch (n) {
    case 0: asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); break;
    case 1: asm volatile("s_waitcnt lgkmcnt(1)" ::: "memory"); break;
    case 2: asm volatile("s_waitcnt lgkmcnt(2)" ::: "memory"); break;
    case 3: asm volatile("s_waitcnt lgkmcnt(3)" ::: "memory"); break;
    case 4: asm volatile("s_waitcnt lgkmcnt(4)" ::: "memory"); break;
    case 5: asm volatile("s_waitcnt lgkmcnt(5)" ::: "memory"); break;
    case 6: asm volatile("s_waitcnt lgkmcnt(6)" ::: "memory"); break;
    case 7: asm volatile("s_waitcnt lgkmcnt(7)" ::: "memory"); break;
    case 8: asm volatile("s_waitcnt lgkmcnt(8)" ::: "memory"); break;
    case 9: asm volatile("s_waitcnt lgkmcnt(9)" ::: "memory"); break;
    case 10: asm volatile("s_waitcnt lgkmcnt(10)" ::: "memory"); break;
    case 11: asm volatile("s_waitcnt lgkmcnt(11)" ::: "memory"); break;
    case 12: asm volatile("s_waitcnt lgkmcnt(12)" ::: "memory"); break;
    case 13: asm volatile("s_waitcnt lgkmcnt(13)" ::: "memory"); break;
    case 14: asm volatile("s_waitcnt lgkmcnt(14)" ::: "memory"); break;
    default: break;
  }
}

// read number q (0..7) of a slice's fragments, in ReadPlan order
template <bool A_K, bool B_K>
AJ_DEV void read_frag4s(int q, bf16x8_t (&na)[4], bf16x8_t (&nb)[4], const uint16_t *as,
                        const uint16_t *bs, int wm, int wn, int kk) {
  using P = ReadPlan<A_K, B_K>;
  const int i = P::index(q);
  if (P::is_b(q)) nb[i] = Tile32<B_K>::frag(bs, wn * 128 + i * 32, kk);
  else na[i] = Tile32<A_K>::frag(as, wm * 128 + i * 32, kk);
}

// One 16-wide k slice of the staged loop: 16 MFMAs in a fixed order, each
// after the partial wait for its fragments, a whole k-step's 8 copies after
// the first 8, the next slice's 8 fragment reads after the last 8.  With kBar
// the k-step's closing wait and barrier sit after the first 8 MFMAs (this
// wave's reads of the current stage are all complete by then), so that the
// reads of the next k-step's first slice, from as / bs, overlap the last 8.
template <bool A_K, bool B_K, bool kCopy, bool kRead, bool kBar = false, int kYoung = 2>
AJ_DEV void slice4s(f32x16_t (&acc)[4][4], bf16x8_t (&fa)[4], bf16x8_t (&fb)[4],
                    bf16x8_t (&na)[4], bf16x8_t (&nb)[4], const uint16_t *as, const uint16_t *bs,
                    int wm, int wn, int kk_next, const Copier32<A_K> &ca,
                    const Copier32<B_K> &cb, uint16_t *la, uint16_t *lb, const bf16_t *ta,
                    const bf16_t *tb) {
  using P = ReadPlan<A_K, B_K>;
#pragma unroll
  for (int t = 0; t < 16; ++t) {
    const int a = t >> 2, b = t & 3;
    if (P::wait_before(t, kRead) >= 0) {
      lgkm_wait(P::wait_before(t, kRead));
      // the MFMA's operands pass through the wait so that it stays below it
      asm volatile("" : "+v"(fa[a]));
      asm volatile("" : "+v"(fb[b]));
    }
    acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[a], fb[b], acc[a][b], 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
    if (kCopy && t < 8) {
      if (t < Copier32<A_K>::kInstr) ca.issue_one(t, la, ta);
      else cb.issue_one(t - Copier32<A_K>::kInstr, lb, tb);
    }
    if (kBar && t == 7) {
      // the next k-step's copies have landed (those of the kYoung after it may fly)
      wait_copies(kYoung);
      bar_nofence();
    }
    if (kRead && t >= 8) read_frag4s<A_K, B_K>(t - 8, na, nb, as, bs, wm, wn, kk_next);
    __builtin_amdgcn_sched_barrier(0);
  }
}

template <bool A_K, bool B_K, int S>
AJ_DEV void mainloop4s(f32x16_t (&acc)[4][4], const bf16_t *A, int64_t lda, const bf16_t *B,
                       int64_t ldb, int M, int N, int m0, int n0, int kbeg, int kend,
                       Smem4s<A_K, B_K, S> &sm) {
  using TA = Tile32<A_K>;
  using TB = Tile32<B_K>;
  static_assert(Copier32<A_K>::kInstr + Copier32<B_K>::kInstr == 8, "copies per k-step");
  static_assert(S == 4 || S == 5, "stages");
  constexpr int BK = 32, AHEAD = S - 1;   // copies run AHEAD k-steps before their products
  const int nk = kend > kbeg ? (kend - kbeg + BK - 1) / BK : 0;
  const int nfull = kend > kbeg ? (kend - kbeg) / BK : 0;
  const int wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  if (nk == 0) return;
  Copier32<A_K> ca;
  Copier32<B_K> cb;
  ca.init(lda, m0, M);
  cb.init(ldb, n0, N);
  const bf16_t *ta = A + (A_K ? (int64_t)m0 * lda + kbeg : (int64_t)kbeg * lda + m0);
  const bf16_t *tb = B + (B_K ? (int64_t)n0 * ldb + kbeg : (int64_t)kbeg * ldb + n0);
  // all 8 copies of k-step kt (< nk) into its stage
  auto copy_step = [&](int kt) {
    const int st = kt % S;
    if (kt < nfull) {
#pragma unroll
      for (int q = 0; q < Copier32<A_K>::kInstr; ++q) ca.issue_one(q, sm.a[st], ta + kt * ca.step);
#pragma unroll
      for (int q = 0; q < Copier32<B_K>::kInstr; ++q) cb.issue_one(q, sm.b[st], tb + kt * cb.step);
    } else {
      TA::load(sm.a[st], A, lda, m0, M, kbeg + kt * BK, kend);
      TB::load(sm.b[st], B, ldb, n0, N, kbeg + kt * BK, kend);
    }
  };
  bf16x8_t f0a[4], f0b[4], f1a[4], f1b[4];
  const int pro = nk < AHEAD ? nk : AHEAD;
  for (int kt = 0; kt < pro; ++kt) copy_step(kt);
  wait_copies(pro - 1);
  bar_nofence();
  auto read_first = [&](int st) {
#pragma unroll
    for (int q = 0; q < 8; ++q) read_frag4s<A_K, B_K>(q, f0a, f0b, sm.a[st], sm.b[st], wm, wn, 0);
  };
  read_first(0);
  int kt = 0, st = 0;   // st = kt % S
  // steady state: the k-step AHEAD on is a full one, copied in the first slice
  for (; kt + AHEAD < nfull; ++kt) {
    const int nx = st == 0 ? S - 1 : st - 1;   // (kt + AHEAD) % S
    const int s1 = st == S - 1 ? 0 : st + 1;
    const uint16_t *as = sm.a[st], *bs = sm.b[st];
    slice4s<A_K, B_K, true, true>(acc, f0a, f0b, f1a, f1b, as, bs, wm, wn, 16, ca, cb, sm.a[nx],
                                  sm.b[nx], ta + (kt + AHEAD) * ca.step,
                                  tb + (kt + AHEAD) * cb.step);
    slice4s<A_K, B_K, false, true, true, AHEAD - 1>(acc, f1a, f1b, f0a, f0b, sm.a[s1], sm.b[s1],
                                                    wm, wn, 0, ca, cb, nullptr, nullptr, nullptr,
                                                    nullptr);
    st = s1;
  }
  // the last AHEAD k-steps (the last may be ragged, its copies bounded)
  for (; kt < nk; ++kt) {
    const uint16_t *as = sm.a[st], *bs = sm.b[st];
    if (kt + AHEAD < nk) copy_step(kt + AHEAD);
    slice4s<A_K, B_K, false, true>(acc, f0a, f0b, f1a, f1b, as, bs, wm, wn, 16, ca, cb, nullptr,
                                   nullptr, nullptr, nullptr);
    slice4s<A_K, B_K, false, false>(acc, f1a, f1b, f0a, f0b, as, bs, wm, wn, 0, ca, cb, nullptr,
                                    nullptr, nullptr, nullptr);
    // k-step kt+1 must have landed; those after it (up to kt+AHEAD) may fly
    const int last = kt + AHEAD < nk - 1 ? kt + AHEAD : nk - 1;
    wait_copies(last > kt + 1 ? last - kt - 1 : 0);
    bar_nofence();
    st = st == S - 1 ? 0 : st + 1;
    if (kt + 1 < nk) read_first(st);
  }
}

// ---------------------------------------------------------------------------
// The 8-wave tiles (Cfg, CfgWide) on the same staged k loop: 32-wide k-steps
// through four LDS stages, copies three k-steps ahead, one fence-free barrier
// per k-step.  A wave holds TM x TN = 8 MFMA tiles, so a slice is 8 MFMAs: the
// k-step's 4 copies per wave follow the first 4 MFMAs of its first slice, the
// closing wait and barrier the 4th MFMA of its second, and the next slice's
// TM + TN fragment reads are spread over the last 4 (two waves per SIMD cover
// each other's waits, so the slices wait for their fragments as a whole).
AJ_DEV void wait_copies8(int n) { wait_steps<4>(n); }   // 4 copies per wave per k-step

template <bool A_K, bool B_K, typename C>
AJ_DEV void read_frag8s(int q, bf16x8_t (&na)[C::TM], bf16x8_t (&nb)[C::TN], const uint16_t *as,
                        const uint16_t *bs, int wm, int wn, int kk) {
  if (q < C::TM) na[q] = Tile32<A_K, 8>::frag(as, wm * C::WTM + q * 32, kk);
  else nb[q - C::TM] = Tile32<B_K, 8>::frag(bs, wn * C::WTN + (q - C::TM) * 32, kk);
}

template <bool A_K, bool B_K, typename C, bool kCopy, bool kRead, bool kBar = false,
          int kYoung = 2>
AJ_DEV void slice8s(f32x16_t (&acc)[C::TM][C::TN], const bf16x8_t (&fa)[C::TM],
                    const bf16x8_t (&fb)[C::TN], bf16x8_t (&na)[C::TM], bf16x8_t (&nb)[C::TN],
                    const uint16_t *as, const uint16_t *bs, int wm, int wn, int kk_next,
                    const Copier32<A_K, 8> &ca, const Copier32<B_K, 8> &cb, uint16_t *la,
                    uint16_t *lb, const bf16_t *ta, const bf16_t *tb) {
  constexpr int R = C::TM + C::TN;
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    const int i = t / C::TN, j = t % C::TN;
    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
    if (kCopy && t < 4) {
      if (t < Copier32<A_K, 8>::kInstr) ca.issue_one(t, la, ta);
      else cb.issue_one(t - Copier32<A_K, 8>::kInstr, lb, tb);
    }
    if (kBar && t == 3) {
      wait_copies8(kYoung);
      bar_nofence();
    }
    if (kRead && t >= 4) {
#pragma unroll
      for (int q = (t - 4) * R / 4; q < (t - 3) * R / 4; ++q)
        read_frag8s<A_K, B_K, C>(q, na, nb, as, bs, wm, wn, kk_next);
    }
    __builtin_amdgcn_sched_barrier(0);
  }
}

template <bool A_K, bool B_K, typename C, int S>
AJ_DEV void mainloop8s(f32x16_t (&acc)[C::TM][C::TN], const bf16_t *A, int64_t lda,
                       const bf16_t *B, int64_t ldb, int M, int N, int m0, int n0, int kbeg,
                       int kend, Smem4s<A_K, B_K, S> &sm) {
  static_assert(C::NT == 512 && C::TM * C::TN == 8, "8 waves of 8 MFMA tiles");
  static_assert(S == 4 || S == 5, "stages");
  using TA = Tile32<A_K, 8>;
  using TB = Tile32<B_K, 8>;
  using CA = Copier32<A_K, 8>;
  using CB = Copier32<B_K, 8>;
  static_assert(CA::kInstr + CB::kInstr == 4, "copies per k-step");
  constexpr int BK = 32, AHEAD = S - 1;
  const int nk = kend > kbeg ? (kend - kbeg + BK - 1) / BK : 0;
  const int nfull = kend > kbeg ? (kend - kbeg) / BK : 0;
  const int wave = threadIdx.x >> 6;
  const int wm = wave / C::WN, wn = wave % C::WN;
#pragma unroll
  for (int i = 0; i < C::TM; ++i)
#pragma unroll
    for (int j = 0; j < C::TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  if (nk == 0) return;
  CA ca;
  CB cb;
  ca.init(lda, m0, M);
  cb.init(ldb, n0, N);
  const bf16_t *ta = A + (A_K ? (int64_t)m0 * lda + kbeg : (int64_t)kbeg * lda + m0);
  const bf16_t *tb = B + (B_K ? (int64_t)n0 * ldb + kbeg : (int64_t)kbeg * ldb + n0);
  auto copy_step = [&](int kt) {
    const int st = kt % S;
    if (kt < nfull) {
#pragma unroll
      for (int q = 0; q < CA::kInstr; ++q) ca.issue_one(q, sm.a[st], ta + kt * ca.step);
#pragma unroll
      for (int q = 0; q < CB::kInstr; ++q) cb.issue_one(q, sm.b[st], tb + kt * cb.step);
    } else {
      TA::load(sm.a[st], A, lda, m0, M, kbeg + kt * BK, kend);
      TB::load(sm.b[st], B, ldb, n0, N, kbeg + kt * BK, kend);
    }
  };
  bf16x8_t f0a[C::TM], f0b[C::TN], f1a[C::TM], f1b[C::TN];
  auto read_first = [&](int st) {
#pragma unroll
    for (int q = 0; q < C::TM + C::TN; ++q)
      read_frag8s<A_K, B_K, C>(q, f0a, f0b, sm.a[st], sm.b[st], wm, wn, 0);
  };
  const int pro = nk < AHEAD ? nk : AHEAD;
  for (int kt = 0; kt < pro; ++kt) copy_step(kt);
  wait_copies8(pro - 1);
  bar_nofence();
  read_first(0);
  int kt = 0, st = 0;   // st = kt % S
  for (; kt + AHEAD < nfull; ++kt) {
    const int nx = st == 0 ? S - 1 : st - 1;   // (kt + AHEAD) % S
    const int s1 = st == S - 1 ? 0 : st + 1;
    const uint16_t *as = sm.a[st], *bs = sm.b[st];
    frag_wait(f0a, f0b);
    slice8s<A_K, B_K, C, true, true>(acc, f0a, f0b, f1a, f1b, as, bs, wm, wn, 16, ca, cb,
                                     sm.a[nx], sm.b[nx], ta + (kt + AHEAD) * ca.step,
                                     tb + (kt + AHEAD) * cb.step);
    frag_wait(f1a, f1b);
    slice8s<A_K, B_K, C, false, true, true, AHEAD - 1>(acc, f1a, f1b, f0a, f0b, sm.a[s1],
                                                       sm.b[s1], wm, wn, 0, ca, cb, nullptr,
                                                       nullptr, nullptr, nullptr);
    st = s1;
  }
  for (; kt < nk; ++kt) {
    const uint16_t *as = sm.a[st], *bs = sm.b[st];
    if (kt + AHEAD < nk) copy_step(kt + AHEAD);
    frag_wait(f0a, f0b);
    slice8s<A_K, B_K, C, false, true>(acc, f0a, f0b, f1a, f1b, as, bs, wm, wn, 16, ca, cb,
                                      nullptr, nullptr, nullptr, nullptr);
    frag_wait(f1a, f1b);
    slice8s<A_K, B_K, C, false, false>(acc, f1a, f1b, f0a, f0b, as, bs, wm, wn, 0, ca, cb,
                                       nullptr, nullptr, nullptr, nullptr);
    const int last = kt + AHEAD < nk - 1 ? kt + AHEAD : nk - 1;
    wait_copies8(last > kt + 1 ? last - kt - 1 : 0);
    bar_nofence();
    st = st == S - 1 ? 0 : st + 1;
    if (kt + 1 < nk) read_first(st);
  }
}

}  // namespace gemm_core
}  // namespace aj
