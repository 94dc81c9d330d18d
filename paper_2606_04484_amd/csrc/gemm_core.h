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

constexpr int kGroupM = 8;
constexpr int kXcds = 8;

struct TileIdx { int tm, tn; };

AJ_DEV TileIdx tile_of(int wg, int nwg, int tiles_m, int tiles_n) {
  const int per = nwg / kXcds, rem = nwg % kXcds;
  const int xcd = wg % kXcds, idx = wg / kXcds;
  const int t = xcd * per + (xcd < rem ? xcd : rem) + idx;
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

// Stages one operand tile through registers into LDS.
//   K-major operand (rows r, k contiguous): LDS [R][BK + 8], 16-byte vectors.
//   M/N-major operand (k rows, r contiguous): copied untransposed into LDS
//   [BK][R + 32]; the MFMA fragments are then read with ds_read_tr16_b64.
template <int R, int BK, int NT, bool KMAJOR>
struct Stager {
  static constexpr int LD = KMAJOR ? BK + 8 : R + 32;    // LDS row pitch (bf16 elements)
  static constexpr int kSlots = R * BK / 8;
  static constexpr int kPer = (kSlots + NT - 1) / NT;
  static constexpr int kBytes = (KMAJOR ? R * LD : BK * LD) * 2;
  u32x4_t v[kPer];

  AJ_DEV void load(const bf16_t *X, int64_t ld, int r0, int rows, int k0, int K) {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int slot = threadIdx.x + i * NT;
      int r, k;
      if (KMAJOR) { r = r0 + slot / (BK / 8); k = k0 + (slot % (BK / 8)) * 8; }
      else { k = k0 + slot / (R / 8); r = r0 + (slot % (R / 8)) * 8; }
      if (slot < kSlots && r < rows && k < K)
        v[i] = KMAJOR ? *(const u32x4_t *)(X + (int64_t)r * ld + k)
                      : *(const u32x4_t *)(X + (int64_t)k * ld + r);
      else
        v[i] = u32x4_t{0, 0, 0, 0};
    }
  }

  AJ_DEV void store(uint16_t *lds) const {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int slot = threadIdx.x + i * NT;
      if (slot >= kSlots) continue;
      if (KMAJOR) *(u32x4_t *)(lds + (slot / (BK / 8)) * LD + (slot % (BK / 8)) * 8) = v[i];
      else *(u32x4_t *)(lds + (slot / (R / 8)) * LD + (slot % (R / 8)) * 8) = v[i];
    }
  }

  // MFMA 32x32x16 operand of rows [rb, rb+32), k [kk, kk+16): lane l gets row
  // rb + l%32 and k = kk + 8*(l/32) + 0..7.
  AJ_DEV bf16x8_t frag(const uint16_t *lds, int rb, int kk) const {
    const int lane = threadIdx.x & 63;
    if (KMAJOR) return *(const bf16x8_t *)(lds + (rb + (lane & 31)) * LD + kk + (lane >> 5) * 8);
    // ds_read_tr16_b64: in each 16-lane group, lane j receives element j%4 of
    // the 4-element run addressed by lane 4e + j/4 (e = 0..3).  Source lane s
    // points at k row k0 + s/4, columns mb + 4*(s%4)..+3, so lane j receives
    // row mb + j at k0..k0+3.
    const int g = lane >> 4, s = lane & 15;
    const int mb = rb + 16 * (g & 1), k0 = kk + 8 * (g >> 1);
    const uint16_t *p = lds + (k0 + (s >> 2)) * LD + mb + 4 * (s & 3);
    typedef short v4i16 __attribute__((ext_vector_type(4)));
    typedef __attribute__((address_space(3))) v4i16 lds_v4i16;
    v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16 *)p);
    v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16 *)(p + 4 * LD));
    u32x2_t a = __builtin_bit_cast(u32x2_t, lo), b = __builtin_bit_cast(u32x2_t, hi);
    return __builtin_bit_cast(bf16x8_t, u32x4_t{a[0], a[1], b[0], b[1]});
  }
};


// The plain GEMM: 8 waves as 2 x 4, each 128 rows x 64 columns.
using Cfg = MfmaCfg<256, 256, 64, 2, 4>;
// The LM-head kernels: 8 waves as 4 x 2, each 64 rows x 128 columns, so that a
// lane holds 4 columns of each of its rows for the per-row epilogue reductions.
using CfgWide = MfmaCfg<256, 256, 64, 4, 2>;

template <bool A_K, bool B_K, typename C = Cfg>
struct Smem {
  using SA = Stager<C::BM, C::BK, C::NT, A_K>;
  using SB = Stager<C::BN, C::BK, C::NT, B_K>;
  uint16_t a[2][SA::kBytes / 2];
  uint16_t b[2][SB::kBytes / 2];
};

// acc[i][j] (lane's share of the wave's block) = sum over k in [kbeg, kend)
// of A(m, k) B(n, k) for the tile at (m0, n0).
template <bool A_K, bool B_K, typename C = Cfg>
AJ_DEV void mainloop(f32x16_t (&acc)[C::TM][C::TN], const bf16_t *A, int64_t lda,
                     const bf16_t *B, int64_t ldb, int M, int N, int m0, int n0, int kbeg,
                     int kend, Smem<A_K, B_K, C> &sm) {
  using Cfg = C;
  constexpr int BK = Cfg::BK;
  using SA = typename Smem<A_K, B_K, C>::SA;
  using SB = typename Smem<A_K, B_K, C>::SB;
  const int nk = kend > kbeg ? (kend - kbeg + BK - 1) / BK : 0;
  const int wave = threadIdx.x >> 6;
  const int wm = wave / Cfg::WN, wn = wave % Cfg::WN;
#pragma unroll
  for (int i = 0; i < Cfg::TM; ++i)
#pragma unroll
    for (int j = 0; j < Cfg::TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  SA sa;
  SB sb;
  if (nk > 0) {
    sa.load(A, lda, m0, M, kbeg, kend);
    sb.load(B, ldb, n0, N, kbeg, kend);
    sa.store(sm.a[0]);
    sb.store(sm.b[0]);
  }
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) {
      sa.load(A, lda, m0, M, kbeg + (kt + 1) * BK, kend);
      sb.load(B, ldb, n0, N, kbeg + (kt + 1) * BK, kend);
    }
#pragma unroll
    for (int kk = 0; kk < BK; kk += 16) {
      bf16x8_t af[Cfg::TM], bfr[Cfg::TN];
#pragma unroll
      for (int i = 0; i < Cfg::TM; ++i) af[i] = sa.frag(sm.a[buf], wm * Cfg::WTM + i * 32, kk);
#pragma unroll
      for (int j = 0; j < Cfg::TN; ++j) bfr[j] = sb.frag(sm.b[buf], wn * Cfg::WTN + j * 32, kk);
#pragma unroll
      for (int i = 0; i < Cfg::TM; ++i)
#pragma unroll
        for (int j = 0; j < Cfg::TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    // the other buffer was last read before the previous barrier; the loads
    // for it had the whole step to arrive
    if (kt + 1 < nk) {
      sa.store(sm.a[buf ^ 1]);
      sb.store(sm.b[buf ^ 1]);
    }
    __syncthreads();
  }
}

// Row / column of accumulator element r of tile (i, j) for this lane: the
// lane holds column lane%32 and rows 8*(r/4) + 4*(lane/32) + r%4 of each 32x32.
template <typename C = Cfg>
AJ_DEV int acc_row(int wm, int i, int r, int lane) {
  return wm * C::WTM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
}
template <typename C = Cfg>
AJ_DEV int acc_col(int wn, int j, int lane) { return wn * C::WTN + j * 32 + (lane & 31); }

}  // namespace gemm_core
}  // namespace aj
