// GEMMs of the block and the LM head.
//
// bfloat16: v_mfma_f32_32x32x16_bf16 tiles, float32 accumulation, LDS
// double-buffered, 256x256x64 workgroup tiles on 8 waves (128x64 per wave).
// Operands are copied into LDS in their memory order: a K-major one as
// [row][k], an M/N-major one (the weight-gradient GEMMs read activations
// [tokens, features]) as [k][row], whose MFMA fragments come out of LDS
// already transposed through ds_read_tr16_b64.  Workgroup ids are
// remapped so that each XCD (ids are dealt round-robin over the 8 XCDs) walks
// a contiguous, row-grouped run of tiles and its L2 sees the reuse.
//
// float32: a plain LDS-tiled FMA kernel (the float32 workload is the small
// correctness case).
#include "ops.h"

namespace aj {
namespace {

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

struct EpArgs {
  int M, N;
  void *C; int64_t ldc;
  int c_f32, accum;
  const void *R;
};

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

template <typename Cfg, bool A_K, bool B_K>
__global__ __launch_bounds__(Cfg::NT, 1) void gemm_mfma_kernel(
    int M, int N, int K, int k_per_split, const bf16_t *A, int64_t lda, const bf16_t *B,
    int64_t ldb, EpArgs ep, float *partial) {
  constexpr int BM = Cfg::BM, BN = Cfg::BN, BK = Cfg::BK, NT = Cfg::NT;
  using SA = Stager<BM, BK, NT, A_K>;
  using SB = Stager<BN, BK, NT, B_K>;
  __shared__ __attribute__((aligned(16))) uint16_t As[2][SA::kBytes / 2];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[2][SB::kBytes / 2];

  const int tiles_m = (M + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
  const TileIdx ti = tile_of(blockIdx.x, gridDim.x, tiles_m, tiles_n);
  const int m0 = ti.tm * BM, n0 = ti.tn * BN;
  const int kbeg = blockIdx.z * k_per_split;
  const int kend = min(K, kbeg + k_per_split);
  const int nk = kend > kbeg ? (kend - kbeg + BK - 1) / BK : 0;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / Cfg::WN, wn = wave % Cfg::WN;

  f32x16_t acc[Cfg::TM][Cfg::TN];
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
    sa.store(As[0]);
    sb.store(Bs[0]);
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
      for (int i = 0; i < Cfg::TM; ++i) af[i] = sa.frag(As[buf], wm * Cfg::WTM + i * 32, kk);
#pragma unroll
      for (int j = 0; j < Cfg::TN; ++j) bfr[j] = sb.frag(Bs[buf], wn * Cfg::WTN + j * 32, kk);
#pragma unroll
      for (int i = 0; i < Cfg::TM; ++i)
#pragma unroll
        for (int j = 0; j < Cfg::TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    // the other buffer was last read before the previous barrier; the loads
    // for it had the whole step to arrive
    if (kt + 1 < nk) {
      sa.store(As[buf ^ 1]);
      sb.store(Bs[buf ^ 1]);
    }
    __syncthreads();
  }

  // epilogue: lane holds column (lane & 31); register r holds row 8*(r/4) + 4*(lane/32) + r%4
#pragma unroll
  for (int i = 0; i < Cfg::TM; ++i)
#pragma unroll
    for (int j = 0; j < Cfg::TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + wm * Cfg::WTM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        const int n = n0 + wn * Cfg::WTN + j * 32 + (lane & 31);
        if (m >= M || n >= N) continue;
        const float v = acc[i][j][r];
        if (partial) {
          partial[((int64_t)blockIdx.z * M + m) * N + n] = v;
        } else if (ep.accum) {
          float *c = (float *)ep.C + (int64_t)m * ep.ldc + n;
          *c += v;
        } else if (ep.c_f32) {
          float *c = (float *)ep.C + (int64_t)m * ep.ldc + n;
          *c = v + (ep.R ? ((const float *)ep.R)[(int64_t)m * ep.ldc + n] : 0.f);
        } else {
          bf16_t *c = (bf16_t *)ep.C + (int64_t)m * ep.ldc + n;
          *c = f2bf(v + (ep.R ? bf2f(((const bf16_t *)ep.R)[(int64_t)m * ep.ldc + n]) : 0.f));
        }
      }
}

// ---------------------------------------------------------------- float32 / fallback
template <typename T>
__global__ __launch_bounds__(256) void gemm_simple_kernel(int M, int N, int K, int k_per_split,
                                                          const T *A, int64_t lda, int a_k,
                                                          const T *B, int64_t ldb, int b_k,
                                                          EpArgs ep, float *partial) {
  constexpr int BM = 64, BN = 64, BK = 16;
  __shared__ float As[BK][BM + 1];
  __shared__ float Bs[BK][BN + 1];
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int tx = threadIdx.x % 16, ty = threadIdx.x / 16;
  const int kbeg = blockIdx.z * k_per_split, kend = min(K, kbeg + k_per_split);
  float acc[4][4] = {};
  for (int k0 = kbeg; k0 < kend; k0 += BK) {
    for (int e = threadIdx.x; e < BM * BK; e += 256) {
      int mm = e % BM, kk = e / BM;
      int m = m0 + mm, k = k0 + kk;
      float va = 0.f, vb = 0.f;
      if (m < M && k < kend) va = ldf(A + (a_k ? (int64_t)m * lda + k : (int64_t)k * lda + m));
      int n = n0 + mm;
      if (n < N && k < kend) vb = ldf(B + (b_k ? (int64_t)n * ldb + k : (int64_t)k * ldb + n));
      As[kk][mm] = va;
      Bs[kk][mm] = vb;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < BK; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) { a[i] = As[kk][ty + 16 * i]; b[i] = Bs[kk][tx + 16 * i]; }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] += a[i] * b[j];
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int m = m0 + ty + 16 * i, n = n0 + tx + 16 * j;
      if (m >= M || n >= N) continue;
      const float v = acc[i][j];
      if (partial) {
        partial[((int64_t)blockIdx.z * M + m) * N + n] = v;
      } else if (ep.accum) {
        ((float *)ep.C)[(int64_t)m * ep.ldc + n] += v;
      } else if (ep.c_f32) {
        ((float *)ep.C)[(int64_t)m * ep.ldc + n] =
            v + (ep.R ? ((const float *)ep.R)[(int64_t)m * ep.ldc + n] : 0.f);
      } else {
        T *c = (T *)ep.C + (int64_t)m * ep.ldc + n;
        stf(c, v + (ep.R ? ldf((const T *)ep.R + (int64_t)m * ep.ldc + n) : 0.f));
      }
    }
}

using CfgBig = MfmaCfg<256, 256, 64, 2, 4>;

template <typename Cfg, bool A_K, bool B_K>
void launch_mfma(const Gemm &g, const EpArgs &ep, int kps, hipStream_t s) {
  const int tiles = ((g.M + Cfg::BM - 1) / Cfg::BM) * ((g.N + Cfg::BN - 1) / Cfg::BN);
  dim3 grid(tiles, 1, g.split_k);
  gemm_mfma_kernel<Cfg, A_K, B_K><<<grid, Cfg::NT, 0, s>>>(
      g.M, g.N, g.K, kps, (const bf16_t *)g.A, g.lda, (const bf16_t *)g.B, g.ldb, ep,
      g.split_k > 1 ? g.partial : nullptr);
}

bool aligned16(const void *p) { return ((uintptr_t)p & 15) == 0; }

}  // namespace

template <typename T>
int gemm(const Gemm &g, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return AJ_OK;
  if (g.split_k > 1 && !g.partial) return fail(AJ_ERR_WORKSPACE, "gemm: split-K without workspace");
  EpArgs ep{g.M, g.N, g.C, g.ldc, g.c_f32 ? 1 : 0, g.out == OUT_ACCUM_F32 ? 1 : 0, g.R};
  if (ep.accum) ep.c_f32 = 1;
  const int S = g.split_k > 1 ? g.split_k : 1;
  int kps = (g.K + S - 1) / S;
  kps = (kps + 63) / 64 * 64;
  if (g.K <= 0) {
    // empty reduction: C = R (or unchanged when accumulating)
    kps = 0;
  }
  bool mfma = false;
  if constexpr (sizeof(T) == 2) {
    // vector loads need the contiguous dimension in whole 8-element groups
    const int a_contig = g.a_kmajor ? g.K : g.M, b_contig = g.b_kmajor ? g.K : g.N;
    mfma = a_contig % 8 == 0 && b_contig % 8 == 0 && g.lda % 8 == 0 && g.ldb % 8 == 0 &&
           aligned16(g.A) && aligned16(g.B);
  }
  if (mfma) {
    const int kc = g.a_kmajor ? (g.b_kmajor ? AJ_KC_GEMM_NT : AJ_KC_GEMM_NN) : AJ_KC_GEMM_TN;
    const int tk = timing_begin(s, kc, g.recompute ? 0.0 : 2.0 * g.M * g.N * (double)g.K);
    if (g.a_kmajor && g.b_kmajor) launch_mfma<CfgBig, true, true>(g, ep, kps, s);
    else if (g.a_kmajor) launch_mfma<CfgBig, true, false>(g, ep, kps, s);
    else if (g.b_kmajor) launch_mfma<CfgBig, false, true>(g, ep, kps, s);
    else launch_mfma<CfgBig, false, false>(g, ep, kps, s);
    timing_end(s, tk);
  } else {
    dim3 grid((g.N + 63) / 64, (g.M + 63) / 64, S);
    gemm_simple_kernel<T><<<grid, 256, 0, s>>>(g.M, g.N, g.K, kps, (const T *)g.A, g.lda,
                                               g.a_kmajor, (const T *)g.B, g.ldb, g.b_kmajor, ep,
                                               S > 1 ? g.partial : nullptr);
  }
  int st = check_launch("gemm");
  if (st != AJ_OK) return st;
  if (S > 1) {
    // fixed-order sum of the split partials into C (float32)
    if (g.ldc != g.N) return fail(AJ_ERR_UNSUPPORTED, "gemm: split-K needs ldc == N");
    splitk_reduce(g.partial, S, (int64_t)g.M * g.N, (float *)g.C, ep.accum != 0, s);
    st = check_launch("gemm split-K reduce");
  }
  return st;
}

template int gemm<float>(const Gemm &, hipStream_t);
template int gemm<bf16_t>(const Gemm &, hipStream_t);

}  // namespace aj
