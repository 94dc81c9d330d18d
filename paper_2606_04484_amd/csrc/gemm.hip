// GEMMs of the block and the LM head.
//
// bfloat16: v_mfma_f32_32x32x16_bf16 tiles, float32 accumulation, LDS
// double-buffered.  Both operands are kept in LDS as [row][k] (k contiguous):
// a K-major operand is copied as is, an M/N-major one (the weight-gradient
// GEMMs read activations [tokens, features]) is transposed in registers on
// its way from HBM to LDS, 4 k-rows x 8 columns per thread.  Workgroup ids are
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
  static constexpr int LDK = BK + 8;            // padded LDS row (bf16 elements)
  static_assert(WTM % 32 == 0 && WTN % 32 == 0 && BK % 16 == 0, "tile shape");
};

// Stages one operand tile (rows [r0, r0+R) of the operand, k in [k0, k0+BK))
// through registers into LDS laid out [R][LDK].
template <int R, int BK, int LDK, int NT, bool KMAJOR>
struct Stager {
  // K-major: 16-byte vectors of 8 k's; MN-major: 4 k-rows x 8 rows per slot,
  // k-blocks varying fastest across threads so that the transposed 8-byte LDS
  // stores of a wave spread over all banks (2 lanes per bank pair).
  static constexpr int kSlots = KMAJOR ? R * BK / 8 : (R / 8) * (BK / 4);
  static constexpr int kPer = (kSlots + NT - 1) / NT;
  static constexpr int kVec = KMAJOR ? 1 : 4;
  u32x4_t v[kPer][kVec];

  AJ_DEV void load(const bf16_t *X, int64_t ld, int r0, int rows, int k0, int K) {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int slot = threadIdx.x + i * NT;
      if (KMAJOR) {
        const int row = slot / (BK / 8), kv = slot % (BK / 8);
        const int r = r0 + row, k = k0 + kv * 8;
        if (slot < kSlots && r < rows && k < K)
          v[i][0] = *(const u32x4_t *)(X + (int64_t)r * ld + k);
        else
          v[i][0] = u32x4_t{0, 0, 0, 0};
      } else {
        const int kb = slot % (BK / 4), rb = slot / (BK / 4);
        const int r = r0 + rb * 8;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
          const int k = k0 + kb * 4 + kk;
          if (slot < kSlots && r < rows && k < K)
            v[i][kk] = *(const u32x4_t *)(X + (int64_t)k * ld + r);
          else
            v[i][kk] = u32x4_t{0, 0, 0, 0};
        }
      }
    }
  }

  AJ_DEV void store(uint16_t *lds) const {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int slot = threadIdx.x + i * NT;
      if (slot >= kSlots) continue;
      if (KMAJOR) {
        const int row = slot / (BK / 8), kv = slot % (BK / 8);
        *(u32x4_t *)(lds + row * LDK + kv * 8) = v[i][0];
      } else {
        const int kb = slot % (BK / 4), rb = slot / (BK / 4);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int w = e >> 1, sh = (e & 1) * 16;
          const uint32_t a0 = (v[i][0][w] >> sh) & 0xffffu, a1 = (v[i][1][w] >> sh) & 0xffffu;
          const uint32_t a2 = (v[i][2][w] >> sh) & 0xffffu, a3 = (v[i][3][w] >> sh) & 0xffffu;
          *(u32x2_t *)(lds + (rb * 8 + e) * LDK + kb * 4) = u32x2_t{a0 | (a1 << 16), a2 | (a3 << 16)};
        }
      }
    }
  }
};

template <typename Cfg, bool A_K, bool B_K>
__global__ __launch_bounds__(Cfg::NT, 1) void gemm_mfma_kernel(
    int M, int N, int K, int k_per_split, const bf16_t *A, int64_t lda, const bf16_t *B,
    int64_t ldb, EpArgs ep, float *partial) {
  constexpr int BM = Cfg::BM, BN = Cfg::BN, BK = Cfg::BK, LDK = Cfg::LDK, NT = Cfg::NT;
  __shared__ __attribute__((aligned(16))) uint16_t As[2][BM * LDK];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[2][BN * LDK];

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

  Stager<BM, BK, LDK, NT, A_K> sa;
  Stager<BN, BK, LDK, NT, B_K> sb;
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
    const uint16_t *as = As[buf] + (wm * Cfg::WTM + (lane & 31)) * LDK + (lane >> 5) * 8;
    const uint16_t *bs = Bs[buf] + (wn * Cfg::WTN + (lane & 31)) * LDK + (lane >> 5) * 8;
#pragma unroll
    for (int kk = 0; kk < BK; kk += 16) {
      bf16x8_t af[Cfg::TM], bfr[Cfg::TN];
#pragma unroll
      for (int i = 0; i < Cfg::TM; ++i) af[i] = *(const bf16x8_t *)(as + i * 32 * LDK + kk);
#pragma unroll
      for (int j = 0; j < Cfg::TN; ++j) bfr[j] = *(const bf16x8_t *)(bs + j * 32 * LDK + kk);
#pragma unroll
      for (int i = 0; i < Cfg::TM; ++i)
#pragma unroll
        for (int j = 0; j < Cfg::TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
      // the other buffer was last read before the previous barrier: fill it
      // while this one is still being consumed
      if (kk == BK / 2 - 16 && kt + 1 < nk) {
        sa.store(As[buf ^ 1]);
        sb.store(Bs[buf ^ 1]);
      }
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
           aligned16(g.A) && aligned16(g.B) && !(!g.a_kmajor && g.b_kmajor);
  }
  if (mfma) {
    const int kc = g.a_kmajor ? (g.b_kmajor ? AJ_KC_GEMM_NT : AJ_KC_GEMM_NN) : AJ_KC_GEMM_TN;
    const int tk = timing_begin(s, kc, g.recompute ? 0.0 : 2.0 * g.M * g.N * (double)g.K);
    if (g.a_kmajor && g.b_kmajor) launch_mfma<CfgBig, true, true>(g, ep, kps, s);
    else if (g.a_kmajor) launch_mfma<CfgBig, true, false>(g, ep, kps, s);
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
