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
#include "gemm_core.h"

namespace aj {
namespace {

struct EpArgs {
  int M, N;
  void *C; int64_t ldc;
  int c_f32, accum;
  const void *R;
  int vec;   // 4-column vector stores are aligned (C, R, partial rows)
  const bf16_t *gu;   // SwiGLU backward: [gate | up] rows (stride ldc), else null
};

// d gate, d up of one SwiGLU element from d s (float32) and bf16 gate / up
AJ_DEV void swiglu_grad(float ds, float g, float u, float &dg, float &du) {
  const float sg = 1.f / (1.f + __expf(-g));
  dg = ds * u * sg * (1.f + g * (1.f - sg));
  du = ds * g * sg;
}

using gemm_core::f32x16_t;

// LDS stages of the staged GEMM kernels (128 KB).  A fifth stage (the whole
// 160 KB, copies four k-steps ahead) measured no faster: the copies are bound
// by the rate of 64-byte row requests, not by how far ahead they run.
constexpr int kStages = 4;

// A second reduction segment with the operand layouts of the first:
// C = A B + A2 B2 over k in [0, K) and [0, K2).
struct Seg2 {
  const bf16_t *A; int64_t lda;
  const bf16_t *B; int64_t ldb;
  int K;
};

// Output modes of the epilogue's fast path (interior tiles, aligned rows).
enum { kEpPartial, kEpAccum, kEpF32, kEpF32R, kEpBf16, kEpBf16R, kEpSwiglu };

// One pass of the fast epilogue: the 64 staged rows (32 of each wave row)
// x 256 columns, 4 columns per thread and instruction; every LDS read of the
// pass is issued before the first store.
template <int MODE, typename Cfg>
AJ_DEV void store_pass(const float *stage, int i, int m0, int n0, int64_t ldo, float *P,
                       const EpArgs &ep) {
  static_assert(Cfg::WTM == 128 && Cfg::BN == 256, "two wave rows of 128, 256 columns");
  constexpr int LDW = Cfg::BN + 8;
  constexpr int Q = 64 * 64 / Cfg::NT;
  float4 v[Q];
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int c = threadIdx.x + Cfg::NT * q;
    v[q] = *reinterpret_cast<const float4 *>(stage + (c >> 6) * LDW + (c & 63) * 4);
  }
  auto offset = [&](int q) {
    const int c = threadIdx.x + Cfg::NT * q;
    const int row = c >> 6;
    return (int64_t)(m0 + (row >> 5) * 128 + 32 * i + (row & 31)) * ldo + n0 + (c & 63) * 4;
  };
  if constexpr (MODE == kEpAccum || MODE == kEpF32R) {
    const float *src = MODE == kEpAccum ? (const float *)ep.C : (const float *)ep.R;
    float4 u[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) u[q] = *reinterpret_cast<const float4 *>(src + offset(q));
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const float4 w = make_float4(v[q].x + u[q].x, v[q].y + u[q].y, v[q].z + u[q].z,
                                   v[q].w + u[q].w);
      *reinterpret_cast<float4 *>((float *)ep.C + offset(q)) = w;
    }
  } else if constexpr (MODE == kEpSwiglu) {
    uint2 g4[Q], u4[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      g4[q] = *reinterpret_cast<const uint2 *>(ep.gu + offset(q));
      u4[q] = *reinterpret_cast<const uint2 *>(ep.gu + offset(q) + ep.N);
    }
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const float dsv[4] = {v[q].x, v[q].y, v[q].z, v[q].w};
      const float gv[4] = {__uint_as_float(g4[q].x << 16), __uint_as_float(g4[q].x & 0xffff0000u),
                           __uint_as_float(g4[q].y << 16), __uint_as_float(g4[q].y & 0xffff0000u)};
      const float uv[4] = {__uint_as_float(u4[q].x << 16), __uint_as_float(u4[q].x & 0xffff0000u),
                           __uint_as_float(u4[q].y << 16), __uint_as_float(u4[q].y & 0xffff0000u)};
      float dg[4], du[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) swiglu_grad(dsv[e], gv[e], uv[e], dg[e], du[e]);
      bf16_t *cp = (bf16_t *)ep.C + offset(q);
      *reinterpret_cast<uint2 *>(cp) = make_uint2(f2bf2(dg[0], dg[1]), f2bf2(dg[2], dg[3]));
      *reinterpret_cast<uint2 *>(cp + ep.N) = make_uint2(f2bf2(du[0], du[1]), f2bf2(du[2], du[3]));
    }
  } else if constexpr (MODE == kEpBf16R) {
    uint2 u[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) u[q] = *reinterpret_cast<const uint2 *>((const bf16_t *)ep.R + offset(q));
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      uint2 out;
      out.x = f2bf2(v[q].x + __uint_as_float(u[q].x << 16),
                    v[q].y + __uint_as_float(u[q].x & 0xffff0000u));
      out.y = f2bf2(v[q].z + __uint_as_float(u[q].y << 16),
                    v[q].w + __uint_as_float(u[q].y & 0xffff0000u));
      *reinterpret_cast<uint2 *>((bf16_t *)ep.C + offset(q)) = out;
    }
  } else {
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      if constexpr (MODE == kEpPartial) {
        *reinterpret_cast<float4 *>(P + offset(q)) = v[q];
      } else if constexpr (MODE == kEpF32) {
        *reinterpret_cast<float4 *>((float *)ep.C + offset(q)) = v[q];
      } else {
        uint2 out;
        out.x = f2bf2(v[q].x, v[q].y);
        out.y = f2bf2(v[q].z, v[q].w);
        *reinterpret_cast<uint2 *>((bf16_t *)ep.C + offset(q)) = out;
      }
    }
  }
}

// LDS writes of the staged rows (or their reads) complete, then a barrier:
// unlike __syncthreads, the tile's global stores stay in flight.
AJ_DEV void epi_barrier() {
  __asm__ volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  gemm_core::bar_nofence();
}

// Shared body of the two GEMM kernels: main loop of configuration C (and the
// second segment's, SEG2), then the epilogue through LDS.
template <bool A_K, bool B_K, typename Cfg, bool SEG2 = false, bool STAGED = false,
          typename SM = gemm_core::Smem<A_K, B_K, Cfg>>
AJ_DEV void gemm_tile(int M, int N, int K, int k_per_split, const bf16_t *A, int64_t lda,
                      const bf16_t *B, int64_t ldb, const EpArgs &ep, float *partial, SM &sm,
                      const Seg2 &s2 = Seg2{}) {
  const int tiles_m = (M + Cfg::BM - 1) / Cfg::BM, tiles_n = (N + Cfg::BN - 1) / Cfg::BN;
  const gemm_core::TileIdx ti = gemm_core::tile_of(blockIdx.x, gridDim.x, tiles_m, tiles_n);
  const int m0 = ti.tm * Cfg::BM, n0 = ti.tn * Cfg::BN;
  const int kbeg = blockIdx.z * k_per_split;
  const int kend = min(K, kbeg + k_per_split);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / Cfg::WN, wn = wave % Cfg::WN;
  f32x16_t acc[Cfg::TM][Cfg::TN];
  if constexpr (STAGED && Cfg::NT == 256) {
    static_assert(!SEG2, "the staged loops take one segment");
    gemm_core::mainloop4s<A_K, B_K, SM::kStages>(acc, A, lda, B, ldb, M, N, m0, n0, kbeg, kend,
                                                 sm);
  } else if constexpr (STAGED) {
    static_assert(!SEG2, "the staged loops take one segment");
    gemm_core::mainloop8s<A_K, B_K, Cfg, SM::kStages>(acc, A, lda, B, ldb, M, N, m0, n0, kbeg,
                                                      kend, sm);
  } else {
    static_assert(Cfg::NT == 512, "8-wave tile");
    gemm_core::mainloop<A_K, B_K, Cfg>(acc, A, lda, B, ldb, M, N, m0, n0, kbeg, kend, sm);
    if constexpr (SEG2)
      gemm_core::mainloop<A_K, B_K, Cfg>(acc, s2.A, s2.lda, s2.B, s2.ldb, M, N, m0, n0, 0, s2.K,
                                         sm, false);
  }
  epi_barrier();

  // Epilogue through LDS, 32 rows of each wave row at a time: the lane's
  // accumulators (column lane%32, rows 8*(r/4) + 4*(lane/32) + r%4 of each
  // 32x32 tile) are staged as rows, then written out 4 columns per lane.
  // Interior tiles with aligned rows take a pass specialised to the output
  // mode (no per-element branches, the pass's LDS reads issued together);
  // edge tiles go element by element.
  float *stage = reinterpret_cast<float *>(&sm);
  constexpr int LDW = Cfg::BN + 8;
  float *P = partial ? partial + (int64_t)blockIdx.z * M * N : nullptr;
  const int64_t ldo = partial ? N : ep.ldc;
  const bool fast = ep.vec && m0 + Cfg::BM <= M && n0 + Cfg::BN <= N;
  const int mode = P ? kEpPartial
                   : ep.gu ? kEpSwiglu
                   : ep.accum ? kEpAccum
                   : ep.c_f32 ? (ep.R ? kEpF32R : kEpF32)
                              : (ep.R ? kEpBf16R : kEpBf16);
#pragma unroll
  for (int i = 0; i < Cfg::TM; ++i) {
#pragma unroll
    for (int j = 0; j < Cfg::TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int lr = wm * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        stage[lr * LDW + wn * Cfg::WTN + j * 32 + (lane & 31)] = acc[i][j][r];
      }
    epi_barrier();
    if (fast) {
      switch (mode) {
        case kEpPartial: store_pass<kEpPartial, Cfg>(stage, i, m0, n0, ldo, P, ep); break;
        case kEpAccum: store_pass<kEpAccum, Cfg>(stage, i, m0, n0, ldo, P, ep); break;
        case kEpF32: store_pass<kEpF32, Cfg>(stage, i, m0, n0, ldo, P, ep); break;
        case kEpF32R: store_pass<kEpF32R, Cfg>(stage, i, m0, n0, ldo, P, ep); break;
        case kEpBf16: store_pass<kEpBf16, Cfg>(stage, i, m0, n0, ldo, P, ep); break;
        case kEpSwiglu:
          // 8-wave tiles only: in the 4-wave one the extra pass pushes the
          // epilogue past full unrolling and the accumulator into scratch
          if constexpr (Cfg::NT == 512) store_pass<kEpSwiglu, Cfg>(stage, i, m0, n0, ldo, P, ep);
          break;
        default: store_pass<kEpBf16R, Cfg>(stage, i, m0, n0, ldo, P, ep); break;
      }
      epi_barrier();
      continue;
    }
#pragma unroll 4
    for (int q = 0; q < 64 * 64 / Cfg::NT; ++q) {
      const int c = threadIdx.x + Cfg::NT * q;
      const int row = c >> 6, c4 = (c & 63) * 4;
      const int m = m0 + (row >> 5) * 128 + 32 * i + (row & 31), n = n0 + c4;
      if (m >= M || n >= N) continue;
      const float4 v = *reinterpret_cast<const float4 *>(stage + row * LDW + c4);
      const int64_t o = (int64_t)m * ldo + n;
      if (ep.gu) {
        const float vv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (n + e >= N) break;
          float dg, du;
          swiglu_grad(vv[e], bf2f(ep.gu[o + e]), bf2f(ep.gu[o + e + N]), dg, du);
          ((bf16_t *)ep.C)[o + e] = f2bf(dg);
          ((bf16_t *)ep.C)[o + e + N] = f2bf(du);
        }
        continue;
      }
      if (ep.vec && n + 4 <= N) {
        if (P) {
          *reinterpret_cast<float4 *>(P + o) = v;
        } else if (ep.c_f32) {
          float4 *cp = reinterpret_cast<float4 *>((float *)ep.C + o);
          float4 w = v;
          if (ep.accum) {
            const float4 u = *cp;
            w.x += u.x; w.y += u.y; w.z += u.z; w.w += u.w;
          } else if (ep.R) {
            const float4 u = *reinterpret_cast<const float4 *>((const float *)ep.R + o);
            w.x += u.x; w.y += u.y; w.z += u.z; w.w += u.w;
          }
          *cp = w;
        } else {
          float w0 = v.x, w1 = v.y, w2 = v.z, w3 = v.w;
          if (ep.R) {
            const uint2 u = *reinterpret_cast<const uint2 *>((const bf16_t *)ep.R + o);
            w0 += __uint_as_float(u.x << 16); w1 += __uint_as_float(u.x & 0xffff0000u);
            w2 += __uint_as_float(u.y << 16); w3 += __uint_as_float(u.y & 0xffff0000u);
          }
          uint2 out;
          out.x = f2bf2(w0, w1);
          out.y = f2bf2(w2, w3);
          *reinterpret_cast<uint2 *>((bf16_t *)ep.C + o) = out;
        }
      } else {
        const float vv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (n + e >= N) break;
          const float x = vv[e];
          if (P) {
            P[o + e] = x;
          } else if (ep.accum) {
            ((float *)ep.C)[o + e] += x;
          } else if (ep.c_f32) {
            ((float *)ep.C)[o + e] = x + (ep.R ? ((const float *)ep.R)[o + e] : 0.f);
          } else {
            ((bf16_t *)ep.C)[o + e] = f2bf(x + (ep.R ? bf2f(((const bf16_t *)ep.R)[o + e]) : 0.f));
          }
        }
      }
    }
    epi_barrier();
  }
}

// 8 waves of 128x64: the default.
template <bool A_K, bool B_K>
__global__ __launch_bounds__(gemm_core::Cfg::NT, 1) void gemm_mfma_kernel(
    int M, int N, int K, int k_per_split, const bf16_t *A, int64_t lda, const bf16_t *B,
    int64_t ldb, EpArgs ep, float *partial) {
  __shared__ __attribute__((aligned(16))) gemm_core::Smem4s<A_K, B_K, kStages> sm;
  gemm_tile<A_K, B_K, gemm_core::Cfg, false, true>(M, N, K, k_per_split, A, lda, B, ldb, ep,
                                                   partial, sm);
}

// 4 waves of 128x128 with 32-wide k-steps in four LDS stages (copies three
// k-steps ahead): reductions of kLongK and more.
template <bool A_K, bool B_K>
__global__ __launch_bounds__(gemm_core::Cfg4::NT, 1) void gemm_mfma4s_kernel(
    int M, int N, int K, int k_per_split, const bf16_t *A, int64_t lda, const bf16_t *B,
    int64_t ldb, EpArgs ep, float *partial) {
  __shared__ __attribute__((aligned(16))) gemm_core::Smem4s<A_K, B_K, kStages> sm;
  gemm_tile<A_K, B_K, gemm_core::Cfg4, false, true>(M, N, K, k_per_split, A, lda, B, ldb, ep,
                                                    partial, sm);
}

// The 8-wave kernel with a second reduction segment (no split-K; used with
// either reduction length).
template <bool A_K, bool B_K>
__global__ __launch_bounds__(gemm_core::Cfg::NT, 1) void gemm_mfma_seg2_kernel(
    int M, int N, int K, const bf16_t *A, int64_t lda, const bf16_t *B, int64_t ldb, Seg2 s2,
    EpArgs ep) {
  __shared__ __attribute__((aligned(16))) gemm_core::Smem<A_K, B_K, gemm_core::Cfg> sm;
  gemm_tile<A_K, B_K, gemm_core::Cfg, true>(M, N, K, K, A, lda, B, ldb, ep, nullptr, sm, s2);
}

constexpr int kLongK = 4096;

// ---------------------------------------------------------------- float32 / fallback
template <typename T>
__global__ __launch_bounds__(256) void gemm_simple_kernel(int M, int N, int K, int k_per_split,
                                                          const T *A, int64_t lda, int a_k,
                                                          const T *B, int64_t ldb, int b_k,
                                                          EpArgs ep, float *partial,
                                                          const T *A2, int64_t lda2,
                                                          const T *B2, int64_t ldb2, int K2) {
  constexpr int BM = 64, BN = 64, BK = 16;
  __shared__ float As[BK][BM + 1];
  __shared__ float Bs[BK][BN + 1];
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int tx = threadIdx.x % 16, ty = threadIdx.x / 16;
  float acc[4][4] = {};
  // segment 0: [kbeg, kend) of (A, B); segment 1 (no split): [0, K2) of (A2, B2)
  for (int seg = 0; seg < (K2 > 0 ? 2 : 1); ++seg) {
    const T *X = seg ? A2 : A, *Y = seg ? B2 : B;
    const int64_t ldx = seg ? lda2 : lda, ldy = seg ? ldb2 : ldb;
    const int kbeg = seg ? 0 : blockIdx.z * k_per_split;
    const int kend = seg ? K2 : min(K, kbeg + k_per_split);
    for (int k0 = kbeg; k0 < kend; k0 += BK) {
      for (int e = threadIdx.x; e < BM * BK; e += 256) {
        int mm = e % BM, kk = e / BM;
        int m = m0 + mm, k = k0 + kk;
        float va = 0.f, vb = 0.f;
        if (m < M && k < kend) va = ldf(X + (a_k ? (int64_t)m * ldx + k : (int64_t)k * ldx + m));
        int n = n0 + mm;
        if (n < N && k < kend) vb = ldf(Y + (b_k ? (int64_t)n * ldy + k : (int64_t)k * ldy + n));
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
      } else if (ep.gu) {
        const int64_t o = (int64_t)m * ep.ldc + n;
        float dg, du;
        swiglu_grad(v, bf2f(ep.gu[o]), bf2f(ep.gu[o + N]), dg, du);
        stf((T *)ep.C + o, dg);
        stf((T *)ep.C + o + N, du);
      } else {
        T *c = (T *)ep.C + (int64_t)m * ep.ldc + n;
        stf(c, v + (ep.R ? ldf((const T *)ep.R + (int64_t)m * ep.ldc + n) : 0.f));
      }
    }
}

template <bool A_K, bool B_K>
void launch_mfma(const Gemm &g, const EpArgs &ep, int kps, bool long_k, hipStream_t s) {
  const int tiles = ((g.M + 255) / 256) * ((g.N + 255) / 256);
  dim3 grid(tiles, 1, g.split_k);
  float *part = g.split_k > 1 ? g.partial : nullptr;
  if (g.K2 > 0) {
    const Seg2 s2{(const bf16_t *)g.A2, g.lda2, (const bf16_t *)g.B2, g.ldb2, g.K2};
    gemm_mfma_seg2_kernel<A_K, B_K><<<tiles, gemm_core::Cfg::NT, 0, s>>>(
        g.M, g.N, g.K, (const bf16_t *)g.A, g.lda, (const bf16_t *)g.B, g.ldb, s2, ep);
    return;
  }
  if (long_k)
    gemm_mfma4s_kernel<A_K, B_K><<<grid, gemm_core::Cfg4::NT, 0, s>>>(
        g.M, g.N, g.K, kps, (const bf16_t *)g.A, g.lda, (const bf16_t *)g.B, g.ldb, ep, part);
  else
    gemm_mfma_kernel<A_K, B_K><<<grid, gemm_core::Cfg::NT, 0, s>>>(
        g.M, g.N, g.K, kps, (const bf16_t *)g.A, g.lda, (const bf16_t *)g.B, g.ldb, ep, part);
}

bool aligned16(const void *p) { return ((uintptr_t)p & 15) == 0; }

}  // namespace

template <typename T>
int gemm(const Gemm &g, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return AJ_OK;
  if (g.split_k > 1 && !g.partial) return fail(AJ_ERR_WORKSPACE, "gemm: split-K without workspace");
  if (g.split_k > 1 && (size_t)g.split_k * g.M * g.N > g.partial_cap)
    return fail(AJ_ERR_WORKSPACE, "gemm: split-K %d of %d x %d needs %zu floats, workspace has %zu",
                g.split_k, g.M, g.N, (size_t)g.split_k * g.M * g.N, g.partial_cap);
  if (g.K2 > 0 && (g.split_k > 1 || !g.A2 || !g.B2))
    return fail(AJ_ERR_UNSUPPORTED, "gemm: a second segment needs its operands and no split-K");
  EpArgs ep{g.M, g.N, g.C, g.ldc, g.c_f32 ? 1 : 0, g.out == OUT_ACCUM_F32 ? 1 : 0, g.R, 0,
            (const bf16_t *)g.swiglu_gu};
  if (g.swiglu_gu && (sizeof(T) != 2 || g.split_k > 1 || ep.accum || ep.c_f32 || g.R ||
                      g.ldc < 2 * (int64_t)g.N))
    return fail(AJ_ERR_UNSUPPORTED, "gemm: SwiGLU epilogue needs bf16 C [n, 2N], no split-K, "
                "accumulation or residual");
  if (ep.accum) ep.c_f32 = 1;
  {
    const uintptr_t al = ep.c_f32 ? 15 : 7;
    const bool split = g.split_k > 1;
    ep.vec = split ? (g.N % 4 == 0 && ((uintptr_t)g.partial & 15) == 0)
                   : (g.ldc % 4 == 0 && ((uintptr_t)g.C & al) == 0 && ((uintptr_t)g.R & al) == 0 &&
                      (!g.swiglu_gu || (g.N % 4 == 0 && ((uintptr_t)g.swiglu_gu & 7) == 0)));
  }
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
    if (g.K2 > 0) {
      const int a2 = g.a_kmajor ? g.K2 : g.M, b2 = g.b_kmajor ? g.K2 : g.N;
      mfma = mfma && a2 % 8 == 0 && b2 % 8 == 0 && g.lda2 % 8 == 0 && g.ldb2 % 8 == 0 &&
             aligned16(g.A2) && aligned16(g.B2);
    }
  }
  if (mfma) {
    // the second segment and the SwiGLU epilogue run 8-wave
    const bool long_k = kps >= kLongK && g.K2 == 0 && !g.swiglu_gu;
    int kc = g.a_kmajor ? (g.b_kmajor ? AJ_KC_GEMM_NT : AJ_KC_GEMM_NN) : AJ_KC_GEMM_TN;
    if (long_k) kc += AJ_KC_GEMM4_NT - AJ_KC_GEMM_NT;
    const int tk =
        timing_begin(s, kc, g.recompute ? 0.0 : 2.0 * g.M * g.N * ((double)g.K + g.K2));
    if (g.a_kmajor && g.b_kmajor) launch_mfma<true, true>(g, ep, kps, long_k, s);
    else if (g.a_kmajor) launch_mfma<true, false>(g, ep, kps, long_k, s);
    else if (g.b_kmajor) launch_mfma<false, true>(g, ep, kps, long_k, s);
    else launch_mfma<false, false>(g, ep, kps, long_k, s);
    timing_end(s, tk);
  } else {
    dim3 grid((g.N + 63) / 64, (g.M + 63) / 64, S);
    gemm_simple_kernel<T><<<grid, 256, 0, s>>>(g.M, g.N, g.K, kps, (const T *)g.A, g.lda,
                                               g.a_kmajor, (const T *)g.B, g.ldb, g.b_kmajor, ep,
                                               S > 1 ? g.partial : nullptr, (const T *)g.A2,
                                               g.lda2, (const T *)g.B2, g.ldb2, g.K2);
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
