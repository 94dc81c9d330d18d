// Internal kernel launchers shared by the block and loss entry points.
#pragma once
#include "common.h"

namespace aj {

template <typename T>
void embed_fwd(const int32_t *tok, int n, const T *emb, int d, int vocab, T *x, int32_t *err,
               hipStream_t s);

// out[i] = RMSNorm(x[r]) * g, r = rows ? rows[i] + shift : i; rstd[i] saved.
template <typename T>
void rmsnorm_fwd(const T *x, const T *g, int n, int d, float eps, const int32_t *rows, int shift,
                 T *out, float *rstd, hipStream_t s);
// Backward of the above; dg += sum over rows (deterministic, via dg_part of
// rmsnorm_bwd_part_floats floats; dg null: the gain is frozen, not reduced).  dx / dx_t (either may be null) receive
// add + d x; with scatter they are indexed by r instead of i.
size_t rmsnorm_bwd_part_floats(int n, int d);
template <typename T>
void rmsnorm_bwd(const float *dy, const T *x, const float *rstd, const T *g, int n, int d,
                 const int32_t *rows, int shift, int scatter, const float *add, float *dx, T *dx_t,
                 float *dg_part, float *dg, hipStream_t s);

// Rotate-half RoPE in place on the first n_rot_heads heads of each row (row
// stride ld); inverse applies the transposed rotation (the backward).
template <typename T>
void rope(T *qkv, int n, const int32_t *pos, int n_rot_heads, int ld, int hd, float theta,
          bool inverse, hipStream_t s);

template <typename T>
void swiglu_fwd(const T *gu, int n, int F, T *out, hipStream_t s);
template <typename TI, typename T>
void swiglu_bwd(const TI *ds, const T *gu, int n, int F, T *dgu, hipStream_t s);

template <typename T>
void cast_from_f32(const float *in, int64_t n, T *out, hipStream_t s);
// out[i] = scale * in[i] rounded once to T; lo (optional) receives the
// rounding residual, also in T, so that out + lo carries ~twice T's precision.
template <typename T>
void scale_cast(const float *in, int64_t n, float scale, T *out, T *lo, hipStream_t s);
void fill_f32(float *p, int64_t n, float v, hipStream_t s);
// dst[c][r] = src[r][c] for a row-major [rows, cols] matrix of 16-bit elements.
void transpose16(const void *src, int rows, int cols, void *dst, hipStream_t s);
void splitk_reduce(const float *part, int S, int64_t n, float *out, bool accumulate, hipStream_t s);

// ---------------------------------------------------------------- GEMM
// C[M,N] (op) sum_k A(m,k) B(n,k)
//   A(m,k) = a_kmajor ? A[m*lda + k] : A[k*lda + m]
//   B(n,k) = b_kmajor ? B[n*ldb + k] : B[k*ldb + n]
enum GemmOut { OUT_STORE = 0, OUT_ACCUM_F32 = 1 };
struct Gemm {
  int M = 0, N = 0, K = 0;
  const void *A = nullptr; int64_t lda = 0; bool a_kmajor = true;
  const void *B = nullptr; int64_t ldb = 0; bool b_kmajor = true;
  void *C = nullptr; int64_t ldc = 0;
  bool c_f32 = false;          // C element type: float32, else the input type
  int out = OUT_STORE;         // OUT_ACCUM_F32: C (float32) += A B
  const void *R = nullptr;     // optional residual, same type/ld as C: C = A B + R
  int split_k = 1;             // > 1: partial sums in `partial`, reduced in fixed order
  float *partial = nullptr;    // split_k * M * N floats (OUT_ACCUM_F32 or c_f32 only)
  size_t partial_cap = 0;      // floats available at `partial` (checked before any launch)
  // SwiGLU backward in the epilogue (bfloat16 only, no split-K): the product is
  // d s (N = F columns); with gate g = gu[m][n] and up u = gu[m][F + n] (row
  // stride ldc = 2F) the epilogue stores d gate = d s u sig(g) (1 + g (1 - sig(g)))
  // at C[m][n] and d up = d s g sig(g) at C[m][F + n]
  const void *swiglu_gu = nullptr;
  bool recompute = false;      // recomputes a forward product: no algorithmic flops
  // optional second reduction segment, same operand layouts, no split-K:
  // C (op) A B + A2 B2 with k in [0, K) and [0, K2)
  const void *A2 = nullptr; int64_t lda2 = 0;
  const void *B2 = nullptr; int64_t ldb2 = 0;
  int K2 = 0;
};
template <typename T>
int gemm(const Gemm &g, hipStream_t s);

// Split-K factor for an M x N output over K (K/S >= 4096): with fewer 256x256
// tiles than CUs, enough splits for ~1.5-2 rounds of 256 workgroups; with
// more, a split of at most 4 when it fills the last round clearly better
// (one workgroup per CU: a part-filled round costs a whole one).
inline int gemm_split_k(int M, int N, int K) {
  const int tiles = ((M + 255) / 256) * ((N + 255) / 256);
  if (K < 8192) return 1;
  const int kmax = K / 4096 < 16 ? K / 4096 : 16;
  if (tiles < 240) {
    const int S = (448 + tiles - 1) / tiles;
    return S > kmax ? kmax : (S < 1 ? 1 : S);
  }
  auto idle = [&](int S) {   // idle fraction of the rounds
    const long t = (long)tiles * S, slots = (t + 255) / 256 * 256;
    return (double)(slots - t) / (double)slots;
  };
  int best = 1;
  for (int S = 2; S <= 4 && S <= kmax; ++S)
    if (idle(S) < idle(best) - 0.08) best = S;
  return best;
}
// Floats of split-K partials gemm() needs for such a GEMM (0 when no split).
inline size_t gemm_split_floats(int M, int N, int K) {
  const int S = gemm_split_k(M, N, K);
  return S > 1 ? (size_t)S * M * N : 0;
}

// ---------------------------------------------------------------- attention
struct AttnArgs {
  int n_tok, n_seg, Hq, Hkv, hd;
  int base;             // cu_seqlens values are row offsets + base
  const int32_t *cu_seqlens;
  const void *qkv;      // [n_tok, (Hq+2Hkv)*hd], q and k already rotated
  void *o;              // [n_tok, Hq*hd]
  float *lse;           // [Hq, n_tok] log-sum-exp of the scaled scores (log2 units on
                        // the matrix-core path, natural log on the plain one)
  float scale;
};
template <typename T>
int attn_fwd(const AttnArgs &a, hipStream_t s);

struct AttnBwdArgs {
  int n_tok, n_seg, Hq, Hkv, hd;
  int base;
  const int32_t *cu_seqlens;
  const void *qkv, *o, *dout;
  const float *lse;
  float *delta;         // [Hq, n_tok] workspace
  void *dqkv;           // [n_tok, (Hq+2Hkv)*hd] written
  float scale;
};
template <typename T>
int attn_bwd(const AttnBwdArgs &a, hipStream_t s);

// bfloat16 MFMA flash attention (head_dim 64 or 128, 16-byte aligned tensors)
bool attn_mfma_supported(int hd, const void *p0, const void *p1, const void *p2);
int attn_fwd_mfma(const AttnArgs &a, hipStream_t s);
int attn_bwd_mfma(const AttnBwdArgs &a, hipStream_t s);

}  // namespace aj
