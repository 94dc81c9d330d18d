// aj_logprob_pg_loss_fwd / _bwd: final RMSNorm, vocab projection,
// log-softmax, token log-prob and the clipped policy-gradient loss.
//
// Only the rows that feed a target are normalised and projected (the loss
// reads no other logits).
// bfloat16: the forward is one MFMA GEMM over the whole vocab whose epilogue
// reduces each 256-column logit tile to a per-row (max, sum of exp) partial
// and picks up the target's logit; a small kernel then combines the partials
// into the log-sum-exp.  The backward recomputes each vocab_chunk-wide slab of
// logits and its epilogue writes
//   dz = g * (onehot(target) - softmax)        g = d loss / d logprob
// in bfloat16, then dhn += dz W_chunk and dW_chunk += dz^T hn are GEMMs.
// With keep_logits the forward epilogue also stores its float32 logits (the
// same values the recomputation would produce: same tiles, same reduction
// order) and the backward forms dz from them element by element, trading the
// second vocab projection for ~3 x 4 bytes of HBM traffic per logit.
// float32 (the small workload): the same arithmetic with each chunk of logits
// written to a float32 buffer and reduced by row kernels.
#include <type_traits>
#include "ops.h"
#include "gemm_core.h"

namespace {

struct LossWs {
  float *z, *run_m, *run_s, *zt, *part, *g, *dhn, *dg_part;
  float2 *tile_ms;        // fused forward: per (row, 256-column tile) (max, sum of exp), log2 units
  float *splitk;          // split-K partials of the dW_vocab GEMM
  size_t splitk_floats;
  void *dz;
  int32_t *tpos, *trow;   // targets clamped into the documented range, and their h rows
  size_t bytes;
};

constexpr int kFinBlocks = 256;

// Vocab chunks per group of the backward's d hidden and d W products: the d
// logits of a group's chunks sit side by side in one [n_tgt, group width]
// buffer, so each product runs once per group.  bfloat16 chunks of up to
// 16384 columns go in pairs (a 32768-wide buffer at most); wider ones, and
// float32, one at a time.
int chunk_group(const aj_loss_cfg &c) {
  return c.dtype == AJ_BF16 && c.vocab_chunk <= 16384 ? 2 : 1;
}

// Widths of the groups: full groups, and the last one (narrower when the
// vocab is not a multiple of the group's width).
void group_widths(const aj_loss_cfg &c, int64_t *full, int64_t *last) {
  const int64_t cw = c.vocab_chunk < c.vocab ? c.vocab_chunk : c.vocab;
  const int64_t gw = cw * chunk_group(c);
  *full = gw < c.vocab ? gw : c.vocab;
  *last = c.vocab % *full == 0 ? *full : c.vocab % *full;
}

LossWs carve_ws(const aj_loss_cfg &c, int n_tgt, void *base) {
  const size_t es = c.dtype == AJ_BF16 ? 2 : 4;
  const int64_t cw = c.vocab_chunk < c.vocab ? c.vocab_chunk : c.vocab;
  int64_t gfull, glast;
  group_widths(c, &gfull, &glast);
  aj::Carver cv(base);
  LossWs w;
  w.z = cv.take<float>(c.dtype == AJ_BF16 ? 1 : (int64_t)n_tgt * cw);
  w.tile_ms = cv.take<float2>(c.dtype == AJ_BF16 ? (int64_t)n_tgt * ((c.vocab + 255) / 256) : 1);
  w.dz = cv.take<char>((int64_t)n_tgt * gfull * es);
  w.run_m = cv.take<float>(n_tgt);
  w.run_s = cv.take<float>(n_tgt);
  w.zt = cv.take<float>(n_tgt);
  w.g = cv.take<float>(n_tgt);
  w.tpos = cv.take<int32_t>(n_tgt);
  w.trow = cv.take<int32_t>(n_tgt);
  w.part = cv.take<float>(kFinBlocks * 8);
  w.dhn = cv.take<float>((int64_t)n_tgt * c.d_model);
  w.dg_part = cv.take<float>(aj::rmsnorm_bwd_part_floats(n_tgt, c.d_model));
  // the dW_vocab GEMM runs on full groups and on the last, narrower one:
  // their split-K factors (tile counts) differ
  const size_t sk = std::max(aj::gemm_split_floats((int)gfull, c.d_model, n_tgt),
                             aj::gemm_split_floats((int)glast, c.d_model, n_tgt));
  w.splitk = cv.take<float>(sk > 0 ? sk : 1);
  w.splitk_floats = sk > 0 ? sk : 1;
  w.bytes = cv.bytes();
  return w;
}

struct LossSaved {
  void *hn;
  float *rstd;
  float *z;               // keep_logits: [n_tgt, vocab] float32 logits, else null
  size_t bytes;
};

bool keeps_logits(const aj_loss_cfg &c) { return c.keep_logits != 0 && c.dtype == AJ_BF16; }

LossSaved carve_saved(const aj_loss_cfg &c, int n_tgt, void *base) {
  const size_t es = c.dtype == AJ_BF16 ? 2 : 4;
  aj::Carver cv(base);
  LossSaved s;
  s.hn = cv.take<char>((int64_t)n_tgt * c.d_model * es);
  s.rstd = cv.take<float>(n_tgt);
  s.z = keeps_logits(c) ? cv.take<float>((int64_t)n_tgt * c.vocab) : nullptr;
  s.bytes = cv.bytes();
  return s;
}

AJ_DEV float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
AJ_DEV float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Target p is scored from h row p - 1 - row_base; anything outside [0, n_tok)
// is reported and clamped so that no access leaves the documented ranges.
__global__ void sanitize_targets_kernel(int n, const int32_t *targets, int row_base, int n_tok,
                                        int32_t *tpos, int32_t *trow, int32_t *err) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  int r = targets[i] - 1 - row_base;
  if (r < 0 || r >= n_tok) {
    if (err) atomicOr(err, AJ_DEVERR_OFFSETS);
    r = r < 0 ? 0 : n_tok - 1;
  }
  trow[i] = r;
  tpos[i] = r + 1 + row_base;
}

__global__ void loss_init_kernel(int n, float *run_m, float *run_s, float *zt) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  run_m[i] = -INFINITY;
  run_s[i] = 0.f;
  zt[i] = 0.f;
}

// One wave per row: fold chunk [c0, c0+cw) of logits into the running max/sum,
// and pick up the target's logit if it lies in the chunk.
__global__ __launch_bounds__(256) void lse_update_kernel(const float *z, int n, int cw, int c0,
                                                         const int32_t *tpos,
                                                         const int32_t *tok, int vocab,
                                                         float *run_m, float *run_s, float *zt,
                                                         int32_t *err) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= n) return;
  const float *zr = z + (int64_t)row * cw;
  float m = -INFINITY;
  for (int j = lane; j < cw; j += 64) m = fmaxf(m, zr[j]);
  m = wave_max(m);
  float s = 0.f;
  for (int j = lane; j < cw; j += 64) s += __expf(zr[j] - m);
  s = wave_sum(s);
  if (lane == 0) {
    const float mo = run_m[row], so = run_s[row];
    const float mn = fmaxf(mo, m);
    run_s[row] = so * __expf(mo - mn) + s * __expf(m - mn);
    run_m[row] = mn;
    const int t = tok[tpos[row]];
    if (t >= c0 && t < c0 + cw) zt[row] = zr[t - c0];
    if (c0 == 0 && (t < 0 || t >= vocab) && err) atomicOr(err, AJ_DEVERR_TOKEN_RANGE);
  }
}

__global__ void token_check_kernel(int n, const int32_t *tpos, const int32_t *tok, int vocab,
                                   int32_t *err) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n || !err) return;
  const int t = tok[tpos[i]];
  if (t < 0 || t >= vocab) atomicOr(err, AJ_DEVERR_TOKEN_RANGE);
}

// d loss / d logprob for one target (unnormalised by N_mask).
AJ_DEV float pg_grad(float lp, float old, float A, float eps, float *term, int *clipped,
                     float *ratio) {
  const float r = __expf(lp - old);
  const float rc = fminf(fmaxf(r, 1.f - eps), 1.f + eps);
  *term = -fminf(r * A, rc * A);
  const bool active = (A > 0.f && r <= 1.f + eps) || (A < 0.f && r >= 1.f - eps);
  *clipped = (!active && A != 0.f) ? 1 : 0;
  *ratio = r;
  return active ? -A * r : 0.f;
}

// Low-variance KL estimate of the policy against the reference at one
// target (delta = ref - lp): exp(delta) - delta - 1, clamped to [-10, 10];
// *dkl = d kl / d lp (0 where clamped).
AJ_DEV float kl_low_var(float lp, float ref, float *dkl) {
  const float delta = ref - lp;
  const float e = __expf(delta);
  const float kl = e - delta - 1.f;
  if (kl > 10.f || kl < -10.f) {
    *dkl = 0.f;
    return kl > 10.f ? 10.f : -10.f;
  }
  *dkl = 1.f - e;
  return kl;
}

constexpr int kStats = 5;

// run_m == nullptr: logprob (and lse) are already written.
__global__ __launch_bounds__(256) void loss_finalize_kernel(
    int n, const int32_t *tpos, const float *old_lp, const float *adv, float eps, float inv_n,
    const float *ref_lp, float kl_coef, const float *run_m, const float *run_s, const float *zt,
    float *logprob, float *lse, float *part) {
  __shared__ float red[kStats][256];
  float acc[kStats] = {0.f, 0.f, 0.f, 0.f, 0.f};
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
    float lp;
    if (run_m) {
      const float l = run_m[i] + logf(run_s[i]);
      lp = zt[i] - l;
      lse[i] = l;
      logprob[i] = lp;
    } else {
      lp = logprob[i];
    }
    const int p = tpos[i];
    float term, r;
    int clipped;
    pg_grad(lp, old_lp[p], adv[p], eps, &term, &clipped, &r);
    float kl = 0.f;
    if (ref_lp) {
      float dkl;
      kl = kl_low_var(lp, ref_lp[i], &dkl);
      term += kl_coef * kl;
    }
    acc[0] += term * inv_n;
    acc[1] += (float)clipped;
    acc[2] += r;
    acc[3] += 1.f;
    acc[4] += kl;
  }
#pragma unroll
  for (int k = 0; k < kStats; ++k) red[k][threadIdx.x] = acc[k];
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if ((int)threadIdx.x < s)
#pragma unroll
      for (int k = 0; k < kStats; ++k) red[k][threadIdx.x] += red[k][threadIdx.x + s];
    __syncthreads();
  }
  if (threadIdx.x < kStats) part[blockIdx.x * kStats + threadIdx.x] = red[threadIdx.x][0];
}

__global__ void stats_reduce_kernel(const float *part, int nb, float *stats) {
  const int k = threadIdx.x;
  if (k >= kStats) return;
  float s = 0.f;
  for (int b = 0; b < nb; ++b) s += part[b * kStats + k];
  stats[k] += s;
}

__global__ void loss_grad_kernel(int n, const int32_t *tpos, const float *logprob,
                                 const float *old_lp, const float *adv, float eps, float inv_n,
                                 const float *ref_lp, float kl_coef, float *g) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int p = tpos[i];
  float term, r;
  int clipped;
  float d = pg_grad(logprob[i], old_lp[p], adv[p], eps, &term, &clipped, &r);
  if (ref_lp) {
    float dkl;
    kl_low_var(logprob[i], ref_lp[i], &dkl);
    d += kl_coef * dkl;
  }
  g[i] = d * inv_n;
}

// dz[i][j] = g_i * ((c0 + j == target_i) - exp(z_ij - lse_i))
template <typename T>
__global__ __launch_bounds__(256) void dz_kernel(const float *z, int n, int cw, int c0,
                                                 const int32_t *tpos, const int32_t *tok,
                                                 const float *lse, const float *g, T *dz) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)n * cw) return;
  const int i = (int)(idx / cw), j = (int)(idx % cw);
  const float gi = g[i];
  const float p = __expf(z[idx] - lse[i]);
  const float oh = (tok[tpos[i]] == c0 + j) ? 1.f : 0.f;
  stf(dz + idx, gi * (oh - p));
}


// ---------------------------------------------------------------- fused (bfloat16)
namespace gemm_core = aj::gemm_core;
using Cfg = gemm_core::CfgWide;
template <bool A_K, bool B_K> using Smem = gemm_core::Smem4s<A_K, B_K>;
using gemm_core::f32x16_t;
constexpr float kLog2e = 1.4426950408889634f;
// 2^x on the hardware unit (v_exp_f32) for arguments <= 0 or -inf (a
// logit minus a running maximum or the log-sum-exp): no range handling needed.
AJ_DEV float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
constexpr float kLn2 = 0.6931471805599453f;

// Reductions over each row of 16 lanes on the DPP network (no LDS traffic):
// swaps within pairs and quads, then the mirrors of 8 and 16 lanes.  Every
// lane of the row ends with the result.
template <int CTRL>
AJ_DEV float dpp(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL,
                                                               0xF, 0xF, false));
}
constexpr int kQuadXor1 = 0xB1, kQuadXor2 = 0x4E, kRowHalfMirror = 0x141, kRowMirror = 0x140;
AJ_DEV float row16_max(float v) {
  v = fmaxf(v, dpp<kQuadXor1>(v));
  v = fmaxf(v, dpp<kQuadXor2>(v));
  v = fmaxf(v, dpp<kRowHalfMirror>(v));
  return fmaxf(v, dpp<kRowMirror>(v));
}
AJ_DEV float row16_sum(float v) {
  v += dpp<kQuadXor1>(v);
  v += dpp<kQuadXor2>(v);
  v += dpp<kRowHalfMirror>(v);
  return v + dpp<kRowMirror>(v);
}

// LDS writes (or reads) complete, then a barrier; unlike __syncthreads this
// does not wait for the workgroup's global stores.
AJ_DEV void lds_barrier() {
  __asm__ volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  gemm_core::bar_nofence();
}

// logits tile z = hn W^T (rows: targets, columns: 256 vocab ids) reduced in
// registers: per row, the tile's max and sum of exp (log2 units) and, in the
// tile that holds it, the target's logit.  Logits never leave the chip.
// B_K: the vocab weights as stored, [V][d] (k-major) or transposed [d][V].
template <bool B_K>
__global__ __launch_bounds__(Cfg::NT, 1) void lm_fwd_fused_kernel(
    int n, int V, int d, const bf16_t *hn, const bf16_t *wv, int ldw, const int32_t *tpos,
    const int32_t *tok, float2 *tile_ms, float *zt, float *zkeep) {
  __shared__ __attribute__((aligned(16))) gemm_core::Smem4s<true, B_K, 4> sm;
  __shared__ int ttok[Cfg::BM];
  __shared__ float2 red[Cfg::WN][Cfg::BM];
  const int tiles_m = (n + Cfg::BM - 1) / Cfg::BM, tiles_n = (V + Cfg::BN - 1) / Cfg::BN;
  const gemm_core::TileIdx ti = gemm_core::tile_of(blockIdx.x, gridDim.x, tiles_m, tiles_n);
  const int m0 = ti.tm * Cfg::BM, n0 = ti.tn * Cfg::BN;
  if (threadIdx.x < Cfg::BM) {
    const int m = m0 + threadIdx.x;
    ttok[threadIdx.x] = m < n ? tok[tpos[m]] : -1;
  }
  f32x16_t acc[Cfg::TM][Cfg::TN];
  gemm_core::mainloop8s<true, B_K, Cfg, 4>(acc, hn, d, wv, ldw, n, V, m0, n0, 0, d, sm);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / Cfg::WN, wn = wave % Cfg::WN;
  // A row of this wave's 128 columns lives in the 32 lanes of a half-wave, 4
  // columns each: reduce over 16 lanes by DPP, then across the two rows of
  // 16 with one exchange per row, issued for all 16 rows of a pass together.
  const int col0 = n0 + wn * Cfg::WTN + (lane & 31);
  if (zkeep) {
    // the tile's logits for the backward: per accumulator row, the 32 lanes
    // of a half-wave store 32 consecutive columns
#pragma unroll
    for (int i = 0; i < Cfg::TM; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + gemm_core::acc_row<Cfg>(wm, i, r, lane);
        if (m >= n) continue;
        float *zr = zkeep + (int64_t)m * V;
#pragma unroll
        for (int j = 0; j < Cfg::TN; ++j)
          if (col0 + 32 * j < V) zr[col0 + 32 * j] = acc[i][j][r];
      }
  }
  auto epilogue = [&](auto inside) {
    constexpr bool kInside = decltype(inside)::value;   // every column < V
#pragma unroll
    for (int i = 0; i < Cfg::TM; ++i) {
      float mx[16], sm_[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float m = -INFINITY;
#pragma unroll
        for (int j = 0; j < Cfg::TN; ++j)
          if (kInside || col0 + 32 * j < V) m = fmaxf(m, acc[i][j][r]);
        mx[r] = row16_max(m * kLog2e);
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) mx[r] = fmaxf(mx[r], __shfl_xor(mx[r], 16, 64));
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float t = 0.f;
#pragma unroll
        for (int j = 0; j < Cfg::TN; ++j)
          if (kInside || col0 + 32 * j < V) t += fast_exp2(acc[i][j][r] * kLog2e - mx[r]);
        sm_[r] = row16_sum(t);
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) sm_[r] += __shfl_xor(sm_[r], 16, 64);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int rl = gemm_core::acc_row<Cfg>(wm, i, r, lane);
        if ((lane & 31) == 0) red[wn][rl] = make_float2(mx[r], sm_[r]);
        // the target's logit, in the lane that holds its column
        const int t = ttok[rl] - col0;
        if (t >= 0 && t < Cfg::TN * 32 && (t & 31) == 0 && m0 + rl < n) {
          float z = acc[i][0][r];
#pragma unroll
          for (int j = 1; j < Cfg::TN; ++j)
            if (t == 32 * j) z = acc[i][j][r];
          zt[m0 + rl] = z;
        }
      }
    }
  };
  if (n0 + Cfg::BN <= V) epilogue(std::true_type{});
  else epilogue(std::false_type{});
  lds_barrier();
  if (threadIdx.x < Cfg::BM && m0 + (int)threadIdx.x < n) {
    float M = -INFINITY, S = 0.f;
#pragma unroll
    for (int w = 0; w < Cfg::WN; ++w) M = fmaxf(M, red[w][threadIdx.x].x);
#pragma unroll
    for (int w = 0; w < Cfg::WN; ++w)   // a wave past the vocab end holds (-inf, 0)
      S += red[w][threadIdx.x].x == -INFINITY ? 0.f
                                               : red[w][threadIdx.x].y * fast_exp2(red[w][threadIdx.x].x - M);
    tile_ms[(int64_t)(m0 + threadIdx.x) * tiles_n + ti.tn] = make_float2(M, S);
  }
}

// One wave per row: combine the row's tile partials into its log-sum-exp.
__global__ __launch_bounds__(256) void lm_combine_kernel(int n, int n_tiles, const float2 *tile_ms,
                                                         const float *zt, float *lse,
                                                         float *logprob) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= n) return;
  const float2 *p = tile_ms + (int64_t)row * n_tiles;
  float M = -INFINITY;
  for (int t = lane; t < n_tiles; t += 64) M = fmaxf(M, p[t].x);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) M = fmaxf(M, __shfl_xor(M, o, 64));
  float S = 0.f;
  for (int t = lane; t < n_tiles; t += 64) S += p[t].x == -INFINITY ? 0.f : p[t].y * fast_exp2(p[t].x - M);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) S += __shfl_xor(S, o, 64);
  if (lane == 0) {
    const float l = (M + log2f(S)) * kLn2;
    lse[row] = l;
    logprob[row] = zt[row] - l;
  }
}

// d logit of logit z in a row with log-sum-exp tl (log2 units) and loss
// gradient g: g (onehot - softmax).  One definition for the recomputing and
// the logit-keeping backward, so that both round identically.
AJ_DEV float dz_value(float z, float tl, float g, bool target) {
  const float p = fast_exp2(fmaf(z, kLog2e, -tl));
  return g * ((target ? 1.f : 0.f) - p);
}

// dz from the kept logits of vocab columns [c0, c0 + cw): 8 columns per
// thread (V, c0 and cw multiples of 8, 16-byte aligned rows) or, on the
// general path, one.
template <bool kVec>
__global__ __launch_bounds__(256) void lm_dz_kept_kernel(int n, int cw, int c0, int V,
                                                         const float *zkeep, const int32_t *tpos,
                                                         const int32_t *tok, const float *lse,
                                                         const float *g, bf16_t *dz, int ldz) {
  constexpr int E = kVec ? 8 : 1;
  const int per_row = cw / E;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)n * per_row) return;
  const int m = (int)(idx / per_row), cb = (int)(idx % per_row) * E;
  const float tl = lse[m] * kLog2e, gm = g[m];
  const int tt = tok[tpos[m]] - c0;
  const float *zr = zkeep + (int64_t)m * V + c0 + cb;
  if (kVec) {
    const float4 a = *reinterpret_cast<const float4 *>(zr);
    const float4 b = *reinterpret_cast<const float4 *>(zr + 4);
    const float v[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      w[e] = f2bf2(dz_value(v[2 * e], tl, gm, cb + 2 * e == tt),
                   dz_value(v[2 * e + 1], tl, gm, cb + 2 * e + 1 == tt));
    *reinterpret_cast<uint4 *>(dz + (int64_t)m * ldz + cb) = make_uint4(w[0], w[1], w[2], w[3]);
  } else {
    dz[(int64_t)m * ldz + cb] = f2bf(dz_value(zr[0], tl, gm, cb == tt));
  }
}

// dz = g (onehot(target) - softmax) for vocab columns [c0, c0 + cw), from the
// recomputed logits, straight to bfloat16.
// wc: the chunk's vocab weights, [cw][d] (B_K) or columns of the transposed
// [d][V] copy, row stride ldw.
template <bool B_K>
__global__ __launch_bounds__(Cfg::NT, 1) void lm_dz_fused_kernel(
    int n, int cw, int c0, int d, const bf16_t *hn, const bf16_t *wc, int ldw,
    const int32_t *tpos, const int32_t *tok, const float *lse, const float *g, bf16_t *dz,
    int ldz) {
  // The body is device code only: this compiler's host pass rejects the
  // main-loop call of the B_K = true instance (its device pass accepts both).
#if defined(__HIP_DEVICE_COMPILE__)
  __shared__ __attribute__((aligned(16))) gemm_core::Smem4s<true, B_K, 4> sm;
  __shared__ int ttok[Cfg::BM];
  __shared__ float tl[Cfg::BM], tg[Cfg::BM];
  const int tiles_m = (n + Cfg::BM - 1) / Cfg::BM, tiles_n = (cw + Cfg::BN - 1) / Cfg::BN;
  const gemm_core::TileIdx ti = gemm_core::tile_of(blockIdx.x, gridDim.x, tiles_m, tiles_n);
  const int m0 = ti.tm * Cfg::BM, n0 = ti.tn * Cfg::BN;
  if (threadIdx.x < Cfg::BM) {
    const int m = m0 + threadIdx.x;
    ttok[threadIdx.x] = m < n ? tok[tpos[m]] - c0 : -1;
    tl[threadIdx.x] = m < n ? lse[m] * kLog2e : 0.f;
    tg[threadIdx.x] = m < n ? g[m] : 0.f;
  }
  f32x16_t acc[Cfg::TM][Cfg::TN];
  gemm_core::mainloop8s<true, B_K, Cfg, 4>(acc, hn, d, wc, ldw, n, cw, m0, n0, 0, d, sm);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / Cfg::WN, wn = wave % Cfg::WN;
  auto dz_of = [&](float a, int rl, int col) { return dz_value(a, tl[rl], tg[rl], col == ttok[rl]); };
  if (m0 + Cfg::BM > n || n0 + Cfg::BN > cw || cw % 8 != 0 || ldz % 8 != 0 ||
      ((uintptr_t)dz & 15) != 0) {
    // edge tile: element by element
#pragma unroll
    for (int i = 0; i < Cfg::TM; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int rl = gemm_core::acc_row<Cfg>(wm, i, r, lane);
        const int m = m0 + rl;
        if (m >= n) continue;
#pragma unroll
        for (int j = 0; j < Cfg::TN; ++j) {
          const int col = n0 + gemm_core::acc_col<Cfg>(wn, j, lane);
          if (col >= cw) continue;
          dz[(int64_t)m * ldz + col] = f2bf(dz_of(acc[i][j][r], rl, col));
        }
      }
    return;
  }
  // Interior tile: dz staged as bfloat16 rows through LDS (the stage ring is
  // free once every wave is past the main loop), 128 rows per pass (32 of each
  // wave row), then written 16 bytes per lane.
  constexpr int LDH = Cfg::BN + 8;   // bf16 elements per staged row
  uint16_t *stage = reinterpret_cast<uint16_t *>(&sm);
  lds_barrier();
#pragma unroll
  for (int i = 0; i < Cfg::TM; ++i) {
    // the pass's per-row values, read before any staging write
    float rl2[16], rg[16];
    int rt[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int rl = gemm_core::acc_row<Cfg>(wm, i, r, lane);
      rl2[r] = tl[rl];
      rg[r] = tg[rl];
      rt[r] = ttok[rl] - n0;
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int ls = wm * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
#pragma unroll
      for (int j = 0; j < Cfg::TN; ++j) {
        const int cl = gemm_core::acc_col<Cfg>(wn, j, lane);
        stage[ls * LDH + cl] = f2bf(dz_value(acc[i][j][r], rl2[r], rg[r], cl == rt[r]));
      }
    }
    lds_barrier();
    constexpr int Q = 128 * (Cfg::BN / 8) / Cfg::NT;   // 16-byte chunks per thread
    uint4 v[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int c = threadIdx.x + Cfg::NT * q;
      v[q] = *reinterpret_cast<const uint4 *>(stage + (c >> 5) * LDH + (c & 31) * 8);
    }
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int c = threadIdx.x + Cfg::NT * q;
      const int ls = c >> 5;
      const int m = m0 + (ls >> 5) * Cfg::WTM + 32 * i + (ls & 31);
      *reinterpret_cast<uint4 *>(dz + (int64_t)m * ldz + n0 + (c & 31) * 8) = v[q];
    }
    lds_barrier();
  }
#endif
}

int check_cfg(const aj_loss_cfg *c, const aj_loss_in *in, const char *name) {
  AJ_REQUIRE(c && in, AJ_ERR_NULL, "%s: null cfg/in", name);
  AJ_REQUIRE(c->dtype == AJ_F32 || c->dtype == AJ_BF16, AJ_ERR_UNSUPPORTED, "%s: dtype", name);
  AJ_REQUIRE(c->d_model > 0 && c->d_model % 8 == 0 && c->d_model <= 8192, AJ_ERR_SHAPE,
             "%s: d_model %d", name, c->d_model);
  AJ_REQUIRE(c->vocab > 0 && c->vocab_chunk > 0 && c->vocab_chunk % 8 == 0, AJ_ERR_SHAPE,
             "%s: vocab %d chunk %d", name, c->vocab, c->vocab_chunk);
  AJ_REQUIRE(c->clip_eps >= 0 && c->rms_eps > 0, AJ_ERR_SHAPE, "%s: eps", name);
  AJ_REQUIRE(in->n_tok >= 0 && in->n_tgt >= 0 && in->n_tgt <= in->n_tok, AJ_ERR_SHAPE,
             "%s: n_tok %d n_tgt %d", name, in->n_tok, in->n_tgt);
  AJ_REQUIRE(!in->w_vocab_t || c->vocab % 8 == 0, AJ_ERR_SHAPE,
             "%s: the transposed vocab weights need vocab %% 8 == 0 (vocab %d)", name, c->vocab);
  AJ_REQUIRE(in->n_tgt == 0 || (in->targets && in->tok && in->old_logprob && in->adv),
             AJ_ERR_NULL, "%s: null input arrays", name);
  return AJ_OK;
}

template <typename T>
int chunk_logits(const aj_loss_cfg &c, int n_tgt, const void *hn, const void *w_vocab, int c0,
                 int cw, float *z, hipStream_t st, bool recompute) {
  aj::Gemm g;
  g.recompute = recompute;
  g.M = n_tgt; g.N = cw; g.K = c.d_model;
  g.A = hn; g.lda = c.d_model;
  g.B = (const T *)w_vocab + (int64_t)c0 * c.d_model; g.ldb = c.d_model;
  g.C = z; g.ldc = cw; g.c_f32 = true;
  return aj::gemm<T>(g, st);
}

template <typename T>
int loss_fwd(const aj_loss_cfg &c, const aj_loss_in &in, const void *h, const void *gf,
             const void *w_vocab, const LossSaved &sv, float *logprob, float *lse, float *stats,
             int32_t *err, const LossWs &w, hipStream_t st) {
  const int n = in.n_tgt, d = c.d_model;
  sanitize_targets_kernel<<<(n + 255) / 256, 256, 0, st>>>(n, in.targets, in.row_base, in.n_tok,
                                                           w.tpos, w.trow, err);
  aj::rmsnorm_fwd<T>((const T *)h, (const T *)gf, n, d, c.rms_eps, w.trow, 0, (T *)sv.hn,
                     sv.rstd, st);
  const bool fused = sizeof(T) == 2;
  if (fused) {
    loss_init_kernel<<<(n + 255) / 256, 256, 0, st>>>(n, w.run_m, w.run_s, w.zt);
    const int tiles_n = (c.vocab + Cfg::BN - 1) / Cfg::BN;
    const int tiles = ((n + Cfg::BM - 1) / Cfg::BM) * tiles_n;
    const int tk = aj::timing_begin(st, AJ_KC_LM_FWD, 2.0 * n * (double)c.vocab * d);
    if (in.w_vocab_t)
      lm_fwd_fused_kernel<false><<<tiles, Cfg::NT, 0, st>>>(
          n, c.vocab, d, (const bf16_t *)sv.hn, (const bf16_t *)in.w_vocab_t, c.vocab, w.tpos,
          in.tok, w.tile_ms, w.zt, sv.z);
    else
      lm_fwd_fused_kernel<true><<<tiles, Cfg::NT, 0, st>>>(
          n, c.vocab, d, (const bf16_t *)sv.hn, (const bf16_t *)w_vocab, d, w.tpos, in.tok,
          w.tile_ms, w.zt, sv.z);
    aj::timing_end(st, tk);
    lm_combine_kernel<<<(n + 3) / 4, 256, 0, st>>>(n, tiles_n, w.tile_ms, w.zt, lse, logprob);
    token_check_kernel<<<(n + 255) / 256, 256, 0, st>>>(n, w.tpos, in.tok, c.vocab, err);
  } else {
    loss_init_kernel<<<(n + 255) / 256, 256, 0, st>>>(n, w.run_m, w.run_s, w.zt);
    for (int c0 = 0; c0 < c.vocab; c0 += c.vocab_chunk) {
      const int cw = c.vocab - c0 < c.vocab_chunk ? c.vocab - c0 : c.vocab_chunk;
      int r = chunk_logits<T>(c, n, sv.hn, w_vocab, c0, cw, w.z, st, false);
      if (r) return r;
      lse_update_kernel<<<(n + 3) / 4, 256, 0, st>>>(w.z, n, cw, c0, w.tpos, in.tok, c.vocab,
                                                    w.run_m, w.run_s, w.zt, err);
    }
  }
  int nb = (n + 255) / 256;
  if (nb > kFinBlocks) nb = kFinBlocks;
  const float *ref = in.kl_coef != 0.f ? in.ref_logprob : nullptr;
  loss_finalize_kernel<<<nb, 256, 0, st>>>(n, w.tpos, in.old_logprob, in.adv, c.clip_eps,
                                           in.inv_n_mask, ref, in.kl_coef,
                                           fused ? nullptr : w.run_m, w.run_s, w.zt, logprob,
                                           lse, w.part);
  stats_reduce_kernel<<<1, 64, 0, st>>>(w.part, nb, stats);
  return aj::check_launch("aj_logprob_pg_loss_fwd");
}

template <typename T>
int loss_bwd(const aj_loss_cfg &c, const aj_loss_in &in, const void *h, const void *gf,
             const void *w_vocab, const LossSaved &sv, const float *logprob, const float *lse,
             float *dh, float *dgf, float *dwv, const LossWs &w, hipStream_t st) {
  const int n = in.n_tgt, d = c.d_model;
  aj::fill_f32(dh, (int64_t)in.n_tok * d, 0.f, st);
  if (n == 0) return aj::check_launch("aj_logprob_pg_loss_bwd");
  sanitize_targets_kernel<<<(n + 255) / 256, 256, 0, st>>>(n, in.targets, in.row_base, in.n_tok,
                                                           w.tpos, w.trow, nullptr);
  const float *ref = in.kl_coef != 0.f ? in.ref_logprob : nullptr;
  loss_grad_kernel<<<(n + 255) / 256, 256, 0, st>>>(n, w.tpos, logprob, in.old_logprob, in.adv,
                                                    c.clip_eps, in.inv_n_mask, ref, in.kl_coef,
                                                    w.g);
  aj::fill_f32(w.dhn, (int64_t)n * d, 0.f, st);
  // groups of chunk_group(c) vocab chunks: the chunks' d logits (one launch
  // each, as in the forward) side by side in w.dz, then one d hidden and one
  // d W product over the whole group
  const int G = chunk_group(c);
  for (int g0 = 0; g0 < c.vocab; g0 += G * c.vocab_chunk) {
    const int gw = c.vocab - g0 < G * c.vocab_chunk ? c.vocab - g0 : G * c.vocab_chunk;
    int r;
    for (int c0 = g0; c0 < g0 + gw; c0 += c.vocab_chunk) {
      const int cw = g0 + gw - c0 < c.vocab_chunk ? g0 + gw - c0 : c.vocab_chunk;
      if (sizeof(T) == 2 && sv.z) {
        bf16_t *dz = (bf16_t *)w.dz + (c0 - g0);
        const bool vec = c.vocab % 8 == 0 && c0 % 8 == 0 && cw % 8 == 0 && gw % 8 == 0 &&
                         (c0 - g0) % 8 == 0 && ((uintptr_t)sv.z & 15) == 0 &&
                         ((uintptr_t)w.dz & 15) == 0;
        const int64_t work = (int64_t)n * (vec ? cw / 8 : cw);
        const unsigned blocks = (unsigned)((work + 255) / 256);
        const int tk = aj::timing_begin(st, AJ_KC_LM_DZ, 0.0);
        if (vec)
          lm_dz_kept_kernel<true><<<blocks, 256, 0, st>>>(n, cw, c0, c.vocab, sv.z, w.tpos,
                                                          in.tok, lse, w.g, dz, gw);
        else
          lm_dz_kept_kernel<false><<<blocks, 256, 0, st>>>(n, cw, c0, c.vocab, sv.z, w.tpos,
                                                           in.tok, lse, w.g, dz, gw);
        aj::timing_end(st, tk);
      } else if (sizeof(T) == 2) {
        bf16_t *dz = (bf16_t *)w.dz + (c0 - g0);
        const int tiles = ((n + Cfg::BM - 1) / Cfg::BM) * ((cw + Cfg::BN - 1) / Cfg::BN);
        const int tk = aj::timing_begin(st, AJ_KC_LM_DZ, 0.0);   // recomputes the forward product
        if (in.w_vocab_t)
          lm_dz_fused_kernel<false><<<tiles, Cfg::NT, 0, st>>>(
              n, cw, c0, d, (const bf16_t *)sv.hn, (const bf16_t *)in.w_vocab_t + c0, c.vocab,
              w.tpos, in.tok, lse, w.g, dz, gw);
        else
          lm_dz_fused_kernel<true><<<tiles, Cfg::NT, 0, st>>>(
              n, cw, c0, d, (const bf16_t *)sv.hn, (const bf16_t *)w_vocab + (int64_t)c0 * d, d,
              w.tpos, in.tok, lse, w.g, dz, gw);
        aj::timing_end(st, tk);
      } else {   // float32: one chunk per group
        if ((r = chunk_logits<T>(c, n, sv.hn, w_vocab, c0, cw, w.z, st, true))) return r;
        const int64_t tot = (int64_t)n * cw;
        dz_kernel<T><<<(unsigned)((tot + 255) / 256), 256, 0, st>>>(w.z, n, cw, c0, w.tpos,
                                                                    in.tok, lse, w.g, (T *)w.dz);
      }
    }
    aj::Gemm g;   // dhn += dz W_group
    g.M = n; g.N = d; g.K = gw; g.A = w.dz; g.lda = gw;
    g.B = (const T *)w_vocab + (int64_t)g0 * d; g.ldb = d; g.b_kmajor = false;
    g.C = w.dhn; g.ldc = d; g.out = aj::OUT_ACCUM_F32;
    if ((r = aj::gemm<T>(g, st))) return r;
    if (!dwv) continue;   // frozen LM head
    g = aj::Gemm();   // dW_group += dz^T hn
    g.M = gw; g.N = d; g.K = n; g.A = w.dz; g.lda = gw; g.a_kmajor = false;
    g.B = sv.hn; g.ldb = d; g.b_kmajor = false;
    g.C = dwv + (int64_t)g0 * d; g.ldc = d; g.out = aj::OUT_ACCUM_F32;
    g.split_k = aj::gemm_split_k(g.M, g.N, g.K); g.partial = w.splitk;
    g.partial_cap = w.splitk_floats;
    if ((r = aj::gemm<T>(g, st))) return r;
  }
  aj::rmsnorm_bwd<T>(w.dhn, (const T *)h, sv.rstd, (const T *)gf, n, d, w.trow, 0, 1,
                     nullptr, dh, nullptr, w.dg_part, dgf, st);
  return aj::check_launch("aj_logprob_pg_loss_bwd");
}

}  // namespace

extern "C" size_t aj_loss_saved_bytes(const aj_loss_cfg *cfg, int32_t n_tgt) {
  if (!cfg || n_tgt < 0) return 0;
  return carve_saved(*cfg, n_tgt, nullptr).bytes;
}

extern "C" size_t aj_loss_workspace_bytes(const aj_loss_cfg *cfg, int32_t n_tgt) {
  if (!cfg || n_tgt < 0) return 0;
  return carve_ws(*cfg, n_tgt, nullptr).bytes;
}

extern "C" int aj_logprob_pg_loss_fwd(const aj_loss_cfg *cfg, const aj_loss_in *in, const void *h,
                                      const void *final_norm, const void *w_vocab, void *saved,
                                      float *logprob, float *lse, float *stats, int32_t *err,
                                      void *ws, size_t ws_bytes, void *stream) {
  const char *name = "aj_logprob_pg_loss_fwd";
  int r;
  if ((r = check_cfg(cfg, in, name))) return r;
  AJ_REQUIRE(stats, AJ_ERR_NULL, "%s: null stats", name);
  if (in->n_tgt == 0) return AJ_OK;
  AJ_REQUIRE(h && final_norm && w_vocab && saved && logprob && lse && ws, AJ_ERR_NULL,
             "%s: null pointer", name);
  LossWs w = carve_ws(*cfg, in->n_tgt, ws);
  AJ_REQUIRE(ws_bytes >= w.bytes, AJ_ERR_WORKSPACE, "%s: workspace %zu < %zu", name, ws_bytes,
             w.bytes);
  LossSaved sv = carve_saved(*cfg, in->n_tgt, saved);
  hipStream_t st = (hipStream_t)stream;
  const aj::StageSpan span(st, AJ_KC_STAGE_LOSS);
  if (cfg->dtype == AJ_BF16)
    return loss_fwd<bf16_t>(*cfg, *in, h, final_norm, w_vocab, sv, logprob, lse, stats, err, w, st);
  return loss_fwd<float>(*cfg, *in, h, final_norm, w_vocab, sv, logprob, lse, stats, err, w, st);
}

extern "C" int aj_logprob_pg_loss_bwd(const aj_loss_cfg *cfg, const aj_loss_in *in, const void *h,
                                      const void *final_norm, const void *w_vocab,
                                      const void *saved, const float *logprob, const float *lse,
                                      float *dh, float *d_final_norm, float *d_w_vocab, void *ws,
                                      size_t ws_bytes, void *stream) {
  const char *name = "aj_logprob_pg_loss_bwd";
  int r;
  if ((r = check_cfg(cfg, in, name))) return r;
  if (in->n_tok == 0) return AJ_OK;
  AJ_REQUIRE(dh, AJ_ERR_NULL, "%s: null dh", name);
  AJ_REQUIRE(in->n_tgt == 0 || (h && final_norm && w_vocab && saved && logprob && lse && ws),
             AJ_ERR_NULL, "%s: null pointer", name);
  LossWs w = carve_ws(*cfg, in->n_tgt, ws);
  AJ_REQUIRE(in->n_tgt == 0 || ws_bytes >= w.bytes, AJ_ERR_WORKSPACE, "%s: workspace %zu < %zu",
             name, ws_bytes, w.bytes);
  LossSaved sv = carve_saved(*cfg, in->n_tgt, const_cast<void *>(saved));
  hipStream_t st = (hipStream_t)stream;
  const aj::StageSpan span(st, AJ_KC_STAGE_LOSS);
  if (cfg->dtype == AJ_BF16)
    return loss_bwd<bf16_t>(*cfg, *in, h, final_norm, w_vocab, sv, logprob, lse, dh, d_final_norm,
                            d_w_vocab, w, st);
  return loss_bwd<float>(*cfg, *in, h, final_norm, w_vocab, sv, logprob, lse, dh, d_final_norm,
                         d_w_vocab, w, st);
}
