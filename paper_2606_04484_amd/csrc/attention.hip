// Causal GQA attention over packed variable-length segments.
//
// Tiles are runs of consecutive packed rows; a row attends to the keys of its
// own segment up to itself, [seg_start(row), row], with seg_start found from
// cu_seqlens.  Query head h reads key/value head floor(h * Hkv / Hq).
//
// These kernels use float FMA with 4 threads per query row (a quarter of the
// head dimension each) and stream keys through LDS; they serve the float32
// workload and head dims other than 64 and 128.  bfloat16 with head_dim 64 or
// 128 goes to the MFMA kernels in attention_mfma.hip.
#include "ops.h"

namespace aj {
namespace {

constexpr int kRows = 64;     // query (or key) rows per workgroup
constexpr int kKv = 32;       // rows staged in LDS per step
constexpr int kMaxHd = 128;

AJ_DEV int seg_of(const int32_t *cu, int n_seg, int base, int row) {
  int lo = 0, hi = n_seg - 1;   // largest s with cu[s] - base <= row
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (cu[mid] - base <= row) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// First row of row's segment, clamped into [0, row] whatever cu_seqlens holds.
template <typename A>
AJ_DEV int seg_start(const A &a, int row) {
  const int v = a.cu_seqlens[seg_of(a.cu_seqlens, a.n_seg, a.base, row)] - a.base;
  return v < 0 ? 0 : (v > row ? row : v);
}

// One past the last row of row's segment, clamped into [row + 1, n_tok].
template <typename A>
AJ_DEV int seg_end(const A &a, int row) {
  const int v = a.cu_seqlens[seg_of(a.cu_seqlens, a.n_seg, a.base, row) + 1] - a.base;
  return v <= row ? row + 1 : (v > a.n_tok ? a.n_tok : v);
}

AJ_DEV float quad_sum(float v) {
  v += __shfl_xor(v, 1, 64);
  v += __shfl_xor(v, 2, 64);
  return v;
}

template <typename T>
__global__ __launch_bounds__(256) void attn_fwd_simple_kernel(AttnArgs a) {
  __shared__ float Ks[kKv][kMaxHd + 1];
  __shared__ float Vs[kKv][kMaxHd + 1];
  __shared__ int range[2];
  const int hd = a.hd, qd = hd / 4;
  const int ld = (a.Hq + 2 * a.Hkv) * hd;
  const int h = blockIdx.y, g = (h * a.Hkv) / a.Hq;
  const int row0 = blockIdx.x * kRows;
  const int rl = threadIdx.x >> 2, part = threadIdx.x & 3;
  const int row = row0 + rl;
  const bool valid = row < a.n_tok;
  const T *qkv = (const T *)a.qkv;
  int start = 0;
  if (valid) start = seg_start(a, row);
  if (threadIdx.x == 0) {
    int last = min(row0 + kRows, a.n_tok) - 1;
    range[0] = seg_start(a, row0);
    range[1] = last;
  }
  float q[kMaxHd / 4], o[kMaxHd / 4];
#pragma unroll
  for (int i = 0; i < kMaxHd / 4; ++i) {
    q[i] = (valid && i < qd) ? ldf(qkv + (int64_t)row * ld + h * hd + part * qd + i) * a.scale : 0.f;
    o[i] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  __syncthreads();
  const int kv_lo = range[0], kv_hi = range[1];
  for (int k0 = kv_lo; k0 <= kv_hi; k0 += kKv) {
    for (int e = threadIdx.x; e < kKv * hd; e += 256) {
      int r = e / hd, c = e % hd, kr = k0 + r;
      float kv = 0.f, vv = 0.f;
      if (kr <= kv_hi) {
        kv = ldf(qkv + (int64_t)kr * ld + (a.Hq + g) * hd + c);
        vv = ldf(qkv + (int64_t)kr * ld + (a.Hq + a.Hkv + g) * hd + c);
      }
      Ks[r][c] = kv;
      Vs[r][c] = vv;
    }
    __syncthreads();
    for (int j = 0; j < kKv; ++j) {
      const int key = k0 + j;
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < kMaxHd / 4; ++i)
        if (i < qd) s += q[i] * Ks[j][part * qd + i];
      s = quad_sum(s);
      if (!valid || key < start || key > row) continue;
      const float mn = fmaxf(m, s);
      const float sc = __expf(m - mn), p = __expf(s - mn);
      l = l * sc + p;
#pragma unroll
      for (int i = 0; i < kMaxHd / 4; ++i)
        if (i < qd) o[i] = o[i] * sc + p * Vs[j][part * qd + i];
      m = mn;
    }
    __syncthreads();
  }
  if (!valid) return;
  T *out = (T *)a.o + (int64_t)row * a.Hq * hd + h * hd + part * qd;
  const float inv = 1.f / l;
#pragma unroll
  for (int i = 0; i < kMaxHd / 4; ++i)
    if (i < qd) stf(out + i, o[i] * inv);
  if (part == 0) a.lse[(int64_t)h * a.n_tok + row] = m + logf(l);
}

// delta[h][row] = sum_d dO * O
template <typename T>
__global__ __launch_bounds__(256) void attn_delta_kernel(AttnBwdArgs a) {
  const int64_t idx = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (idx >= (int64_t)a.n_tok * a.Hq) return;
  const int row = (int)(idx / a.Hq), h = (int)(idx % a.Hq);
  const T *o = (const T *)a.o + (int64_t)row * a.Hq * a.hd + h * a.hd;
  const T *d = (const T *)a.dout + (int64_t)row * a.Hq * a.hd + h * a.hd;
  float s = 0.f;
  for (int c = lane; c < a.hd; c += 64) s += ldf(o + c) * ldf(d + c);
#pragma unroll
  for (int w = 32; w > 0; w >>= 1) s += __shfl_xor(s, w, 64);
  if (lane == 0) a.delta[(int64_t)h * a.n_tok + row] = s;
}

// dQ rows: dq = scale * sum_j P_j (dO.V_j - delta) K_j
template <typename T>
__global__ __launch_bounds__(256) void attn_dq_simple_kernel(AttnBwdArgs a) {
  __shared__ float Ks[kKv][kMaxHd + 1];
  __shared__ float Vs[kKv][kMaxHd + 1];
  __shared__ int range[2];
  const int hd = a.hd, qd = hd / 4;
  const int ld = (a.Hq + 2 * a.Hkv) * hd;
  const int h = blockIdx.y, g = (h * a.Hkv) / a.Hq;
  const int row0 = blockIdx.x * kRows;
  const int rl = threadIdx.x >> 2, part = threadIdx.x & 3;
  const int row = row0 + rl;
  const bool valid = row < a.n_tok;
  const T *qkv = (const T *)a.qkv;
  int start = 0;
  float lse = 0.f, delta = 0.f;
  if (valid) {
    start = seg_start(a, row);
    lse = a.lse[(int64_t)h * a.n_tok + row];
    delta = a.delta[(int64_t)h * a.n_tok + row];
  }
  if (threadIdx.x == 0) {
    range[0] = seg_start(a, row0);
    range[1] = min(row0 + kRows, a.n_tok) - 1;
  }
  float q[kMaxHd / 4], dob[kMaxHd / 4], dq[kMaxHd / 4];
  const T *dout = (const T *)a.dout + (int64_t)row * a.Hq * hd + h * hd + part * qd;
#pragma unroll
  for (int i = 0; i < kMaxHd / 4; ++i) {
    q[i] = (valid && i < qd) ? ldf(qkv + (int64_t)row * ld + h * hd + part * qd + i) : 0.f;
    dob[i] = (valid && i < qd) ? ldf(dout + i) : 0.f;
    dq[i] = 0.f;
  }
  __syncthreads();
  const int kv_lo = range[0], kv_hi = range[1];
  for (int k0 = kv_lo; k0 <= kv_hi; k0 += kKv) {
    for (int e = threadIdx.x; e < kKv * hd; e += 256) {
      int r = e / hd, c = e % hd, kr = k0 + r;
      float kv = 0.f, vv = 0.f;
      if (kr <= kv_hi) {
        kv = ldf(qkv + (int64_t)kr * ld + (a.Hq + g) * hd + c);
        vv = ldf(qkv + (int64_t)kr * ld + (a.Hq + a.Hkv + g) * hd + c);
      }
      Ks[r][c] = kv;
      Vs[r][c] = vv;
    }
    __syncthreads();
    for (int j = 0; j < kKv; ++j) {
      const int key = k0 + j;
      float s = 0.f, dp = 0.f;
#pragma unroll
      for (int i = 0; i < kMaxHd / 4; ++i)
        if (i < qd) { s += q[i] * Ks[j][part * qd + i]; dp += dob[i] * Vs[j][part * qd + i]; }
      s = quad_sum(s);
      dp = quad_sum(dp);
      if (!valid || key < start || key > row) continue;
      const float p = __expf(s * a.scale - lse);
      const float ds = p * (dp - delta) * a.scale;
#pragma unroll
      for (int i = 0; i < kMaxHd / 4; ++i)
        if (i < qd) dq[i] += ds * Ks[j][part * qd + i];
    }
    __syncthreads();
  }
  if (!valid) return;
  T *out = (T *)a.dqkv + (int64_t)row * ld + h * hd + part * qd;
#pragma unroll
  for (int i = 0; i < kMaxHd / 4; ++i)
    if (i < qd) stf(out + i, dq[i]);
}

// dK, dV rows of kv head g: sum over the query heads of the group and the
// queries of the same segment at or after the key.
template <typename T>
__global__ __launch_bounds__(256) void attn_dkv_simple_kernel(AttnBwdArgs a) {
  __shared__ float Qs[kKv][kMaxHd + 1];
  __shared__ float Ds[kKv][kMaxHd + 1];
  __shared__ float Ls[kKv], Dl[kKv];
  __shared__ int range[2];
  const int hd = a.hd, qd = hd / 4;
  const int ld = (a.Hq + 2 * a.Hkv) * hd;
  const int g = blockIdx.y;
  const int row0 = blockIdx.x * kRows;
  const int rl = threadIdx.x >> 2, part = threadIdx.x & 3;
  const int row = row0 + rl;           // the key row
  const bool valid = row < a.n_tok;
  const T *qkv = (const T *)a.qkv;
  int end = 0;
  if (valid) end = seg_end(a, row);
  if (threadIdx.x == 0) {
    const int last = min(row0 + kRows, a.n_tok) - 1;
    range[0] = row0;
    range[1] = seg_end(a, last) - 1;
  }
  float k[kMaxHd / 4], v[kMaxHd / 4], dk[kMaxHd / 4], dv[kMaxHd / 4];
#pragma unroll
  for (int i = 0; i < kMaxHd / 4; ++i) {
    k[i] = (valid && i < qd) ? ldf(qkv + (int64_t)row * ld + (a.Hq + g) * hd + part * qd + i) : 0.f;
    v[i] = (valid && i < qd) ? ldf(qkv + (int64_t)row * ld + (a.Hq + a.Hkv + g) * hd + part * qd + i) : 0.f;
    dk[i] = 0.f;
    dv[i] = 0.f;
  }
  __syncthreads();
  const int q_lo = range[0], q_hi = range[1];
  const int group = a.Hq / a.Hkv;
  for (int hh = 0; hh < group; ++hh) {
    const int h = g * group + hh;
    for (int q0 = q_lo; q0 <= q_hi; q0 += kKv) {
      for (int e = threadIdx.x; e < kKv * hd; e += 256) {
        int r = e / hd, c = e % hd, qr = q0 + r;
        float qv = 0.f, dv_ = 0.f;
        if (qr <= q_hi) {
          qv = ldf(qkv + (int64_t)qr * ld + h * hd + c);
          dv_ = ldf((const T *)a.dout + (int64_t)qr * a.Hq * hd + h * hd + c);
        }
        Qs[r][c] = qv;
        Ds[r][c] = dv_;
      }
      if (threadIdx.x < kKv) {
        int qr = q0 + threadIdx.x;
        Ls[threadIdx.x] = qr <= q_hi ? a.lse[(int64_t)h * a.n_tok + qr] : 0.f;
        Dl[threadIdx.x] = qr <= q_hi ? a.delta[(int64_t)h * a.n_tok + qr] : 0.f;
      }
      __syncthreads();
      for (int j = 0; j < kKv; ++j) {
        const int qrow = q0 + j;
        float s = 0.f, dp = 0.f;
#pragma unroll
        for (int i = 0; i < kMaxHd / 4; ++i)
          if (i < qd) { s += k[i] * Qs[j][part * qd + i]; dp += v[i] * Ds[j][part * qd + i]; }
        s = quad_sum(s);
        dp = quad_sum(dp);
        if (!valid || qrow < row || qrow >= end) continue;
        const float p = __expf(s * a.scale - Ls[j]);
        const float ds = p * (dp - Dl[j]) * a.scale;
#pragma unroll
        for (int i = 0; i < kMaxHd / 4; ++i)
          if (i < qd) {
            dv[i] += p * Ds[j][part * qd + i];
            dk[i] += ds * Qs[j][part * qd + i];
          }
      }
      __syncthreads();
    }
  }
  if (!valid) return;
  T *base = (T *)a.dqkv + (int64_t)row * ld;
#pragma unroll
  for (int i = 0; i < kMaxHd / 4; ++i)
    if (i < qd) {
      stf(base + (a.Hq + g) * hd + part * qd + i, dk[i]);
      stf(base + (a.Hq + a.Hkv + g) * hd + part * qd + i, dv[i]);
    }
}

}  // namespace

template <typename T>
int attn_fwd(const AttnArgs &a, hipStream_t s) {
  if (a.n_tok <= 0) return AJ_OK;
  if (a.hd > kMaxHd || a.hd % 8) return fail(AJ_ERR_UNSUPPORTED, "attention: head_dim %d", a.hd);
  if (sizeof(T) == 2 && attn_mfma_supported(a.hd, a.qkv, a.o, a.o)) return attn_fwd_mfma(a, s);
  dim3 grid((a.n_tok + kRows - 1) / kRows, a.Hq);
  const int tk = timing_begin(s, AJ_KC_ATTN_FWD, 0.0);
  attn_fwd_simple_kernel<T><<<grid, 256, 0, s>>>(a);
  timing_end(s, tk);
  return check_launch("attention forward");
}

template <typename T>
int attn_bwd(const AttnBwdArgs &a, hipStream_t s) {
  if (a.n_tok <= 0) return AJ_OK;
  if (a.hd > kMaxHd || a.hd % 8) return fail(AJ_ERR_UNSUPPORTED, "attention: head_dim %d", a.hd);
  // the matrix-core forward saves its log-sum-exp in log2 units, the plain
  // kernels in natural ones: the backward must take the forward's path
  const bool fwd_mfma = sizeof(T) == 2 && attn_mfma_supported(a.hd, a.qkv, a.o, a.o);
  if (fwd_mfma) {
    if (!attn_mfma_supported(a.hd, a.qkv, a.dout, a.dqkv))
      return fail(AJ_ERR_UNSUPPORTED, "attention backward: d out / d qkv not 16-byte aligned");
    return attn_bwd_mfma(a, s);
  }
  const int64_t nd = (int64_t)a.n_tok * a.Hq;
  const int tk = timing_begin(s, AJ_KC_ATTN_BWD, 0.0);
  attn_delta_kernel<T><<<(unsigned)((nd + 3) / 4), 256, 0, s>>>(a);
  attn_dq_simple_kernel<T><<<dim3((a.n_tok + kRows - 1) / kRows, a.Hq), 256, 0, s>>>(a);
  attn_dkv_simple_kernel<T><<<dim3((a.n_tok + kRows - 1) / kRows, a.Hkv), 256, 0, s>>>(a);
  timing_end(s, tk);
  return check_launch("attention backward");
}

template int attn_fwd<float>(const AttnArgs &, hipStream_t);
template int attn_fwd<bf16_t>(const AttnArgs &, hipStream_t);
template int attn_bwd<float>(const AttnBwdArgs &, hipStream_t);
template int attn_bwd<bf16_t>(const AttnBwdArgs &, hipStream_t);

}  // namespace aj
