// bfloat16 causal GQA attention over packed segments on v_mfma_f32_32x32x16_bf16.
//
// Orientation.  The 32x32 MFMA accumulator gives each lane one COLUMN and 16
// rows.  The forward and the dQ pass compute S^T = K Q^T so that a lane owns
// one query (a column) and holds 32 of the key scores of each 64-key tile: the
// online softmax is per lane plus one exchange with lane^32.  The probabilities
// then feed O^T = V^T P^T directly as the B operand: within one k-step a lane
// half contributes 8 keys, and the A operand (V^T, staged transposed in LDS)
// is read for exactly the same 8 keys, so the k order inside the instruction
// never has to match memory order.  The dK/dV pass computes S = Q K^T so that a
// lane owns one KEY, and accumulates dV^T = dO^T P and dK^T = Q^T dS the same
// way.  Segment masking: a query row attends to [segment start, itself].
//
// Workgroups: 256 threads, 4 waves of 32 query (or key) rows each.  Query
// tiles are visited from the end of the pack (the longest rows first) and the
// head index varies fastest, so the query heads that share a key/value head run
// side by side on one XCD (ids are dealt round-robin over 8 XCDs) and share its L2.
#include "ops.h"

namespace aj {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr int kKT = 64;       // keys per staged tile (forward, dQ)
constexpr int kQT = 64;       // queries per staged tile (dK/dV)

AJ_DEV f32x16_t mfma(bf16x8_t a, bf16x8_t b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

AJ_DEV uint32_t pack2(float lo, float hi) {
  return (uint32_t)f2bf(lo) | ((uint32_t)f2bf(hi) << 16);
}

// 8 accumulator values r0..r0+7 -> one bf16x8 operand
AJ_DEV bf16x8_t pack8(const f32x16_t &v, int r0) {
  u32x4_t u{pack2(v[r0], v[r0 + 1]), pack2(v[r0 + 2], v[r0 + 3]), pack2(v[r0 + 4], v[r0 + 5]),
            pack2(v[r0 + 6], v[r0 + 7])};
  return __builtin_bit_cast(bf16x8_t, u);
}

// Two 4-element runs from a transposed LDS row: [p, p+4) and [p+8, p+12).
AJ_DEV bf16x8_t ld_split(const uint16_t *p) {
  u32x2_t a = *(const u32x2_t *)p, b = *(const u32x2_t *)(p + 8);
  u32x4_t u{a[0], a[1], b[0], b[1]};
  return __builtin_bit_cast(bf16x8_t, u);
}

AJ_DEV int seg_of(const int32_t *cu, int n_seg, int base, int row) {
  int lo = 0, hi = n_seg - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (cu[mid] - base <= row) lo = mid; else hi = mid - 1;
  }
  return lo;
}
template <typename A> AJ_DEV int seg_start(const A &a, int row) {
  const int v = a.cu_seqlens[seg_of(a.cu_seqlens, a.n_seg, a.base, row)] - a.base;
  return v < 0 ? 0 : (v > row ? row : v);
}
template <typename A> AJ_DEV int seg_end(const A &a, int row) {
  const int v = a.cu_seqlens[seg_of(a.cu_seqlens, a.n_seg, a.base, row) + 1] - a.base;
  return v <= row ? row + 1 : (v > a.n_tok ? a.n_tok : v);
}

AJ_DEV int xcd_remap(int wg, int nwg) {
  const int per = nwg / 8, rem = nwg % 8, xcd = wg % 8, idx = wg / 8;
  return xcd * per + (xcd < rem ? xcd : rem) + idx;
}

AJ_DEV float wave_min_f(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fminf(v, __shfl_xor(v, o, 64));
  return v;
}

// rows [r0, r0+R) x HD of a strided bf16 matrix -> LDS [R][LDR], zero past `rows`
template <int R, int HD, int LDR>
AJ_DEV void stage_rows(uint16_t *lds, const bf16_t *src, int64_t ld, int r0, int rows) {
  constexpr int kVec = R * HD / 8;
  for (int v = threadIdx.x; v < kVec; v += 256) {
    const int r = v / (HD / 8), c = (v % (HD / 8)) * 8;
    u32x4_t x{0, 0, 0, 0};
    if (r0 + r < rows) x = *(const u32x4_t *)(src + (int64_t)(r0 + r) * ld + c);
    *(u32x4_t *)(lds + r * LDR + c) = x;
  }
}

// rows [r0, r0+R) x HD -> LDS transposed [HD][LDT] (LDT >= R), zero past `rows`
template <int R, int HD, int LDT>
AJ_DEV void stage_rows_t(uint16_t *lds, const bf16_t *src, int64_t ld, int r0, int rows) {
  constexpr int kSlots = (R / 4) * (HD / 8);
  for (int s = threadIdx.x; s < kSlots; s += 256) {
    const int cb = s % (HD / 8), rb = s / (HD / 8);
    u32x4_t x[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int r = r0 + rb * 4 + k;
      x[k] = r < rows ? *(const u32x4_t *)(src + (int64_t)r * ld + cb * 8) : u32x4_t{0, 0, 0, 0};
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int w = e >> 1, sh = (e & 1) * 16;
      const uint32_t a0 = (x[0][w] >> sh) & 0xffffu, a1 = (x[1][w] >> sh) & 0xffffu;
      const uint32_t a2 = (x[2][w] >> sh) & 0xffffu, a3 = (x[3][w] >> sh) & 0xffffu;
      *(u32x2_t *)(lds + (cb * 8 + e) * LDT + rb * 4) = u32x2_t{a0 | (a1 << 16), a2 | (a3 << 16)};
    }
  }
}

// ------------------------------------------------------------------ forward
template <int HD>
__global__ __launch_bounds__(256, 2) void attn_fwd_mfma_kernel(AttnArgs a, int n_qt) {
  constexpr int LDK = HD + 8, LDV = kKT + 8, KS = HD / 16, DT = HD / 32;
  __shared__ __attribute__((aligned(16))) uint16_t Ks[kKT * LDK];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[HD * LDV];
  __shared__ int rng[2];
  const int t = xcd_remap(blockIdx.x, gridDim.x);
  const int h = t % a.Hq, qt = n_qt - 1 - t / a.Hq;
  const int g = (h * a.Hkv) / a.Hq;
  const int ld = (a.Hq + 2 * a.Hkv) * HD;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, hl = lane >> 5, lq = lane & 31;
  const int q0 = qt * 128;
  const int q = q0 + 32 * w + lq;
  const bool qv = q < a.n_tok;
  const int qs = qv ? seg_start(a, q) : a.n_tok;
  const bf16_t *qkv = (const bf16_t *)a.qkv;
  if (threadIdx.x == 0) {
    rng[0] = seg_start(a, q0);
    rng[1] = min(q0 + 127, a.n_tok - 1);
  }
  bf16x8_t qf[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    u32x4_t x{0, 0, 0, 0};
    if (qv) x = *(const u32x4_t *)(qkv + (int64_t)q * ld + h * HD + 16 * kk + 8 * hl);
    qf[kk] = __builtin_bit_cast(bf16x8_t, x);
  }
  f32x16_t o[DT];
#pragma unroll
  for (int i = 0; i < DT; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[i][r] = 0.f;
  float m = -INFINITY, lsum = 0.f;
  const float c = a.scale * kLog2e;
  const int w_lo = (int)wave_min_f((float)qs);          // earliest key any row of the wave reads
  const int w_hi = min(q0 + 32 * w + 31, a.n_tok - 1);   // latest query row of the wave
  __syncthreads();
  const int kv_lo = rng[0], kv_hi = rng[1];
  const bf16_t *kbase = qkv + (a.Hq + g) * HD, *vbase = qkv + (a.Hq + a.Hkv + g) * HD;
  for (int k0 = kv_lo; k0 <= kv_hi; k0 += kKT) {
    stage_rows<kKT, HD, LDK>(Ks, kbase, ld, k0, kv_hi + 1);
    stage_rows_t<kKT, HD, LDV>(Vt, vbase, ld, k0, kv_hi + 1);
    __syncthreads();
    if (k0 <= w_hi && k0 + kKT - 1 >= w_lo) {
      f32x16_t s[2];
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int r = 0; r < 16; ++r) s[tt][r] = 0.f;
#pragma unroll
      for (int kk = 0; kk < KS; ++kk)
#pragma unroll
        for (int tt = 0; tt < 2; ++tt) {
          bf16x8_t kf = *(const bf16x8_t *)(Ks + (32 * tt + lq) * LDK + 16 * kk + 8 * hl);
          s[tt] = mfma(kf, qf[kk], s[tt]);
        }
      float mx = -INFINITY;
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int kv = k0 + 32 * tt + 8 * (r >> 2) + 4 * hl + (r & 3);
          const bool ok = kv >= qs && kv <= q;
          s[tt][r] = ok ? s[tt][r] * c : -INFINITY;
          mx = fmaxf(mx, s[tt][r]);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float mn = fmaxf(m, mx);
      const float alpha = mn == -INFINITY ? 1.f : exp2f(m - mn);
      float ls = 0.f;
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float p = mn == -INFINITY ? 0.f : exp2f(s[tt][r] - mn);
          s[tt][r] = p;
          ls += p;
        }
      ls += __shfl_xor(ls, 32, 64);
      lsum = lsum * alpha + ls;
      m = mn;
#pragma unroll
      for (int i = 0; i < DT; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[i][r] *= alpha;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const bf16x8_t pf = pack8(s[j >> 1], 8 * (j & 1));
        const int kvo = 32 * (j >> 1) + 16 * (j & 1) + 4 * hl;
#pragma unroll
        for (int i = 0; i < DT; ++i) {
          const bf16x8_t vf = ld_split(Vt + (32 * i + lq) * LDV + kvo);
          o[i] = mfma(vf, pf, o[i]);
        }
      }
    }
    __syncthreads();
  }
  if (!qv) return;
  const float inv = 1.f / lsum;
  bf16_t *out = (bf16_t *)a.o + (int64_t)q * a.Hq * HD + h * HD;
#pragma unroll
  for (int i = 0; i < DT; ++i)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const int d = 32 * i + 8 * r4 + 4 * hl;
      *(u32x2_t *)(out + d) = u32x2_t{pack2(o[i][4 * r4] * inv, o[i][4 * r4 + 1] * inv),
                                      pack2(o[i][4 * r4 + 2] * inv, o[i][4 * r4 + 3] * inv)};
    }
  if (hl == 0) a.lse[(int64_t)h * a.n_tok + q] = (m + log2f(lsum)) / kLog2e;
}

// ------------------------------------------------------------------ dQ
template <int HD>
__global__ __launch_bounds__(256, 2) void attn_dq_mfma_kernel(AttnBwdArgs a, int n_qt) {
  constexpr int LDK = HD + 8, LDT = kKT + 8, KS = HD / 16, DT = HD / 32;
  __shared__ __attribute__((aligned(16))) uint16_t Ks[kKT * LDK];
  __shared__ __attribute__((aligned(16))) uint16_t Vs[kKT * LDK];
  __shared__ __attribute__((aligned(16))) uint16_t Kt[HD * LDT];
  __shared__ int rng[2];
  const int t = xcd_remap(blockIdx.x, gridDim.x);
  const int h = t % a.Hq, qt = n_qt - 1 - t / a.Hq;
  const int g = (h * a.Hkv) / a.Hq;
  const int ld = (a.Hq + 2 * a.Hkv) * HD;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, hl = lane >> 5, lq = lane & 31;
  const int q0 = qt * 128;
  const int q = q0 + 32 * w + lq;
  const bool qv = q < a.n_tok;
  const int qs = qv ? seg_start(a, q) : a.n_tok;
  const bf16_t *qkv = (const bf16_t *)a.qkv;
  const bf16_t *dout = (const bf16_t *)a.dout;
  if (threadIdx.x == 0) {
    rng[0] = seg_start(a, q0);
    rng[1] = min(q0 + 127, a.n_tok - 1);
  }
  bf16x8_t qf[KS], df[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    u32x4_t x{0, 0, 0, 0}, y{0, 0, 0, 0};
    if (qv) {
      x = *(const u32x4_t *)(qkv + (int64_t)q * ld + h * HD + 16 * kk + 8 * hl);
      y = *(const u32x4_t *)(dout + (int64_t)q * a.Hq * HD + h * HD + 16 * kk + 8 * hl);
    }
    qf[kk] = __builtin_bit_cast(bf16x8_t, x);
    df[kk] = __builtin_bit_cast(bf16x8_t, y);
  }
  const float lse2 = qv ? a.lse[(int64_t)h * a.n_tok + q] * kLog2e : 0.f;
  const float dlt = qv ? a.delta[(int64_t)h * a.n_tok + q] : 0.f;
  f32x16_t acc[DT];
#pragma unroll
  for (int i = 0; i < DT; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[i][r] = 0.f;
  const float c = a.scale * kLog2e;
  const int w_lo = (int)wave_min_f((float)qs);
  const int w_hi = min(q0 + 32 * w + 31, a.n_tok - 1);
  __syncthreads();
  const int kv_lo = rng[0], kv_hi = rng[1];
  const bf16_t *kbase = qkv + (a.Hq + g) * HD, *vbase = qkv + (a.Hq + a.Hkv + g) * HD;
  for (int k0 = kv_lo; k0 <= kv_hi; k0 += kKT) {
    stage_rows<kKT, HD, LDK>(Ks, kbase, ld, k0, kv_hi + 1);
    stage_rows<kKT, HD, LDK>(Vs, vbase, ld, k0, kv_hi + 1);
    stage_rows_t<kKT, HD, LDT>(Kt, kbase, ld, k0, kv_hi + 1);
    __syncthreads();
    if (k0 <= w_hi && k0 + kKT - 1 >= w_lo) {
      f32x16_t s[2], dp[2];
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int r = 0; r < 16; ++r) { s[tt][r] = 0.f; dp[tt][r] = 0.f; }
#pragma unroll
      for (int kk = 0; kk < KS; ++kk)
#pragma unroll
        for (int tt = 0; tt < 2; ++tt) {
          const int off = (32 * tt + lq) * LDK + 16 * kk + 8 * hl;
          s[tt] = mfma(*(const bf16x8_t *)(Ks + off), qf[kk], s[tt]);
          dp[tt] = mfma(*(const bf16x8_t *)(Vs + off), df[kk], dp[tt]);
        }
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int kv = k0 + 32 * tt + 8 * (r >> 2) + 4 * hl + (r & 3);
          const bool ok = kv >= qs && kv <= q;
          const float p = ok ? exp2f(s[tt][r] * c - lse2) : 0.f;
          s[tt][r] = p * (dp[tt][r] - dlt);
        }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const bf16x8_t sf = pack8(s[j >> 1], 8 * (j & 1));
        const int kvo = 32 * (j >> 1) + 16 * (j & 1) + 4 * hl;
#pragma unroll
        for (int i = 0; i < DT; ++i)
          acc[i] = mfma(ld_split(Kt + (32 * i + lq) * LDT + kvo), sf, acc[i]);
      }
    }
    __syncthreads();
  }
  if (!qv) return;
  bf16_t *out = (bf16_t *)a.dqkv + (int64_t)q * ld + h * HD;
#pragma unroll
  for (int i = 0; i < DT; ++i)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const int d = 32 * i + 8 * r4 + 4 * hl;
      *(u32x2_t *)(out + d) = u32x2_t{pack2(acc[i][4 * r4] * a.scale, acc[i][4 * r4 + 1] * a.scale),
                                      pack2(acc[i][4 * r4 + 2] * a.scale, acc[i][4 * r4 + 3] * a.scale)};
    }
}

// ------------------------------------------------------------------ dK, dV
template <int HD>
__global__ __launch_bounds__(256) void attn_dkv_mfma_kernel(AttnBwdArgs a, int n_kt) {
  constexpr int LDQ = HD + 8, LDT = kQT + 8, KS = HD / 16, DT = HD / 32;
  __shared__ __attribute__((aligned(16))) uint16_t Qs[kQT * LDQ];
  __shared__ __attribute__((aligned(16))) uint16_t Ds[kQT * LDQ];
  __shared__ __attribute__((aligned(16))) uint16_t Qt[HD * LDT];
  __shared__ __attribute__((aligned(16))) uint16_t Dt[HD * LDT];
  __shared__ float Ls[kQT], Dl[kQT];
  __shared__ int rng[1];
  const int t = xcd_remap(blockIdx.x, gridDim.x);
  const int g = t % a.Hkv, kt = t / a.Hkv;   // early keys of a segment see the most queries
  const int ld = (a.Hq + 2 * a.Hkv) * HD;
  const int ldo = a.Hq * HD;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, hl = lane >> 5, lq = lane & 31;
  const int k0 = kt * 128;
  const int kv = k0 + 32 * w + lq;            // the key row this lane owns
  const bool kvv = kv < a.n_tok;
  const int ke = kvv ? seg_end(a, kv) : 0;    // queries of the key: [kv, ke)
  const bf16_t *qkv = (const bf16_t *)a.qkv;
  const bf16_t *dout = (const bf16_t *)a.dout;
  if (threadIdx.x == 0) rng[0] = seg_end(a, min(k0 + 127, a.n_tok - 1));
  bf16x8_t kf[KS], vf[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    u32x4_t x{0, 0, 0, 0}, y{0, 0, 0, 0};
    if (kvv) {
      x = *(const u32x4_t *)(qkv + (int64_t)kv * ld + (a.Hq + g) * HD + 16 * kk + 8 * hl);
      y = *(const u32x4_t *)(qkv + (int64_t)kv * ld + (a.Hq + a.Hkv + g) * HD + 16 * kk + 8 * hl);
    }
    kf[kk] = __builtin_bit_cast(bf16x8_t, x);
    vf[kk] = __builtin_bit_cast(bf16x8_t, y);
  }
  f32x16_t dk[DT], dv[DT];
#pragma unroll
  for (int i = 0; i < DT; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) { dk[i][r] = 0.f; dv[i][r] = 0.f; }
  const float c = a.scale * kLog2e;
  const int w_lo = min(k0 + 32 * w, a.n_tok);               // first query any key of the wave sees
  const int w_hi = (int)-wave_min_f(kvv ? -(float)(ke - 1) : 1.f);   // last one
  __syncthreads();
  const int q_hi = rng[0];    // queries [k0, q_hi)
  const int group = a.Hq / a.Hkv;
  for (int hh = 0; hh < group; ++hh) {
    const int h = g * group + hh;
    for (int qb = k0; qb < q_hi; qb += kQT) {
      stage_rows<kQT, HD, LDQ>(Qs, qkv + h * HD, ld, qb, q_hi);
      stage_rows<kQT, HD, LDQ>(Ds, dout + h * HD, ldo, qb, q_hi);
      stage_rows_t<kQT, HD, LDT>(Qt, qkv + h * HD, ld, qb, q_hi);
      stage_rows_t<kQT, HD, LDT>(Dt, dout + h * HD, ldo, qb, q_hi);
      if (threadIdx.x < kQT) {
        const int qr = qb + threadIdx.x;
        Ls[threadIdx.x] = qr < q_hi ? a.lse[(int64_t)h * a.n_tok + qr] * kLog2e : 0.f;
        Dl[threadIdx.x] = qr < q_hi ? a.delta[(int64_t)h * a.n_tok + qr] : 0.f;
      }
      __syncthreads();
      if (qb + kQT - 1 >= w_lo && qb <= w_hi) {
        // S = Q K^T, dP = dO V^T: [64 queries x 32 keys] as two row tiles
        f32x16_t s[2], dp[2];
#pragma unroll
        for (int tt = 0; tt < 2; ++tt)
#pragma unroll
          for (int r = 0; r < 16; ++r) { s[tt][r] = 0.f; dp[tt][r] = 0.f; }
#pragma unroll
        for (int kk = 0; kk < KS; ++kk)
#pragma unroll
          for (int tt = 0; tt < 2; ++tt) {
            const int off = (32 * tt + lq) * LDQ + 16 * kk + 8 * hl;
            s[tt] = mfma(*(const bf16x8_t *)(Qs + off), kf[kk], s[tt]);
            dp[tt] = mfma(*(const bf16x8_t *)(Ds + off), vf[kk], dp[tt]);
          }
#pragma unroll
        for (int tt = 0; tt < 2; ++tt)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int ql = 32 * tt + 8 * (r >> 2) + 4 * hl + (r & 3);
            const int qr = qb + ql;
            const bool ok = kvv && qr >= kv && qr < ke;
            const float p = ok ? exp2f(s[tt][r] * c - Ls[ql]) : 0.f;
            s[tt][r] = p;
            dp[tt][r] = p * (dp[tt][r] - Dl[ql]);
          }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const bf16x8_t pf = pack8(s[j >> 1], 8 * (j & 1));
          const bf16x8_t sf = pack8(dp[j >> 1], 8 * (j & 1));
          const int qo = 32 * (j >> 1) + 16 * (j & 1) + 4 * hl;
#pragma unroll
          for (int i = 0; i < DT; ++i) {
            dv[i] = mfma(ld_split(Dt + (32 * i + lq) * LDT + qo), pf, dv[i]);
            dk[i] = mfma(ld_split(Qt + (32 * i + lq) * LDT + qo), sf, dk[i]);
          }
        }
      }
      __syncthreads();
    }
  }
  if (!kvv) return;
  bf16_t *base = (bf16_t *)a.dqkv + (int64_t)kv * ld;
#pragma unroll
  for (int i = 0; i < DT; ++i)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const int d = 32 * i + 8 * r4 + 4 * hl;
      *(u32x2_t *)(base + (a.Hq + g) * HD + d) =
          u32x2_t{pack2(dk[i][4 * r4] * a.scale, dk[i][4 * r4 + 1] * a.scale),
                  pack2(dk[i][4 * r4 + 2] * a.scale, dk[i][4 * r4 + 3] * a.scale)};
      *(u32x2_t *)(base + (a.Hq + a.Hkv + g) * HD + d) =
          u32x2_t{pack2(dv[i][4 * r4], dv[i][4 * r4 + 1]), pack2(dv[i][4 * r4 + 2], dv[i][4 * r4 + 3])};
    }
}

__global__ __launch_bounds__(256) void attn_delta_bf16_kernel(AttnBwdArgs a) {
  const int64_t idx = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (idx >= (int64_t)a.n_tok * a.Hq) return;
  const int row = (int)(idx / a.Hq), h = (int)(idx % a.Hq);
  const bf16_t *o = (const bf16_t *)a.o + (int64_t)row * a.Hq * a.hd + h * a.hd;
  const bf16_t *d = (const bf16_t *)a.dout + (int64_t)row * a.Hq * a.hd + h * a.hd;
  float s = 0.f;
  for (int c = lane; c < a.hd; c += 64) s += bf2f(o[c]) * bf2f(d[c]);
#pragma unroll
  for (int w = 32; w > 0; w >>= 1) s += __shfl_xor(s, w, 64);
  if (lane == 0) a.delta[(int64_t)h * a.n_tok + row] = s;
}

bool aligned16(const void *p) { return ((uintptr_t)p & 15) == 0; }

}  // namespace

bool attn_mfma_supported(int hd, const void *p0, const void *p1, const void *p2) {
  return (hd == 64 || hd == 128) && aligned16(p0) && aligned16(p1) && aligned16(p2);
}

int attn_fwd_mfma(const AttnArgs &a, hipStream_t s) {
  const int n_qt = (a.n_tok + 127) / 128;
  const unsigned grid = (unsigned)n_qt * a.Hq;
  const int tk = timing_begin(s, AJ_KC_ATTN_FWD, 0.0);
  if (a.hd == 128) attn_fwd_mfma_kernel<128><<<grid, 256, 0, s>>>(a, n_qt);
  else attn_fwd_mfma_kernel<64><<<grid, 256, 0, s>>>(a, n_qt);
  timing_end(s, tk);
  return check_launch("attention forward (mfma)");
}

int attn_bwd_mfma(const AttnBwdArgs &a, hipStream_t s) {
  const int n_qt = (a.n_tok + 127) / 128;
  const int64_t nd = (int64_t)a.n_tok * a.Hq;
  const int tk = timing_begin(s, AJ_KC_ATTN_BWD, 0.0);
  attn_delta_bf16_kernel<<<(unsigned)((nd + 3) / 4), 256, 0, s>>>(a);
  if (a.hd == 128) {
    attn_dq_mfma_kernel<128><<<(unsigned)n_qt * a.Hq, 256, 0, s>>>(a, n_qt);
    attn_dkv_mfma_kernel<128><<<(unsigned)n_qt * a.Hkv, 256, 0, s>>>(a, n_qt);
  } else {
    attn_dq_mfma_kernel<64><<<(unsigned)n_qt * a.Hq, 256, 0, s>>>(a, n_qt);
    attn_dkv_mfma_kernel<64><<<(unsigned)n_qt * a.Hkv, 256, 0, s>>>(a, n_qt);
  }
  timing_end(s, tk);
  return check_launch("attention backward (mfma)");
}

}  // namespace aj
