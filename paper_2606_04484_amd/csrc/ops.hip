// Row-wise and elementwise kernels of the decoder block and the LM head.
// All of them are HBM-bound; rows are handled one wavefront (64 lanes) each.
#include "ops.h"

namespace aj {
namespace {

constexpr int kRowsPerBlock = 4;   // 4 waves of 64 lanes

AJ_DEV float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// ---------------------------------------------------------------- RMSNorm
// One wave per row; lane handles columns 8*(lane + 64*v) + e, v < NV, e < 8,
// so every access is a 16-byte (bf16) or 32-byte (float) vector.  NV is the
// smallest instantiated value with 512*NV >= d; the row stays in registers
// between the reduction and the output pass.
typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));

AJ_DEV void load8(const float *p, float (&v)[8]) {
  const float4 a = *(const float4 *)p, b = *(const float4 *)(p + 4);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
AJ_DEV void load8(const bf16_t *p, float (&v)[8]) {
  const u32x4v u = *(const u32x4v *)p;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    v[2 * k] = __uint_as_float(u[k] << 16);
    v[2 * k + 1] = __uint_as_float(u[k] & 0xffff0000u);
  }
}
AJ_DEV void store8(float *p, const float (&v)[8]) {
  *(float4 *)p = make_float4(v[0], v[1], v[2], v[3]);
  *(float4 *)(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
}
AJ_DEV void store8(bf16_t *p, const float (&v)[8]) {
  u32x4v u;
#pragma unroll
  for (int k = 0; k < 4; ++k) u[k] = f2bf2(v[2 * k], v[2 * k + 1]);
  *(u32x4v *)p = u;
}

// out[i] = x[r] * rstd * g, r = rows ? rows[i] + row_shift : i
template <typename T, int NV>
__global__ __launch_bounds__(256) void rmsnorm_fwd_kernel(const T *x, const T *g, int n, int d,
                                                          float eps, const int32_t *rows,
                                                          int row_shift, T *out, float *rstd) {
  const int i = blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (i >= n) return;
  const int64_t r = rows ? (int64_t)rows[i] + row_shift : i;
  const T *xr = x + r * d;
  float xv[NV][8];
  float ss = 0.f;
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    const int c = 8 * (lane + 64 * v);
    if (c < d) {
      load8(xr + c, xv[v]);
#pragma unroll
      for (int e = 0; e < 8; ++e) ss += xv[v][e] * xv[v][e];
    }
  }
  ss = wave_sum(ss);
  const float rs = 1.0f / sqrtf(ss / d + eps);
  if (lane == 0 && rstd) rstd[i] = rs;
  T *o = out + (int64_t)i * d;
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    const int c = 8 * (lane + 64 * v);
    if (c < d) {
      float gv[8], y[8];
      load8(g + c, gv);
#pragma unroll
      for (int e = 0; e < 8; ++e) y[e] = xv[v][e] * rs * gv[e];
      store8(o + c, y);
    }
  }
}

// dx = add + rstd * (g*dy - x * rstd^2 * mean(g*dy*x)).
// Input row i reads x row r (gather as in the forward); output row i goes to
// out row r when scatter is set, else row i.  Each wave walks a fixed set of
// rows and keeps its share of dg = sum_rows dy*x*rstd in registers; the four
// waves of a block then add theirs in a fixed order, and the per-block rows
// are summed in order by col_reduce_kernel.
constexpr int kBwdBlocks = 1024;
template <typename T, int NV>
__global__ __launch_bounds__(256) void rmsnorm_bwd_kernel(
    const float *dy, const T *x, const float *rstd, const T *g, int n, int d,
    const int32_t *rows, int row_shift, int scatter, const float *add, float *dx, T *dx_t,
    float *dg_part) {
  __shared__ float red[NV * 512];
  const int w = threadIdx.x >> 6;
  const int gw = blockIdx.x * kRowsPerBlock + w;
  const int nw = gridDim.x * kRowsPerBlock;
  const int lane = threadIdx.x & 63;
  float acc[NV][8];
#pragma unroll
  for (int v = 0; v < NV; ++v)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[v][e] = 0.f;
  for (int i = gw; i < n; i += nw) {
    const int64_t r = rows ? (int64_t)rows[i] + row_shift : i;
    const int64_t o = scatter ? r : i;
    const float *dyr = dy + (int64_t)i * d;
    const T *xr = x + r * d;
    const float rs = rstd[i];
    float dv[NV][8], xv[NV][8];
    float dot = 0.f;
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int c = 8 * (lane + 64 * v);
      if (c < d) {
        float gv[8];
        load8(dyr + c, dv[v]);
        load8(xr + c, xv[v]);
        load8(g + c, gv);
#pragma unroll
        for (int e = 0; e < 8; ++e) dot += gv[e] * dv[v][e] * xv[v][e];
      }
    }
    dot = wave_sum(dot) / d;
    const float k2 = rs * rs * dot;
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int c = 8 * (lane + 64 * v);
      if (c < d) {
        float y[8], gv[8];
        load8(g + c, gv);
        if (add) load8(add + o * d + c, y);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float val = rs * (gv[e] * dv[v][e] - xv[v][e] * k2);
          y[e] = add ? y[e] + val : val;
          acc[v][e] += dv[v][e] * xv[v][e] * rs;
        }
        if (dx) store8(dx + o * d + c, y);
        if (dx_t) store8(dx_t + o * d + c, y);
      }
    }
  }
  // fixed-order combine of the four waves' dg shares
  for (int ww = 0; ww < kRowsPerBlock; ++ww) {
    if (w == ww) {
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const int c = 8 * (lane + 64 * v);
        if (c < d)
#pragma unroll
          for (int e = 0; e < 8; ++e) red[c + e] = (ww == 0 ? 0.f : red[c + e]) + acc[v][e];
      }
    }
    __syncthreads();
  }
  for (int c = threadIdx.x; c < d; c += blockDim.x) dg_part[(int64_t)blockIdx.x * d + c] = red[c];
}

// out[c] += sum_b part[b][c] in a fixed order (deterministic): a block takes
// 64 columns; thread (phase p, column) sums rows b = p + 4k with four
// independent accumulators (k mod 4), combined in order, then the four
// phases are added in order.  Coalesced 256-byte rows, 16 loads in flight.
__global__ __launch_bounds__(256) void col_reduce_kernel(const float *part, int nb, int d,
                                                         float *out) {
  __shared__ float ph[4][64];
  const int lane = threadIdx.x & 63, p = threadIdx.x >> 6;
  const int c = blockIdx.x * 64 + lane;
  float a[4] = {0.f, 0.f, 0.f, 0.f};
  if (c < d) {
    int b = p;
    for (; b + 12 < nb; b += 16) {
#pragma unroll
      for (int u = 0; u < 4; ++u) a[u] += part[(int64_t)(b + 4 * u) * d + c];
    }
    for (int u = 0; b < nb; b += 4, ++u) a[u & 3] += part[(int64_t)b * d + c];
  }
  ph[p][lane] = (a[0] + a[1]) + (a[2] + a[3]);
  __syncthreads();
  if (p == 0 && c < d) out[c] += ((ph[0][lane] + ph[1][lane]) + ph[2][lane]) + ph[3][lane];
}

// ---------------------------------------------------------------- RoPE
// In place on the q and k heads of qkv [n, (Hq+2Hkv)*hd], 4 rotation pairs
// (i, i + hd/2) per thread.  pos * theta^(-2i/hd) reaches ~1e5 rad, so the
// angle is formed in double precision as a number of turns and reduced to
// its fraction, whose sine and cosine are then taken in single precision
// (|angle| <= pi: error ~2e-7 rad).
AJ_DEV void load4(const float *p, float (&v)[4]) {
  const float4 a = *(const float4 *)p;
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
}
AJ_DEV void load4(const bf16_t *p, float (&v)[4]) {
  const uint2 u = *(const uint2 *)p;
  v[0] = __uint_as_float(u.x << 16); v[1] = __uint_as_float(u.x & 0xffff0000u);
  v[2] = __uint_as_float(u.y << 16); v[3] = __uint_as_float(u.y & 0xffff0000u);
}
AJ_DEV void store4(float *p, const float (&v)[4]) { *(float4 *)p = make_float4(v[0], v[1], v[2], v[3]); }
AJ_DEV void store4(bf16_t *p, const float (&v)[4]) {
  *(uint2 *)p = make_uint2(f2bf2(v[0], v[1]), f2bf2(v[2], v[3]));
}

template <typename T>
__global__ __launch_bounds__(256) void rope_kernel(T *qkv, int n, const int32_t *pos, int n_rot_heads,
                                                   int ld, int hd, double log_theta, int inverse) {
  __shared__ double turns_per_pos[64];      // theta^(-2i/hd) / (2 pi), hd <= 128
  const int half = hd >> 1, q4 = half >> 2;
  if ((int)threadIdx.x < half)
    turns_per_pos[threadIdx.x] =
        exp(-(2.0 * (int)threadIdx.x / hd) * log_theta) * 0.15915494309189535;   // 1 / (2 pi)
  __syncthreads();
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t total = (int64_t)n * n_rot_heads * q4;
  if (idx >= total) return;
  const int i0 = (int)(idx % q4) * 4;
  const int64_t t = idx / q4;
  const int h = (int)(t % n_rot_heads);
  const int row = (int)(t / n_rot_heads);
  T *p = qkv + (int64_t)row * ld + (int64_t)h * hd;
  float x1[4], x2[4], y1[4], y2[4];
  load4(p + i0, x1);
  load4(p + i0 + half, x2);
  const double ps = (double)pos[row];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const double turns = ps * turns_per_pos[i0 + e];
    const float ang = (float)(turns - rint(turns)) * 6.2831853071795865f;
    float sn, cs;
    sincosf(ang, &sn, &cs);
    if (inverse) sn = -sn;
    y1[e] = x1[e] * cs - x2[e] * sn;
    y2[e] = x2[e] * cs + x1[e] * sn;
  }
  store4(p + i0, y1);
  store4(p + i0 + half, y2);
}

// ---------------------------------------------------------------- SwiGLU
// 8 features per thread (d_ff is a multiple of 8): 16-byte bf16 vectors.
template <typename T>
__global__ __launch_bounds__(256) void swiglu_fwd_kernel(const T *gu, int n, int F, T *s) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int F8 = F >> 3;
  if (idx >= (int64_t)n * F8) return;
  const int64_t r = idx / F8, f = (idx % F8) * 8;
  float g[8], u[8], y[8];
  load8(gu + r * 2 * F + f, g);
  load8(gu + r * 2 * F + F + f, u);
#pragma unroll
  for (int e = 0; e < 8; ++e) y[e] = g[e] / (1.f + __expf(-g[e])) * u[e];
  store8(s + r * F + f, y);
}

template <typename TI, typename T>
__global__ __launch_bounds__(256) void swiglu_bwd_kernel(const TI *ds, const T *gu, int n, int F,
                                                         T *dgu) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int F8 = F >> 3;
  if (idx >= (int64_t)n * F8) return;
  const int64_t r = idx / F8, f = (idx % F8) * 8;
  float g[8], u[8], dv[8], dg[8], du[8];
  load8(gu + r * 2 * F + f, g);
  load8(gu + r * 2 * F + F + f, u);
  load8(ds + r * F + f, dv);
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float sg = 1.f / (1.f + __expf(-g[e]));
    dg[e] = dv[e] * u[e] * sg * (1.f + g[e] * (1.f - sg));
    du[e] = dv[e] * g[e] * sg;
  }
  store8(dgu + r * 2 * F + f, dg);
  store8(dgu + r * 2 * F + F + f, du);
}

template <typename T>
__global__ void cast_kernel(const float *in, int64_t n, T *out) {
  const int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 8;
  if (i + 8 <= n) {
    float v[8];
    load8(in + i, v);
    store8(out + i, v);
  } else {
    for (int64_t k = i; k < n; ++k) stf(out + k, in[k]);
  }
}

template <typename T>
__global__ void scale_cast_kernel(const float *in, int64_t n, float scale, T *out, T *lo) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const float v = scale * in[i];
  stf(out + i, v);
  if (lo) stf(lo + i, v - ldf(out + i));
}

__global__ void fill_kernel(float *p, int64_t n, float v) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

// out[i] += sum_s part[s][i], s ascending.
__global__ void splitk_reduce_kernel(const float *part, int S, int64_t n, float *out, int accumulate) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  float v = accumulate ? out[i] : 0.f;
  for (int s = 0; s < S; ++s) v += part[(int64_t)s * n + i];
  out[i] = v;
}

inline unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

// ---------------------------------------------------------------- transpose
// dst[c][r] = src[r][c], 16-bit elements, 64 x 64 tiles through LDS: a tile's
// rows are read as 16-byte chunks (8 per row, 2 per thread) and written out
// as 16-byte chunks of its columns; tiles past the matrix edge go element by
// element.  The padding of 8 elements per LDS row spreads a column's reads
// over the banks.
__global__ __launch_bounds__(256) void transpose16_kernel(const uint16_t *src, int rows, int cols,
                                                          uint16_t *dst) {
  __shared__ __attribute__((aligned(16))) uint16_t t[64][64 + 8];
  const int tiles_c = (cols + 63) / 64;
  const int r0 = (int)(blockIdx.x / tiles_c) * 64, c0 = (int)(blockIdx.x % tiles_c) * 64;
  const bool full = r0 + 64 <= rows && c0 + 64 <= cols && cols % 8 == 0 && rows % 8 == 0 &&
                    (((uintptr_t)src | (uintptr_t)dst) & 15) == 0;
  if (full) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int q = threadIdx.x + 256 * h, r = q >> 3, c = (q & 7) * 8;
      const uint4 v = *reinterpret_cast<const uint4 *>(src + (int64_t)(r0 + r) * cols + c0 + c);
      *reinterpret_cast<uint4 *>(&t[r][c]) = v;
    }
    __syncthreads();
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int q = threadIdx.x + 256 * h, c = q >> 3, r = (q & 7) * 8;
      uint16_t e[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) e[k] = t[r + k][c];
      uint4 v;
      v.x = e[0] | (uint32_t)e[1] << 16;
      v.y = e[2] | (uint32_t)e[3] << 16;
      v.z = e[4] | (uint32_t)e[5] << 16;
      v.w = e[6] | (uint32_t)e[7] << 16;
      *reinterpret_cast<uint4 *>(dst + (int64_t)(c0 + c) * rows + r0 + r) = v;
    }
    return;
  }
  for (int q = threadIdx.x; q < 64 * 64; q += 256) {
    const int r = r0 + (q >> 6), c = c0 + (q & 63);
    if (r < rows && c < cols) dst[(int64_t)c * rows + r] = src[(int64_t)r * cols + c];
  }
}

}  // namespace


// Dispatch on the number of 512-column groups per row (d <= 8192).
#define AJ_NV_DISPATCH(d, CALL)                      \
  do {                                               \
    const int nv_ = ((d) + 511) / 512;               \
    if (nv_ <= 1) { constexpr int NV = 1; CALL; }     \
    else if (nv_ <= 2) { constexpr int NV = 2; CALL; } \
    else if (nv_ <= 3) { constexpr int NV = 3; CALL; } \
    else if (nv_ <= 4) { constexpr int NV = 4; CALL; } \
    else if (nv_ <= 7) { constexpr int NV = 7; CALL; } \
    else if (nv_ <= 10) { constexpr int NV = 10; CALL; } \
    else { constexpr int NV = 16; CALL; }             \
  } while (0)

template <typename T>
void rmsnorm_fwd(const T *x, const T *g, int n, int d, float eps, const int32_t *rows, int shift,
                 T *out, float *rstd, hipStream_t s) {
  if (n <= 0) return;
  AJ_NV_DISPATCH(d, (rmsnorm_fwd_kernel<T, NV><<<blocks_for(n, kRowsPerBlock), 256, 0, s>>>(
                        x, g, n, d, eps, rows, shift, out, rstd)));
}

size_t rmsnorm_bwd_part_floats(int n, int d) {
  (void)n;
  return (size_t)kBwdBlocks * d;
}

template <typename T>
void rmsnorm_bwd(const float *dy, const T *x, const float *rstd, const T *g, int n, int d,
                 const int32_t *rows, int shift, int scatter, const float *add, float *dx, T *dx_t,
                 float *dg_part, float *dg, hipStream_t s) {
  if (n <= 0) return;
  unsigned nb = blocks_for(n, 8 * kRowsPerBlock);     // ~8 rows per wave
  if (nb > (unsigned)kBwdBlocks) nb = kBwdBlocks;
  AJ_NV_DISPATCH(d, (rmsnorm_bwd_kernel<T, NV><<<nb, 256, 0, s>>>(
                        dy, x, rstd, g, n, d, rows, shift, scatter, add, dx, dx_t, dg_part)));
  if (dg) col_reduce_kernel<<<(d + 63) / 64, 256, 0, s>>>(dg_part, (int)nb, d, dg);
}

template <typename T>
void rope(T *qkv, int n, const int32_t *pos, int n_rot_heads, int ld, int hd, float theta,
          bool inverse, hipStream_t s) {
  const int64_t total = (int64_t)n * n_rot_heads * (hd / 8);   // hd is a multiple of 8
  if (total > 0)
    rope_kernel<T><<<blocks_for(total, 256), 256, 0, s>>>(qkv, n, pos, n_rot_heads, ld, hd,
                                                         log((double)theta), inverse ? 1 : 0);
}

template <typename T>
void swiglu_fwd(const T *gu, int n, int F, T *out, hipStream_t s) {
  const int64_t total = (int64_t)n * (F / 8);
  if (total > 0) swiglu_fwd_kernel<T><<<blocks_for(total, 256), 256, 0, s>>>(gu, n, F, out);
}

template <typename TI, typename T>
void swiglu_bwd(const TI *ds, const T *gu, int n, int F, T *dgu, hipStream_t s) {
  const int64_t total = (int64_t)n * (F / 8);
  if (total > 0) swiglu_bwd_kernel<TI, T><<<blocks_for(total, 256), 256, 0, s>>>(ds, gu, n, F, dgu);
}

template <typename T>
void cast_from_f32(const float *in, int64_t n, T *out, hipStream_t s) {
  if (n > 0) cast_kernel<T><<<blocks_for((n + 7) / 8, 256), 256, 0, s>>>(in, n, out);
}

template <typename T>
void scale_cast(const float *in, int64_t n, float scale, T *out, T *lo, hipStream_t s) {
  if (n > 0) scale_cast_kernel<T><<<blocks_for(n, 256), 256, 0, s>>>(in, n, scale, out, lo);
}

void transpose16(const void *src, int rows, int cols, void *dst, hipStream_t s) {
  if (rows <= 0 || cols <= 0) return;
  const int64_t tiles = (int64_t)((rows + 63) / 64) * ((cols + 63) / 64);
  transpose16_kernel<<<(unsigned)tiles, 256, 0, s>>>((const uint16_t *)src, rows, cols,
                                                     (uint16_t *)dst);
}

void fill_f32(float *p, int64_t n, float v, hipStream_t s) {
  if (n > 0) fill_kernel<<<blocks_for(n, 256), 256, 0, s>>>(p, n, v);
}

void splitk_reduce(const float *part, int S, int64_t n, float *out, bool accumulate, hipStream_t s) {
  if (n > 0) splitk_reduce_kernel<<<blocks_for(n, 256), 256, 0, s>>>(part, S, n, out, accumulate ? 1 : 0);
}

#define AJ_INST(T)                                                                              \
  template void rmsnorm_fwd<T>(const T *, const T *, int, int, float, const int32_t *, int, T *, \
                               float *, hipStream_t);                                          \
  template void rmsnorm_bwd<T>(const float *, const T *, const float *, const T *, int, int,    \
                               const int32_t *, int, int, const float *, float *, T *, float *, \
                               float *, hipStream_t);                                          \
  template void rope<T>(T *, int, const int32_t *, int, int, int, float, bool, hipStream_t);    \
  template void swiglu_fwd<T>(const T *, int, int, T *, hipStream_t);                           \
  template void swiglu_bwd<float, T>(const float *, const T *, int, int, T *, hipStream_t);     \
  template void cast_from_f32<T>(const float *, int64_t, T *, hipStream_t);                     \
  template void scale_cast<T>(const float *, int64_t, float, T *, T *, hipStream_t);
AJ_INST(float)
AJ_INST(bf16_t)
template void swiglu_bwd<bf16_t, bf16_t>(const bf16_t *, const bf16_t *, int, int, bf16_t *, hipStream_t);

}  // namespace aj
