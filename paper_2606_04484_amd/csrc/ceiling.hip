// Measured ceilings of the device, for reading the rooflines against what the
// chip sustains rather than its published peaks alone:
//   * the bf16 matrix-core rate with no memory traffic at all: every wave runs
//     v_mfma_f32_32x32x16_bf16 on 8 independent accumulators from registers
//     (one wave per SIMD: the kernel holds 260 registers per lane), with
//     random operands (every product's inputs toggle, as in a GEMM over
//     trained or random weights) or constant ones;
//   * the HBM rates of a streaming copy and of a read-only stream (16-byte
//     loads and stores, a grid over the whole buffer).
#include "common.h"

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kMfmaIters = 4000;

AJ_DEV uint32_t mix(uint32_t x) {
  x ^= x >> 15;
  x *= 2246822519u;
  x ^= x >> 13;
  x *= 3266489917u;
  return x ^ (x >> 16);
}

// Two bfloat16 values with random signs and mantissas, exponents near 2^-4
// (products and sums stay far from overflow over the whole loop).
AJ_DEV uint32_t rand_bf16x2(uint32_t x) {
  return (x & 0x80008000u) | ((0x3d00u + ((x >> 3) & 0x7fu)) << 16) | (0x3d00u + ((x >> 19) & 0x7fu));
}

template <bool RANDOM>
__global__ __launch_bounds__(256) void mfma_ceiling_kernel(float *out, int iters) {
  const uint32_t t = blockIdx.x * 256 + threadIdx.x;
  bf16x8_t a[8], b[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    u32x4_t ua, ub;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      ua[e] = RANDOM ? rand_bf16x2(mix(t * 64 + j * 8 + e)) : 0x3d803d80u;
      ub[e] = RANDOM ? rand_bf16x2(mix(t * 64 + j * 8 + e + 4) ^ 0x9e3779b9u) : 0x3d803d80u;
    }
    a[j] = __builtin_bit_cast(bf16x8_t, ua);
    b[j] = __builtin_bit_cast(bf16x8_t, ub);
  }
  f32x16_t acc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[j][r] = 0.f;
  for (int it = 0; it < iters; ++it) {
    // each accumulator meets a different operand pair at every step
#pragma unroll
    for (int k = 0; k < 8; ++k)
#pragma unroll
      for (int j = 0; j < 8; ++j)
        acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[j], b[(j + k) & 7], acc[j], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[j][r];
  out[t] = s;   // keeps the products live
}

// One 16-byte item per thread, a grid over the whole buffer (the access
// pattern of the path's elementwise kernels, which stream faster than a
// grid-stride loop here).
__global__ __launch_bounds__(256) void copy_ceiling_kernel(const u32x4_t *src, u32x4_t *dst,
                                                           int64_t n) {
  const int64_t i = blockIdx.x * 256 + (int64_t)threadIdx.x;
  if (i < n) dst[i] = src[i];
}

// Read-only: four 16-byte items per thread (each load instruction of a wave
// reads 1 KB contiguous), folded into one word that is stored only if it
// equals a constant -- the loads stay live, the writes are nil.
__global__ __launch_bounds__(256) void read_ceiling_kernel(const u32x4_t *src, int64_t n,
                                                           uint32_t *out) {
  const int64_t i0 = blockIdx.x * 1024 + (int64_t)threadIdx.x;
  uint32_t x = 0;
  u32x4_t v[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) v[r] = src[min(i0 + 256 * r, n - 1)];
#pragma unroll
  for (int r = 0; r < 4; ++r) x ^= v[r][0] ^ v[r][1] ^ v[r][2] ^ v[r][3];
  if (x == 0x9e3779b9u) out[0] = x;
}

// Two timing events, destroyed on every return path.
struct Events {
  hipEvent_t e0 = nullptr, e1 = nullptr;
  Events() {
    if (hipEventCreate(&e0) != hipSuccess) e0 = nullptr;
    if (hipEventCreate(&e1) != hipSuccess) e1 = nullptr;
  }
  ~Events() {
    if (e0) (void)hipEventDestroy(e0);
    if (e1) (void)hipEventDestroy(e1);
  }
  bool ok() const { return e0 && e1; }
  // records e1 on s after the work since e0, waits for it, the time between
  bool elapsed(hipStream_t s, float *ms) {
    return hipEventRecord(e1, s) == hipSuccess && hipEventSynchronize(e1) == hipSuccess &&
           hipEventElapsedTime(ms, e0, e1) == hipSuccess;
  }
};

}  // namespace

extern "C" int aj_ceiling_mfma_bf16(int random_operands, void *out, size_t out_bytes, void *stream,
                                    double *tflops) {
  AJ_REQUIRE(out && tflops, AJ_ERR_NULL, "aj_ceiling_mfma_bf16: null pointer");
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      cus <= 0)
    return aj::fail(AJ_ERR_HIP, "aj_ceiling_mfma_bf16: no device");
  const int wgs = 2 * cus;   // two rounds of one 4-wave workgroup per CU
  AJ_REQUIRE(out_bytes >= (size_t)wgs * 256 * sizeof(float), AJ_ERR_WORKSPACE,
             "aj_ceiling_mfma_bf16: out holds %zu bytes, needs %zu", out_bytes,
             (size_t)wgs * 256 * sizeof(float));
  hipStream_t s = (hipStream_t)stream;
  Events ev;
  if (!ev.ok()) return aj::fail(AJ_ERR_HIP, "aj_ceiling_mfma_bf16: event");
  double best = 0.0;
  for (int rep = 0; rep < 3; ++rep) {
    if (hipEventRecord(ev.e0, s) != hipSuccess)
      return aj::fail(AJ_ERR_HIP, "aj_ceiling_mfma_bf16: event record");
    if (random_operands)
      mfma_ceiling_kernel<true><<<wgs, 256, 0, s>>>((float *)out, kMfmaIters);
    else
      mfma_ceiling_kernel<false><<<wgs, 256, 0, s>>>((float *)out, kMfmaIters);
    float ms = 0.f;
    if (!ev.elapsed(s, &ms))
      return aj::fail(AJ_ERR_HIP, "aj_ceiling_mfma_bf16: %s", hipGetErrorString(hipGetLastError()));
    const double flops = (double)wgs * 4 * kMfmaIters * 64 * (2.0 * 32 * 32 * 16);
    const double r = flops / (ms * 1e-3) / 1e12;
    if (r > best) best = r;
  }
  *tflops = best;
  return aj::check_launch("aj_ceiling_mfma_bf16");
}

extern "C" int aj_ceiling_copy(void *buf, size_t bytes, void *stream, double *gbps,
                               double *read_gbps) {
  AJ_REQUIRE(buf && gbps && read_gbps, AJ_ERR_NULL, "aj_ceiling_copy: null pointer");
  AJ_REQUIRE(bytes >= 2 * 16 && bytes <= ((size_t)1 << 40) && ((uintptr_t)buf & 15) == 0,
             AJ_ERR_SHAPE, "aj_ceiling_copy: %zu bytes at %p (16-byte aligned, 32 B .. 1 TiB)",
             bytes, buf);
  const int64_t n = (int64_t)(bytes / 2 / 16);   // 16-byte items per half
  const u32x4_t *src = (const u32x4_t *)buf;
  u32x4_t *dst = (u32x4_t *)buf + n;
  hipStream_t s = (hipStream_t)stream;
  Events ev;
  if (!ev.ok()) return aj::fail(AJ_ERR_HIP, "aj_ceiling_copy: event");
  double best = 0.0, best_r = 0.0;
  for (int rep = 0; rep < 8; ++rep) {
    const bool rd = rep >= 4;   // the read-only stream writes its words over dst
    if (hipEventRecord(ev.e0, s) != hipSuccess)
      return aj::fail(AJ_ERR_HIP, "aj_ceiling_copy: event record");
    if (rd) read_ceiling_kernel<<<(int)((n + 1023) / 1024), 256, 0, s>>>(src, n, (uint32_t *)dst);
    else copy_ceiling_kernel<<<(int)((n + 255) / 256), 256, 0, s>>>(src, dst, n);
    float ms = 0.f;
    if (!ev.elapsed(s, &ms))
      return aj::fail(AJ_ERR_HIP, "aj_ceiling_copy: %s", hipGetErrorString(hipGetLastError()));
    const double r = (rd ? 1.0 : 2.0) * 16 * n / (ms * 1e-3) / 1e9;
    if (rep == 0 || rep == 4) continue;   // the first run of each pages the buffer in
    if (rd) best_r = r > best_r ? r : best_r;
    else best = r > best ? r : best;
  }
  *gbps = best;
  *read_gbps = best_r;
  return aj::check_launch("aj_ceiling_copy");
}
