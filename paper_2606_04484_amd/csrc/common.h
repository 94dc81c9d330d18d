// Shared device helpers and host-side error plumbing for libaj (gfx950 only).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>
#include "aj.h"

#define AJ_DEV __device__ __forceinline__

typedef uint16_t bf16_t;   // bfloat16 storage (upper half of a float32)

AJ_DEV float bf2f(bf16_t v) { return __uint_as_float((uint32_t)v << 16); }

// float32 -> bfloat16, round to nearest even; NaN stays NaN.
AJ_DEV bf16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (bf16_t)((u >> 16) | 0x40);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

template <typename T> AJ_DEV float ldf(const T *p);
template <> AJ_DEV float ldf<float>(const float *p) { return *p; }
template <> AJ_DEV float ldf<bf16_t>(const bf16_t *p) { return bf2f(*p); }
template <typename T> AJ_DEV void stf(T *p, float v);
template <> AJ_DEV void stf<float>(float *p, float v) { *p = v; }
template <> AJ_DEV void stf<bf16_t>(bf16_t *p, float v) { *p = f2bf(v); }

// ---------------------------------------------------------------- host side
namespace aj {
void set_error(const char *fmt, ...);
int fail(int status, const char *fmt, ...);
// Returns AJ_OK or AJ_ERR_HIP (with the HIP error text) after a launch.
int check_launch(const char *what);

// Benchmark timing (aj_timing_enable): returns a record index or -1 when off.
int timing_begin(hipStream_t s, int kclass, double flops);
void timing_end(hipStream_t s, int idx);

inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// Carves aligned sub-buffers out of a caller-provided workspace.
struct Carver {
  char *base;
  size_t off = 0;
  explicit Carver(void *b) : base((char *)b) {}
  template <typename T> T *take(size_t n) {
    off = align_up(off, 256);
    T *p = base ? (T *)(base + off) : nullptr;
    off += n * sizeof(T);
    return p;
  }
  size_t bytes() const { return align_up(off, 256); }
};
}  // namespace aj

#define AJ_REQUIRE(cond, status, ...) \
  do { if (!(cond)) return aj::fail((status), __VA_ARGS__); } while (0)
