// Shared device helpers and host-side error plumbing for libaj (gfx950 only).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>
#include "aj.h"

#define AJ_DEV __device__ __forceinline__

typedef uint16_t bf16_t;   // bfloat16 storage (upper half of a float32)

AJ_DEV float bf2f(bf16_t v) { return __uint_as_float((uint32_t)v << 16); }

typedef __bf16 bf16x2_hw_t __attribute__((ext_vector_type(2)));
typedef float f32x2_hw_t __attribute__((ext_vector_type(2)));

// Two float32 -> two bfloat16 in one word (lo in bits 0..15), round to
// nearest even, NaN stays NaN: one v_cvt_pk_bf16_f32 on gfx950.
AJ_DEV uint32_t f2bf2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_hw_t{lo, hi}, bf16x2_hw_t));
}

// float32 -> bfloat16, round to nearest even; NaN stays NaN.
AJ_DEV bf16_t f2bf(float f) { return (bf16_t)(f2bf2(f, 0.f) & 0xffffu); }

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
// Brackets every launch of one library call (a stage of the path) for the
// benchmark timing: the end event is recorded when the span leaves scope,
// after the call's last launch.
struct StageSpan {
  hipStream_t s;
  int idx;
  StageSpan(hipStream_t s_, int kc) : s(s_), idx(timing_begin(s_, kc, 0.0)) {}
  ~StageSpan() { timing_end(s, idx); }
  StageSpan(const StageSpan &) = delete;
  StageSpan &operator=(const StageSpan &) = delete;
};

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
