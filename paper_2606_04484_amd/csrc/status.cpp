// Status strings, the thread-local error text and the device error read-back.
#include <hip/hip_runtime.h>
#include <cstdarg>
#include <cstdio>
#include <vector>
#include "common.h"

namespace aj {
static thread_local char g_err[512] = "";

void set_error(const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
}

int fail(int status, const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return status;
}

namespace {
struct Rec { hipEvent_t a, b; int kc; double flops; };
std::vector<Rec> g_recs;
std::vector<hipEvent_t> g_pool;
bool g_timing = false;

hipEvent_t take_event() {
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}
}  // namespace

int timing_begin(hipStream_t s, int kc, double flops) {
  if (!g_timing) return -1;
  Rec r{take_event(), take_event(), kc, flops};
  if (!r.a || !r.b) return -1;
  hipEventRecord(r.a, s);
  g_recs.push_back(r);
  return (int)g_recs.size() - 1;
}

void timing_end(hipStream_t s, int idx) {
  if (idx >= 0 && idx < (int)g_recs.size()) hipEventRecord(g_recs[idx].b, s);
}

static void timing_clear() {
  for (auto &r : g_recs) {
    hipEventSynchronize(r.b);
    g_pool.push_back(r.a);
    g_pool.push_back(r.b);
  }
  g_recs.clear();
}

int check_launch(const char *what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(AJ_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return AJ_OK;
}
}  // namespace aj

extern "C" const char *aj_status_str(int s) {
  switch (s) {
    case AJ_OK: return "ok";
    case AJ_ERR_NULL: return "null pointer";
    case AJ_ERR_SHAPE: return "bad size or offset";
    case AJ_ERR_UNSUPPORTED: return "unsupported";
    case AJ_ERR_WORKSPACE: return "workspace too small";
    case AJ_ERR_HIP: return "HIP error";
    default: return "unknown status";
  }
}

extern "C" const char *aj_last_error(void) { return aj::g_err; }

extern "C" int aj_timing_enable(int on) {
  aj::timing_clear();
  aj::g_timing = on != 0;
  return AJ_OK;
}

extern "C" int aj_timing_read(double *ms, int64_t *launches, double *flops) {
  AJ_REQUIRE(ms && launches && flops, AJ_ERR_NULL, "aj_timing_read: null pointer");
  for (int k = 0; k < AJ_KC_COUNT; ++k) { ms[k] = 0; launches[k] = 0; flops[k] = 0; }
  for (auto &r : aj::g_recs) {
    float t = 0.f;
    if (hipEventSynchronize(r.b) != hipSuccess || hipEventElapsedTime(&t, r.a, r.b) != hipSuccess)
      return aj::fail(AJ_ERR_HIP, "aj_timing_read: %s", hipGetErrorString(hipGetLastError()));
    if (r.kc < 0 || r.kc >= AJ_KC_COUNT) continue;
    ms[r.kc] += t;
    launches[r.kc] += 1;
    flops[r.kc] += r.flops;
  }
  return AJ_OK;
}

extern "C" int aj_read_device_error(const int32_t *err, void *stream, int32_t *host_err) {
  AJ_REQUIRE(err && host_err, AJ_ERR_NULL, "aj_read_device_error: null pointer");
  hipStream_t s = (hipStream_t)stream;
  if (hipMemcpyAsync(host_err, err, sizeof(int32_t), hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    return aj::fail(AJ_ERR_HIP, "aj_read_device_error: %s", hipGetErrorString(hipGetLastError()));
  return AJ_OK;
}
