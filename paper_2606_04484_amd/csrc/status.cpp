// Status strings, the thread-local error text and the device error read-back.
#include <hip/hip_runtime.h>
#include <cstdarg>
#include <cstdio>
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

extern "C" int aj_read_device_error(const int32_t *err, void *stream, int32_t *host_err) {
  AJ_REQUIRE(err && host_err, AJ_ERR_NULL, "aj_read_device_error: null pointer");
  hipStream_t s = (hipStream_t)stream;
  if (hipMemcpyAsync(host_err, err, sizeof(int32_t), hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    return aj::fail(AJ_ERR_HIP, "aj_read_device_error: %s", hipGetErrorString(hipGetLastError()));
  return AJ_OK;
}
