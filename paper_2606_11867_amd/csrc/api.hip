// Host utilities of the C ABI: status strings, per-thread error text,
// launch checks and the cached compute-unit count.
#include <stdarg.h>
#include <stdio.h>

#include "common.h"

namespace foremoe {

static thread_local char g_last_error[512] = "";

int set_error(int status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return status;
}

int check_launch(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return set_error(FOREMOE_EHIP, "%s: %s", what, hipGetErrorString(e));
  return FOREMOE_OK;
}

int num_cus() {
  // Cached per device: compute units of the current device.
  static thread_local int cached_dev = -1;
  static thread_local int cached_cus = 0;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  if (dev != cached_dev) {
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
      cus = 256;
    cached_dev = dev;
    cached_cus = cus;
  }
  return cached_cus;
}

}  // namespace foremoe

extern "C" {

const char* foremoe_status_string(int status) {
  switch (status) {
    case FOREMOE_OK: return "ok";
    case FOREMOE_EINVAL: return "invalid argument";
    case FOREMOE_EUNSUPPORTED: return "unsupported shape or dtype";
    case FOREMOE_EHIP: return "HIP launch failure";
    default: return "unknown status";
  }
}

const char* foremoe_last_error(void) { return foremoe::g_last_error; }

const char* foremoe_version(void) { return "foremoe-mi355x 0.1 (gfx950)"; }

size_t foremoe_workspace_size(int64_t T, int32_t K, int32_t E) {
  if (T < 0 || K < 1 || K > FOREMOE_MAX_TOPK || E < 1 || E > FOREMOE_MAX_EXPERTS) return 0;
  return foremoe::ws_bytes_needed(T, K, E);
}

}  // extern "C"
