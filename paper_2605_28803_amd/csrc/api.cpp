// Status strings, version and the device check shared by every entry point.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstring>

#include "common.h"

namespace oq {

int device_check() {
  // Cached per device id: 0 = unknown, 1 = gfx950, 2 = other.
  static std::atomic<int> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return OQ_ERR_HIP;
  if (dev < 0 || dev >= 64) return OQ_ERR_DEVICE;
  int c = cache[dev].load(std::memory_order_relaxed);
  if (c == 0) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return OQ_ERR_HIP;
    c = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0 ? 1 : 2;
    cache[dev].store(c, std::memory_order_relaxed);
  }
  return c == 1 ? OQ_OK : OQ_ERR_DEVICE;
}

}  // namespace oq

extern "C" const char* oq_status_string(int status) {
  switch (status) {
    case OQ_OK: return "OQ_OK";
    case OQ_ERR_NULL: return "OQ_ERR_NULL: required pointer is NULL";
    case OQ_ERR_SHAPE: return "OQ_ERR_SHAPE: size out of range or inconsistent";
    case OQ_ERR_ALIGN: return "OQ_ERR_ALIGN: pointer or leading dimension misaligned";
    case OQ_ERR_DEVICE: return "OQ_ERR_DEVICE: current device is not gfx950";
    case OQ_ERR_HIP: return "OQ_ERR_HIP: HIP runtime call or launch failed";
    case OQ_ERR_WORKSPACE: return "OQ_ERR_WORKSPACE: workspace missing or too small";
    case OQ_ERR_ARG: return "OQ_ERR_ARG: invalid argument";
    default: return "unknown oq_status";
  }
}

extern "C" const char* oq_version(void) { return "oq 0.1.0 (gfx950)"; }

extern "C" int oq_check_device(void) { return oq::device_check(); }
