// libcure: status strings, version and the cached device-property query.
#include <hip/hip_runtime.h>

#include <mutex>

#include "cure.h"
#include "host_util.hpp"

namespace cure {

int device_cu_count() {
  static std::mutex mu;
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) dev = 0;
  const int slot = dev < 64 ? dev : 63;
  std::lock_guard<std::mutex> lock(mu);
  if (cached[slot] == 0) {
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
      cus = 256;
    cached[slot] = cus;
  }
  return cached[slot];
}

}  // namespace cure

extern "C" const char* cure_status_string(int status) {
  switch (status) {
    case CURE_OK: return "CURE_OK";
    case CURE_ERR_INVALID_ARG: return "CURE_ERR_INVALID_ARG";
    case CURE_ERR_UNSUPPORTED: return "CURE_ERR_UNSUPPORTED";
    case CURE_ERR_BAD_TREE: return "CURE_ERR_BAD_TREE";
    case CURE_ERR_HIP: return "CURE_ERR_HIP";
    case CURE_ERR_WORKSPACE: return "CURE_ERR_WORKSPACE";
    default: return "CURE_ERR_UNKNOWN";
  }
}

extern "C" int cure_version(void) { return 100; }   // 0.1.0
