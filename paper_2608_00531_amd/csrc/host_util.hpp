// Host-side helpers for the libcure C ABI: device properties and launch checks.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "cure.h"

namespace cure {

// Compute-unit count of the current device (cached per device id).
int device_cu_count();

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

// Converts the result of a kernel launch into a status code.
inline cure_status launch_status() {
  return hipGetLastError() == hipSuccess ? CURE_OK : CURE_ERR_HIP;
}

}  // namespace cure
