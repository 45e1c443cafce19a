// cure_read_ceiling: a plain streaming read of a device buffer, the practical
// HBM read ceiling that the hot path's bandwidth is compared against.
//
// One 256-thread workgroup per 256 KB chunk. Lanes read 16-byte vectors with
// the non-temporal hint through a range-checked buffer resource (two loop steps
// of two vectors in flight, as the margin pass reads its rows), XOR all words
// of the chunk together and write that one word per chunk, so the read is both
// necessary and checkable.
#include <hip/hip_runtime.h>

#include "common.hpp"
#include "host_util.hpp"

namespace cure {
namespace {

constexpr int kThreads = 256;
constexpr uint32_t kChunkBytes = 256u << 10;
constexpr int kVecPerStep = 2;

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(kThreads) void read_ceiling_kernel(const uint8_t* buf, size_t bytes,
                                                                uint32_t* chunk_xor) {
  const size_t begin = (size_t)blockIdx.x * kChunkBytes;
  const uint32_t len = (uint32_t)min((size_t)kChunkBytes, bytes - begin);
  // Reads at or past `len` return zeros without touching memory.
  const __amdgpu_buffer_rsrc_t r =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(buf + begin), 0, (int)len, 0x00020000);
  const uint32_t step = kThreads * kVecPerStep * 16;
  u32x4 acc = {0, 0, 0, 0};
  u32x4 a[kVecPerStep], b[kVecPerStep];
  auto issue = [&](u32x4 (&x)[kVecPerStep], uint32_t base) {
#pragma unroll
    for (int u = 0; u < kVecPerStep; ++u)
      x[u] = __builtin_amdgcn_raw_buffer_load_b128(r, (int)(base + (u * kThreads + threadIdx.x) * 16), 0, 2);
  };
  issue(a, 0);
  for (uint32_t base = 0; base < len; base += 2 * step) {
    issue(b, base + step);
#pragma unroll
    for (int u = 0; u < kVecPerStep; ++u) acc ^= a[u];
    issue(a, base + 2 * step);
#pragma unroll
    for (int u = 0; u < kVecPerStep; ++u) acc ^= b[u];
  }
  uint32_t x = acc.x ^ acc.y ^ acc.z ^ acc.w;
  x ^= partner<1>((int)x);
  x ^= partner<2>((int)x);
  x ^= partner<4>((int)x);
  x ^= partner<8>((int)x);
  x ^= partner<16>((int)x);
  x ^= partner<32>((int)x);
  __shared__ uint32_t s[kThreads / kWave];
  if ((threadIdx.x & (kWave - 1)) == 0) s[threadIdx.x / kWave] = x;
  __syncthreads();
  if (threadIdx.x == 0) chunk_xor[blockIdx.x] = s[0] ^ s[1] ^ s[2] ^ s[3];
}

}  // namespace
}  // namespace cure

using namespace cure;

extern "C" size_t cure_read_ceiling_chunks(size_t bytes) {
  return (bytes + kChunkBytes - 1) / kChunkBytes;
}

extern "C" cure_status cure_read_ceiling(const void* buf, size_t bytes, uint32_t* chunk_xor,
                                         void* stream) {
  if (bytes == 0) return CURE_OK;
  if (!buf || !chunk_xor || bytes % 16 != 0) return CURE_ERR_INVALID_ARG;
  const size_t chunks = cure_read_ceiling_chunks(bytes);
  if (chunks > INT32_MAX) return CURE_ERR_UNSUPPORTED;
  hipLaunchKernelGGL(read_ceiling_kernel, dim3((unsigned)chunks), dim3(kThreads), 0,
                     as_stream(stream), static_cast<const uint8_t*>(buf), bytes, chunk_xor);
  return launch_status();
}
