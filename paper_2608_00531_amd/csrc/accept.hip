// cure_accept: greedy acceptance over the candidate tree (Sec. 3.1 Eq. 1,
// Sec. 3.5 Eq. 4). One workgroup per sequence, one thread per node: a single
// wave (no barriers) for trees of up to 64 nodes, else 256 threads. The walk itself
// (accept_walk.hpp) is shared with the margin pass's acceptance epilogue.
#include <hip/hip_runtime.h>

#include "accept_walk.hpp"
#include "common.hpp"
#include "host_util.hpp"

namespace cure {
namespace {

constexpr int kMaxNodes = CURE_MAX_TREE_NODES;   // 256

struct Args {
  const int32_t* parent;
  const int32_t* token;
  const int32_t* tgt;
  const int32_t* root_tgt;
  const int32_t* n_nodes;
  int32_t chain_len, n_max;
  AcceptOut out;
};

// NT threads, NT >= n_max.
template <int NT>
__global__ __launch_bounds__(NT) void accept_kernel(Args a) {
  __shared__ AcceptLds<NT> s;
  // Every global read is independent of the others (one memory round trip):
  // each thread loads its node's parent, token and target argmax.
  const int b = blockIdx.x;
  const int n = threadIdx.x;
  const int64_t row = (int64_t)b * a.n_max;
  const int nn = a.n_nodes[b];
  const int root_tgt = a.root_tgt[b];
  int p = -1, tok = 0;
  if (n < a.n_max) {
    p = a.parent[row + n];
    tok = a.token[row + n];
    s.tgt[n] = a.tgt[row + n];
  }
  accept_walk<NT, NT == kWave>(s, n, b, p, tok, nn, root_tgt, a.n_max, a.chain_len, a.out);
}

}  // namespace
}  // namespace cure

using namespace cure;

extern "C" cure_status cure_accept(const int32_t* parent, const int32_t* token,
                                   const int32_t* tgt, const int32_t* root_tgt,
                                   const int32_t* n_nodes, int32_t chain_len, int32_t batch,
                                   int32_t n_max, int32_t* acc_len, int32_t* path,
                                   int32_t* best, int32_t* bonus, int32_t* resync,
                                   void* stream) {
  if (batch < 0 || n_max < 0 || chain_len < 0) return CURE_ERR_INVALID_ARG;
  if (batch == 0) return CURE_OK;
  if (n_max > CURE_MAX_TREE_NODES) return CURE_ERR_UNSUPPORTED;
  if (!parent || !token || !tgt || !root_tgt || !n_nodes || !acc_len || !best || !bonus ||
      !resync || (n_max > 0 && !path))
    return CURE_ERR_INVALID_ARG;
  Args a{parent, token, tgt, root_tgt, n_nodes, chain_len, n_max,
         AcceptOut{acc_len, path, best, bonus, resync}};
  if (n_max <= kWave)
    hipLaunchKernelGGL(accept_kernel<kWave>, dim3(batch), dim3(kWave), 0, as_stream(stream), a);
  else
    hipLaunchKernelGGL(accept_kernel<kMaxNodes>, dim3(batch), dim3(kMaxNodes), 0, as_stream(stream), a);
  return launch_status();
}
