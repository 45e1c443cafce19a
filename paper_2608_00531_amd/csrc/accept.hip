// cure_accept: greedy acceptance over the candidate tree (Sec. 3.1 Eq. 1,
// Sec. 3.5 Eq. 4). One 256-thread workgroup per sequence, one thread per node.
//
// A node matches when its token equals the target's argmax before it (root_tgt
// for a node hanging off the context, else tgt[parent]). It is accepted when
// every node on its root path matches; each thread checks its own path by
// following parent pointers in LDS (parent[n] < n bounds every walk by the
// node's depth). The winner is the accepted node maximising (depth, -index),
// found with one packed-key max reduction; its root path is then written out.
#include <hip/hip_runtime.h>

#include "common.hpp"
#include "host_util.hpp"

namespace cure {
namespace {

constexpr int kThreads = CURE_MAX_TREE_NODES;   // 256: one thread per node

struct Args {
  const int32_t* parent;
  const int32_t* token;
  const int32_t* tgt;
  const int32_t* root_tgt;
  const int32_t* n_nodes;
  int32_t chain_len, n_max;
  int32_t* acc_len;
  int32_t* path;
  int32_t* best;
  int32_t* bonus;
  int32_t* resync;
};

__global__ __launch_bounds__(kThreads) void accept_kernel(Args a) {
  __shared__ int s_parent[kThreads];
  __shared__ int s_tgt[kThreads];
  __shared__ int s_match[kThreads];
  __shared__ int s_bad;
  __shared__ int s_key[kThreads / kWave];

  // Every global read is independent of the others (one memory round trip):
  // each thread loads its node's parent, token and target argmax.
  const int b = blockIdx.x;
  const int n = threadIdx.x;
  const int64_t row = (int64_t)b * a.n_max;
  const int nn = a.n_nodes[b];
  const int root_tgt = a.root_tgt[b];
  const int N = min(max(nn, 0), a.n_max);
  int p = -1, tok = 0;
  if (n < a.n_max) {
    p = a.parent[row + n];
    tok = a.token[row + n];
    s_tgt[n] = a.tgt[row + n];
  }
  if (n == 0) s_bad = (nn < 0 || nn > a.n_max);
  __syncthreads();
  if (n < N) {
    s_parent[n] = p;
    const bool valid = p >= -1 && p < n;
    if (!valid) s_bad = 1;
    // tgt is read only through a validated parent index.
    const int want = p < 0 ? root_tgt : (valid ? s_tgt[p] : root_tgt);
    s_match[n] = tok == want;
  }
  __syncthreads();

  if (s_bad) {
    for (int i = n; i < a.n_max; i += kThreads) a.path[row + i] = -1;
    if (n == 0) {
      a.acc_len[b] = -1;
      a.best[b] = -1;
      a.bonus[b] = root_tgt;
      a.resync[b] = -1;
    }
    return;
  }

  // Own path: accepted iff every node on it matches; depth = its length - 1.
  int key = -1;
  if (n < N) {
    int ok = 1, depth = 0;
    for (int j = n; j >= 0; j = s_parent[j]) {
      ok &= s_match[j];
      depth += (j != n);
    }
    if (ok) key = (depth << 8) | (kThreads - 1 - n);   // larger depth, then lower index
  }
  key = wave_max(key);
  if ((n & (kWave - 1)) == 0) s_key[n / kWave] = key;
  __syncthreads();
  int top = s_key[0];
#pragma unroll
  for (int w = 1; w < kThreads / kWave; ++w) top = max(top, s_key[w]);

  const int win = top < 0 ? -1 : (kThreads - 1 - (top & 0xff));
  const int len = top < 0 ? 0 : (top >> 8) + 1;
  // path[i] for i < len is the ancestor of win at depth i; the rest is -1.
  for (int i = n; i < a.n_max; i += kThreads) {
    int v = -1;
    if (i < len) {
      int j = win;
      for (int up = len - 1 - i; up > 0; --up) j = s_parent[j];
      v = j;
    }
    a.path[row + i] = v;
  }
  if (n == 0) {
    int repair = 0;
    for (int j = win; j >= 0; j = s_parent[j]) repair |= (j >= a.chain_len);
    a.acc_len[b] = len;
    a.best[b] = win;
    a.bonus[b] = win < 0 ? root_tgt : s_tgt[win];
    a.resync[b] = repair;
  }
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
         acc_len, path, best, bonus, resync};
  hipLaunchKernelGGL(accept_kernel, dim3(batch), dim3(kThreads), 0, as_stream(stream), a);
  return launch_status();
}
