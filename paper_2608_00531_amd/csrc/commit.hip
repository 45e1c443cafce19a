// cure_commit: commit the winning path of a verify step (Sec. 3.5, Algorithm 1).
//
// The accepted tokens become context for the next step, so each layer's target
// cache must hold their keys and values right after the old context, in depth
// order. Tree node n's rows sit at ctx_len + n, so the node at depth j of the
// winning path moves from ctx_len + path[j] to ctx_len + j. The step also
// emits the accepted tokens and the bonus token, the new context length, and
// where the draft-cache replay starts (the first repair node of the path).
//
// Work split: one 256-thread workgroup per (sequence, 256 columns), where a
// column is one 16-byte slice of a cache row in one layer's K or V. Every
// column is moved by one thread, and no two threads touch the same bytes, so
// the in-place move needs no cross-thread ordering. Within a thread, rows move
// in increasing depth, a group of up to kGroup rows at a time (all loads of a
// group, then its stores). A root path in topological order is strictly
// increasing with path[j] >= j, so a row that a later depth reads, path[i] with
// i > j, is never a row an earlier depth j has already overwritten. The same
// property makes the rows with path[j] == j a prefix of the path: those rows
// are already in place and are skipped.
#include <hip/hip_runtime.h>

#include "common.hpp"
#include "host_util.hpp"

namespace cure {
namespace {

constexpr int kThreads = 256;
constexpr int kGroup = 16;   // rows in flight per thread: 16 x 16 B = 64 VGPRs

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

struct Args {
  uint8_t* k;
  uint8_t* v;
  int64_t layer_stride_bytes;
  int64_t row_bytes;
  int32_t vecs_per_row;   // row_bytes / 16
  int32_t cols;           // n_layers * 2 * vecs_per_row
  const int64_t* kv_off;
  const int32_t* ctx_len;
  const int32_t* n_nodes;
  const int32_t* path;
  const int32_t* acc_len;
  const int32_t* token;
  const int32_t* bonus;
  int32_t chain_len, n_max;
  int32_t* new_ctx_len;
  int32_t* emit;
  int32_t* emit_cnt;
  int32_t* replay_start;
  int32_t* status;
};

__global__ __launch_bounds__(kThreads) void commit_kernel(Args a) {
  const int b = blockIdx.y;
  const int t = threadIdx.x;
  const int64_t prow = (int64_t)b * a.n_max;

  // One round trip: the sequence's sizes and this thread's path entry with its
  // predecessor (the predecessor check makes the path strictly increasing).
  const int acc = a.acc_len[b];
  const int nn = a.n_nodes[b];
  const int ctx = a.ctx_len[b];
  const int64_t off = a.kv_off[b];
  const int len = min(max(acc, 0), a.n_max);
  __shared__ int s_path[CURE_MAX_TREE_NODES];
  int p = 0, pp = -1;
  if (t < len) {
    p = a.path[prow + t];
    if (t > 0) pp = a.path[prow + t - 1];
    s_path[t] = p;
  }
  const bool seq_ok = acc >= 0 && nn >= 0 && nn <= a.n_max && acc <= nn && ctx >= 0 && off >= 0;
  // Barriers with a reduction; every thread reaches them.
  const bool any_bad = __syncthreads_or(t < len && !(p > pp && p < nn));
  const bool bad = !seq_ok || any_bad;
  // Rows already in place (path[j] == j) form a prefix; so do the chain nodes
  // (path[j] < chain_len), whose end is where the replay starts.
  const int first_moved = __syncthreads_count(t < len && p == t);
  const int replay = __syncthreads_count(t < len && p < a.chain_len);

  if (blockIdx.x == 0) {
    // Tokens: the accepted path, then the bonus, padded with -1 to n_max + 1.
    const int64_t erow = (int64_t)b * (a.n_max + 1);
    for (int j = t; j <= a.n_max; j += kThreads) {
      int tok = -1;
      if (!bad && j < acc) tok = a.token[prow + p];   // j < acc <= 256: j == t
      if (!bad && j == acc) tok = a.bonus[b];
      a.emit[erow + j] = tok;
    }
    if (t == 0) {
      a.emit_cnt[b] = bad ? 0 : acc + 1;
      a.new_ctx_len[b] = bad ? ctx : ctx + acc;
      a.replay_start[b] = bad ? 0 : replay;
      a.status[b] = bad ? CURE_ERR_BAD_TREE : CURE_OK;
    }
  }
  if (bad || first_moved >= acc) return;

  const int col = blockIdx.x * kThreads + t;
  if (col >= a.cols) return;
  const int per_layer = 2 * a.vecs_per_row;
  const int layer = col / per_layer;
  const int rem = col - layer * per_layer;
  const int tensor = rem / a.vecs_per_row;
  const int c = rem - tensor * a.vecs_per_row;
  uint8_t* base = (tensor ? a.v : a.k) + (int64_t)layer * a.layer_stride_bytes +
                  (off + ctx) * a.row_bytes + (int64_t)c * 16;

  for (int j0 = first_moved; j0 < acc; j0 += kGroup) {
    // A group past the path's end reloads its last row instead of branching,
    // so the group stays in registers; those extra rows are not stored.
    u32x4 buf[kGroup];
#pragma unroll
    for (int i = 0; i < kGroup; ++i) {
      const int src = s_path[min(j0 + i, acc - 1)];
      buf[i] = *reinterpret_cast<const u32x4*>(base + (int64_t)src * a.row_bytes);
    }
    // Every load of the group has returned before any of its stores is issued.
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
#pragma unroll
    for (int i = 0; i < kGroup; ++i) {
      if (j0 + i < acc) *reinterpret_cast<u32x4*>(base + (int64_t)(j0 + i) * a.row_bytes) = buf[i];
    }
  }
}

}  // namespace
}  // namespace cure

using namespace cure;

extern "C" cure_status cure_commit(void* k, void* v, int32_t dtype, int32_t n_layers,
                                   int64_t layer_stride, int32_t hkv, int32_t d, int32_t batch,
                                   const int64_t* kv_off, const int32_t* ctx_len,
                                   const int32_t* n_nodes, const int32_t* path,
                                   const int32_t* acc_len, const int32_t* token,
                                   const int32_t* bonus, int32_t chain_len, int32_t n_max,
                                   int32_t* new_ctx_len, int32_t* emit, int32_t* emit_cnt,
                                   int32_t* replay_start, int32_t* commit_status,
                                   void* stream) {
  if (dtype != CURE_F32 && dtype != CURE_BF16) return CURE_ERR_INVALID_ARG;
  if (batch < 0 || n_layers < 0 || hkv <= 0 || d <= 0 || n_max < 0 || chain_len < 0)
    return CURE_ERR_INVALID_ARG;
  if (n_layers > 1 && (layer_stride <= 0 || layer_stride > INT64_MAX / 4))
    return CURE_ERR_INVALID_ARG;
  if (batch == 0) return CURE_OK;
  if (n_max > CURE_MAX_TREE_NODES) return CURE_ERR_UNSUPPORTED;
  if (!kv_off || !ctx_len || !n_nodes || !acc_len || !token || !bonus || !new_ctx_len ||
      !emit || !emit_cnt || !replay_start || !commit_status || (n_max > 0 && !path) ||
      (n_layers > 0 && (!k || !v)))
    return CURE_ERR_INVALID_ARG;
  // new_ctx_len is written while other workgroups still read ctx_len.
  if (static_cast<const void*>(new_ctx_len) == static_cast<const void*>(ctx_len))
    return CURE_ERR_INVALID_ARG;
  const int64_t elem = dtype == CURE_BF16 ? 2 : 4;
  const int64_t row_bytes = (int64_t)hkv * d * elem;
  if (row_bytes % 16 != 0) return CURE_ERR_UNSUPPORTED;
  const int64_t cols = (int64_t)n_layers * 2 * (row_bytes / 16);
  if (row_bytes / 16 > INT32_MAX / 2 || cols > INT32_MAX - kThreads) return CURE_ERR_UNSUPPORTED;
  const int64_t blocks_x = cols == 0 ? 1 : (cols + kThreads - 1) / kThreads;
  if (blocks_x > INT32_MAX || batch > 65535) return CURE_ERR_UNSUPPORTED;
  Args a{static_cast<uint8_t*>(k), static_cast<uint8_t*>(v), layer_stride * elem, row_bytes,
         (int32_t)(row_bytes / 16), (int32_t)cols, kv_off, ctx_len, n_nodes, path, acc_len,
         token, bonus, chain_len, n_max, new_ctx_len, emit, emit_cnt, replay_start,
         commit_status};
  hipLaunchKernelGGL(commit_kernel, dim3((unsigned)blocks_x, (unsigned)batch), dim3(kThreads), 0,
                     as_stream(stream), a);
  return launch_status();
}
