// The acceptance walk of one sequence by one workgroup (Sec. 3.1 Eq. 1,
// Sec. 3.5 Eq. 4, greedy decoding), shared by cure_accept's kernel and the
// acceptance epilogue of the margin pass (cure_margins_accept).
//
// Thread n stands for tree node n. A node matches when its token equals the
// target's argmax before it (root_tgt for a node hanging off the context, else
// the argmax at its parent); it is accepted when every node on its root path
// matches. Each thread checks its own path by following parent pointers in
// LDS (parent[n] < n bounds every walk by the node's depth), stopping at the
// first node that does not match (the thread's node is then not accepted, and
// its depth does not matter), and notes on the same walk whether the path
// holds a repair node (index >= chain_len). A wave's walks thus take about as
// many steps as its longest matching run, not its deepest node. The
// winner is the accepted node maximising (depth, -index), found with one
// packed-key max reduction; its root path is then written out, one thread per
// path position.
#pragma once

#include <hip/hip_runtime.h>

#include "common.hpp"

namespace cure {

struct AcceptOut {
  int32_t* acc_len;   // [batch]
  int32_t* path;      // [batch][n_max]
  int32_t* best;      // [batch]
  int32_t* bonus;     // [batch]
  int32_t* resync;    // [batch]
};

// LDS of the walk for NT threads (NT >= n_max, at most CURE_MAX_TREE_NODES).
template <int NT>
struct AcceptLds {
  int link[NT];       // (parent + 1) << 1 | match: one LDS read per walk step
  int tgt[NT];        // the target's argmax at each node
  int repair[NT];     // the node's root path holds a repair node
  int bad;
  int key[NT > kWave ? NT / kWave : 1];
};

// Orders one thread's LDS writes before other threads' later reads. Across a
// workgroup that is a barrier. Inside one wave the LDS executes the wave's
// instructions in issue order, so only the compiler must keep program order
// (a wavefront-scope fence, which emits no instruction).
template <bool kOneWave>
CURE_DEV void walk_sync() {
  if (kOneWave) {
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
  } else {
    __syncthreads();
  }
}

// Sequence b's walk by NT threads: the whole workgroup, or (kOneWave, NT = 64)
// a single wave of it. Before the call the caller has written s.tgt[i] for
// every i < n_max (the call's first sync publishes it); the thread standing
// for node n (n = 0 .. NT - 1) passes n, node n's parent p and token tok
// (anything for n >= n_max), and every participating thread the sequence's
// node count nn and root_tgt. Every participating thread must make the call.
template <int NT, bool kOneWave, int NL>
CURE_DEV void accept_walk(AcceptLds<NL>& s, int n, int b, int p, int tok, int nn, int root_tgt,
                          int n_max, int chain_len, const AcceptOut& out) {
  static_assert(!kOneWave || NT == kWave, "a one-wave walk has 64 threads");
  static_assert(NT <= NL, "LDS arrays cover every thread");
  constexpr int kMaxNodes = CURE_MAX_TREE_NODES;
  const int64_t row = (int64_t)b * n_max;
  const int N = min(max(nn, 0), n_max);
  if (n == 0) s.bad = (nn < 0 || nn > n_max);
  walk_sync<kOneWave>();
  if (n < N) {
    const bool valid = p >= -1 && p < n;
    if (!valid) s.bad = 1;
    // The argmax is read only through a validated parent index.
    const int want = p < 0 ? root_tgt : (valid ? s.tgt[p] : root_tgt);
    s.link[n] = ((valid ? p + 1 : 0) << 1) | (tok == want ? 1 : 0);
  }
  walk_sync<kOneWave>();

  if (s.bad) {
    for (int i = n; i < n_max; i += NT) out.path[row + i] = -1;
    if (n == 0) {
      out.acc_len[b] = -1;
      out.best[b] = -1;
      out.bonus[b] = root_tgt;
      out.resync[b] = -1;
    }
    return;
  }

  // Own path: accepted iff every node on it matches; depth = its length - 1;
  // repair iff it holds a node at or past the chain.
  int key = -1;
  if (n < N) {
    bool ok = true;
    int depth = 0, repair = 0;
    for (int j = n;;) {
      const int link = s.link[j];
      if (!(link & 1)) {
        ok = false;
        break;
      }
      repair |= j >= chain_len;
      const int up = (link >> 1) - 1;
      if (up < 0) break;
      j = up;
      ++depth;
    }
    s.repair[n] = repair;
    if (ok) key = (depth << 8) | (kMaxNodes - 1 - n);   // larger depth, then lower index
  }
  key = wave_max(key);
  if (NT > kWave && (n & (kWave - 1)) == 0) s.key[n / kWave] = key;
  walk_sync<kOneWave>();
  int top = key;
  if (NT > kWave) {
    top = s.key[0];
#pragma unroll
    for (int w = 1; w < NT / kWave; ++w) top = max(top, s.key[w]);
  }

  const int win = top < 0 ? -1 : (kMaxNodes - 1 - (top & 0xff));
  const int len = top < 0 ? 0 : (top >> 8) + 1;
  // path[i] for i < len is the ancestor of win at depth i; the rest is -1.
  for (int i = n; i < n_max; i += NT) {
    int v = -1;
    if (i < len) {
      int j = win;
      for (int up = len - 1 - i; up > 0; --up) j = (s.link[j] >> 1) - 1;
      v = j;
    }
    out.path[row + i] = v;
  }
  if (n == 0) {
    out.acc_len[b] = len;
    out.best[b] = win;
    out.bonus[b] = win < 0 ? root_tgt : s.tgt[win];
    out.resync[b] = win < 0 ? 0 : s.repair[win];
  }
}

}  // namespace cure
