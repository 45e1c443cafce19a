// cure_margins: one streaming pass over each logits row computing the top-1 /
// top-2 entries, the log-sum-exp and the predictive confidence margin
// (Sec. 3.3, Eq. 2), plus the UFP selection of Algorithm 1 as an epilogue.
//
// Work decomposition: each row is cut into `splits` contiguous chunks, one
// 256-thread workgroup per (row, chunk). A lane reads 16-byte vectors of 8
// entries and keeps an online log-sum-exp plus its two best vectors ranked by
// (vector maximum descending, position ascending). The top-2 entries of any
// set of vectors always lie in its two best vectors: the top-1 sits in the
// first vector holding the largest value, and the top-2 is either beside it or
// is the maximum of the best other vector. So the streaming loop tracks only
// each lane's two best records -- a record is a vector, or for long chunks a
// loop step's two vectors -- as maxima and positions, branch-free; at the end
// the wave merges its lanes' records, rereads the entries of its own two best
// records (one per lane) and ranks them exactly (value descending, index
// ascending).
//
// With one chunk per row the workgroup writes the row's results itself. With
// several, chunk results go to the workspace and margins_finish (one workgroup
// per sequence) merges them with an associative (value desc, index asc) top-2
// merge; the same kernel runs the UFP selection and, for cure_margins_accept,
// the acceptance walk over the rows' argmaxes (Eq. 1, Eq. 4). Workgroups never wait on each
// other inside a kernel: on a multi-die GPU the device-scope fences such a
// hand-off needs cost far more than a second, tiny launch.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>

#include "accept_walk.hpp"
#include "common.hpp"
#include "host_util.hpp"

namespace cure {
namespace {

constexpr int kThreads = 256;
constexpr int kVec = 8;            // entries per lane per vector step
constexpr int kUnroll = 2;         // vector steps per lane per loop step
// Chunks of at least this many loop steps track their best records per loop
// step (two vectors) rather than per vector; see margins_kernel.
constexpr int kStepRecordIters = 8;
static_assert(kUnroll == 2, "a step record covers a loop step's two vectors");
constexpr int kMaxSplits = 32;
constexpr int kMinChunk = 8192;    // entries per workgroup, about
constexpr int kTargetWgsPerCu = 2;
constexpr int kMaxGateChain = 1024;
constexpr float kRescaleAt = 16.f; // re-reference the exp sum when a value exceeds ref + 16

struct Partial {
  float ref, sum, v1, v2;
  int32_t i1, i2, pad0, pad1;
};
static_assert(sizeof(Partial) == 32, "partial record is 32 bytes");

struct Args {
  const void* logits;
  int64_t ld;
  int32_t rows, vocab, splits, chunk, iters;
  float* top1_val;
  int32_t* top1_idx;
  float* top2_val;
  int32_t* top2_idx;
  float* lse;
  float* margin;
  int32_t chain_len, max_ufp;
  float tau;
  int32_t* ufp_pos;
  int32_t* ufp_cnt;
  Partial* partials;     // [rows total][splits], only when splits > 1
  // Acceptance epilogue (cure_margins_accept; acc.acc_len == nullptr: none).
  // The rows of a sequence are its tree's nodes, row n = node n.
  const int32_t* parent;
  const int32_t* token;
  const int32_t* root_tgt;
  const int32_t* n_nodes;
  int32_t acc_chain;
  AcceptOut acc;
};

// Raw buffer loads: the chunk is described by a buffer resource (base, size)
// and every load carries a 32-bit per-lane offset, so the loop carries no
// 64-bit address arithmetic. The hardware range-checks the per-lane (VGPR)
// offset against the resource size -- the scalar offset operand is not
// checked, so it is always 0 here -- and reads at or past the size return zero
// without touching memory.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
constexpr int kRsrcWord3 = 0x00020000;   // raw (untyped) 32-bit access, gfx9 family
constexpr int kNonTemporal = 2;          // cache-policy bit: streaming data, read once

CURE_DEV __amdgpu_buffer_rsrc_t chunk_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, kRsrcWord3);
}

// One lane's 8 entries as raw registers, then widened.
template <typename T>
struct Raw8;
template <>
struct Raw8<uint16_t> {
  u32x4 w;
  CURE_DEV void load(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    w = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, kNonTemporal);
  }
  static constexpr uint32_t kBytes = 16;
  CURE_DEV void widen(float (&f)[kVec]) const {
    f[0] = bf16_lo(w.x); f[1] = bf16_hi(w.x);
    f[2] = bf16_lo(w.y); f[3] = bf16_hi(w.y);
    f[4] = bf16_lo(w.z); f[5] = bf16_hi(w.z);
    f[6] = bf16_lo(w.w); f[7] = bf16_hi(w.w);
  }
};
template <>
struct Raw8<float> {
  u32x4 a, b;
  CURE_DEV void load(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    a = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, kNonTemporal);
    b = __builtin_amdgcn_raw_buffer_load_b128(r, (int)(off + 16), 0, kNonTemporal);
  }
  static constexpr uint32_t kBytes = 32;
  CURE_DEV void widen(float (&f)[kVec]) const {
    f[0] = __uint_as_float(a.x); f[1] = __uint_as_float(a.y);
    f[2] = __uint_as_float(a.z); f[3] = __uint_as_float(a.w);
    f[4] = __uint_as_float(b.x); f[5] = __uint_as_float(b.y);
    f[6] = __uint_as_float(b.z); f[7] = __uint_as_float(b.w);
  }
};

// Three-input maximum on the VALU. The inputs are never NaN (the interface
// excludes NaN logits), so no quieting of the operands is needed.
CURE_DEV float max3(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// Two-input maximum and minimum on the VALU, without the operand quieting
// fmaxf/fminf add for values of unknown origin (the inputs are never NaN).
CURE_DEV float max_raw(float a, float b) {
  float r;
  asm("v_max_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}
CURE_DEV float min_raw(float a, float b) {
  float r;
  asm("v_min_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}

CURE_DEV float max8(const float (&f)[kVec]) {
  return max3(max3(f[0], f[1], f[2]), max3(f[3], f[4], f[5]), max3(f[6], f[7], f[7]));
}

// Wave-wide maximum (float) and minimum (int), every lane getting the result:
// DPP stages 1-8, then the 16- and 32-lane swaps, all on the VALU.
CURE_DEV float wave_max_raw(float x) {
  x = max_raw(x, partner<1>(x));
  x = max_raw(x, partner<2>(x));
  x = max_raw(x, partner<4>(x));
  x = max_raw(x, partner<8>(x));
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = max_raw(__uint_as_float(r[0]), __uint_as_float(r[1]));
  const auto q = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return max_raw(__uint_as_float(q[0]), __uint_as_float(q[1]));
}
CURE_DEV int wave_min_int(int x) {
  x = min(x, partner<1>(x));
  x = min(x, partner<2>(x));
  x = min(x, partner<4>(x));
  x = min(x, partner<8>(x));
  const auto r = __builtin_amdgcn_permlane16_swap((unsigned)x, (unsigned)x, false, false);
  x = min((int)r[0], (int)r[1]);
  const auto q = __builtin_amdgcn_permlane32_swap((unsigned)x, (unsigned)x, false, false);
  return min((int)q[0], (int)q[1]);
}

// The wave's top 2 (value descending, index ascending) when each lane's own
// pair is ordered -- (v1, i1) beats (v2, i2) -- and real indices are unique
// across lanes: first the best of the lanes' first entries, then the best of
// the other lanes' first entries and the winner's second. Four scalar
// reductions instead of a butterfly of whole records. With no real entry
// anywhere every lane is a "winner" and both results are the empty slot.
CURE_DEV Top2 top2_wave_ordered(const Top2& t) {
  const float m1 = wave_max_raw(t.v1);
  const int i1 = wave_min_int(t.v1 == m1 ? t.i1 : INT32_MAX);
  const bool win = t.v1 == m1 && t.i1 == i1;
  const float cv = win ? t.v2 : t.v1;
  const int ci = win ? t.i2 : t.i1;
  const float m2 = wave_max_raw(cv);
  const int i2 = wave_min_int(cv == m2 ? ci : INT32_MAX);
  return {m1, m2, i1, i2};
}

template <typename T>
CURE_DEV float load1(const T* p);
template <>
CURE_DEV float load1<uint16_t>(const uint16_t* p) { return bf16_to_f32(*p); }
template <>
CURE_DEV float load1<float>(const float* p) { return *p; }

CURE_DEV void write_row(const Args& a, int row, const Top2& t, float lse) {
  a.top1_val[row] = t.v1;
  a.top1_idx[row] = t.i1;
  a.top2_val[row] = t.v2;
  a.top2_idx[row] = t.i2;
  a.lse[row] = lse;
  a.margin[row] = t.v1 - t.v2;
}

// UFP selection for sequence b: candidates m < tau, ranked by (m, position).
// sm holds the sequence's first chain_len margins (LDS, filled by the caller).
CURE_DEV void select_ufp(const Args& a, int b, const float* sm) {
  const int K = a.chain_len;
  int local = 0;
  for (int i = threadIdx.x; i < K; i += kThreads) {
    const float mi = sm[i];
    if (!(mi < a.tau)) continue;
    ++local;
    int rank = 0;
    for (int j = 0; j < K; ++j) {
      const float mj = sm[j];
      rank += (mj < a.tau) && (mj < mi || (mj == mi && j < i));
    }
    if (rank < a.max_ufp) a.ufp_pos[(int64_t)b * K + rank] = i;
  }
  // Count candidates across the block.
  __shared__ int s_cnt;
  if (threadIdx.x == 0) s_cnt = 0;
  __syncthreads();
  if (local) atomicAdd(&s_cnt, local);
  __syncthreads();
  const int cnt = min(s_cnt, a.max_ufp);
  for (int p = cnt + threadIdx.x; p < K; p += kThreads) a.ufp_pos[(int64_t)b * K + p] = -1;
  if (threadIdx.x == 0) a.ufp_cnt[b] = cnt;
}

// The same selection by one wave, for chain_len <= 64: lane i ranks position i
// and the candidates are counted with a ballot, so no barrier is needed.
CURE_DEV void select_ufp_wave(const Args& a, int b, const float* sm) {
  const int K = a.chain_len;
  const int i = threadIdx.x % kWave;
  const float mi = i < K ? sm[i] : 0.f;
  const bool cand = i < K && mi < a.tau;
  int rank = 0;
  if (cand)
    for (int j = 0; j < K; ++j) {
      const float mj = sm[j];
      rank += (mj < a.tau) && (mj < mi || (mj == mi && j < i));
    }
  const int cnt = min((int)__popcll(__ballot(cand)), a.max_ufp);
  if (cand && rank < a.max_ufp) a.ufp_pos[(int64_t)b * K + rank] = i;
  for (int q = cnt + i; q < K; q += kWave) a.ufp_pos[(int64_t)b * K + q] = -1;
  if (i == 0) a.ufp_cnt[b] = cnt;
}

template <typename T, bool kVecPath, bool kStepRecords>
__global__ __launch_bounds__(kThreads) void margins_kernel(Args a) {
  __shared__ Top2 s_top[kThreads / kWave];
  __shared__ Lse s_lse[kThreads / kWave];

  const int row = blockIdx.x / a.splits;
  const int split = blockIdx.x - row * a.splits;
  const T* x = reinterpret_cast<const T*>(a.logits) + (int64_t)row * a.ld;
  const int begin = split * a.chunk;
  const int end = min(a.vocab, begin + a.chunk);
  const int tid = threadIdx.x;

  Top2 t = top2_empty();
  float ref = kLseEmptyRef, sum = 0.f;
  float nref = -ref * kLog2e;

  int scalar_from = begin;
  // The lane's two best records (vectors, or loop steps when kStepRecords):
  // their maxima and positions, in vectors, within the chunk (-1 = none). A
  // lane's first record is taken as its best even if it is all -inf, so a lane
  // with data always has one; positions arrive in ascending order, so strict
  // comparisons keep the first record attaining each maximum. Per-step records
  // save about half of the tracking's VALU work per vector, and their reread is
  // twice as wide: they pay on long chunks (ragged batch 40.5 -> 39.8 us per
  // call) and cost on short ones (default step 12.14 -> 12.32).
  float bm1 = -INFINITY, bm2 = -INFINITY;
  int bv1 = -1, bv2 = -1;
  const int nvec = kVecPath ? (end - begin) / kVec : 0;
  if (kVecPath) {
    scalar_from = begin + nvec * kVec;
    if (nvec > 0) {
      // Lanes past the chunk's last vector read zeros (outside the buffer
      // resource) and ignore them, so every load is unconditional. Two register
      // sets alternate: one step's loads are in flight while the previous step
      // is processed. Steps in which every lane's vectors lie inside the chunk
      // run without per-vector range checks; only the last step checks.
      const __amdgpu_buffer_rsrc_t rsrc = chunk_rsrc(x + begin, (uint32_t)nvec * Raw8<T>::kBytes);
      const uint32_t lane_off = (uint32_t)tid * Raw8<T>::kBytes;
      const int full_iters = nvec / (kUnroll * kThreads);
      Raw8<T> ra[kUnroll], rb[kUnroll];
      auto issue = [&](Raw8<T>(&r)[kUnroll], int it) {
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
          r[u].load(rsrc, lane_off + (uint32_t)((it * kUnroll + u) * kThreads) * Raw8<T>::kBytes);
      };
      auto process = [&](const Raw8<T>(&r)[kUnroll], int it, bool checked) {
        float f[kUnroll][kVec], m8[kUnroll];
        float step_max = -INFINITY;
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
          const int v = (it * kUnroll + u) * kThreads + tid;
          const bool ok = !checked || v < nvec;
          r[u].widen(f[u]);
          m8[u] = ok ? max8(f[u]) : -INFINITY;
          if (!kStepRecords) {
            // Best-two-records update, a record per vector (values by max/min,
            // positions by select).
            const bool c1 = ok && (m8[u] > bm1 || bv1 < 0);
            const bool c2 = ok && m8[u] > bm2;
            bv2 = c1 ? bv1 : (c2 ? v : bv2);
            bv1 = c1 ? v : bv1;
            bm2 = max_raw(bm2, min_raw(m8[u], bm1));
            bm1 = max_raw(bm1, m8[u]);
          }
          step_max = max_raw(step_max, m8[u]);
        }
        if (kStepRecords) {
          // One record for the step's two vectors: their maximum, positioned at
          // the first of them that attains it, so that records compare exactly
          // as those vectors do under (maximum descending, position ascending).
          const int v0 = it * kUnroll * kThreads + tid;
          const bool ok = !checked || v0 < nvec;
          const int pos = m8[0] == step_max ? v0 : v0 + kThreads;
          const bool c1 = ok && (step_max > bm1 || bv1 < 0);
          const bool c2 = ok && step_max > bm2;
          bv2 = c1 ? bv1 : (c2 ? pos : bv2);
          bv1 = c1 ? pos : bv1;
          bm2 = max_raw(bm2, min_raw(step_max, bm1));
          bm1 = max_raw(bm1, step_max);
        }
        // Log-sum-exp against a lagging reference, moved only on large jumps
        // (checked once per step, before the step's terms are added).
        const bool resc = step_max > ref + kRescaleAt;
        if (__builtin_expect(__ballot(resc) != 0, 0)) {
          if (resc) {
            sum *= fast_exp2((ref - step_max) * kLog2e);
            ref = step_max;
            nref = -ref * kLog2e;
          }
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
          const int v = (it * kUnroll + u) * kThreads + tid;
          if (!checked || v < nvec) {
            // Exponentials are never negative, so starting each partial sum at
            // its first term gives the same bits as starting at zero.
            float s0 = fast_exp2(fmaf(f[u][0], kLog2e, nref));
            float s1 = fast_exp2(fmaf(f[u][1], kLog2e, nref));
#pragma unroll
            for (int j = 2; j < kVec; j += 2) {
              s0 += fast_exp2(fmaf(f[u][j], kLog2e, nref));
              s1 += fast_exp2(fmaf(f[u][j + 1], kLog2e, nref));
            }
            sum += s0 + s1;
          }
        }
      };
      // Prefetches past the last step fall outside the resource and read zeros,
      // so they need no guard and the waits before each step stay partial.
      issue(ra, 0);
      int it = 0;
      for (; it + 1 < full_iters; it += 2) {
        issue(rb, it + 1);
        process(ra, it, false);
        issue(ra, it + 2);
        process(rb, it + 1, false);
      }
      // At most two steps remain (ra holds step `it`): one full or checked
      // step, then possibly a checked one.
      if (it < a.iters) {
        issue(rb, it + 1);
        process(ra, it, it >= full_iters);
        if (it + 1 < a.iters) process(rb, it + 1, true);
      }
    }
  }
  for (int i = scalar_from + tid; i < end; i += kThreads) {
    const float xv = load1<T>(x + i);
    top2_push(t, xv, i);
    if (xv > ref + kRescaleAt) {
      sum *= fast_exp2((ref - xv) * kLog2e);
      ref = xv;
      nref = -ref * kLog2e;
    }
    sum += fast_exp2(fmaf(xv, kLog2e, nref));
  }

  // The wave's top-2 entries lie in its two best vectors (by maximum
  // descending, position ascending) together with the lanes' scalar-tail
  // entries. The lanes' vector records are merged first (positions as indices;
  // "none" is (-inf, INT32_MAX), which every real vector beats); then lanes
  // 0-7 reread the entries of the best vector and lanes 8-15 those of the
  // second, one entry per lane, so that each lane adds a single entry to its
  // own top 2. The log-sum-exp reduction runs while the reads are in flight.
  // Every lane's top 2 is ordered and its indices are its own, so the wave
  // reductions take the ordered form.
  const int lane = tid & (kWave - 1);
  int mine = INT32_MAX;                          // entry index within the chunk
  uint32_t raw = 0;
  if (kVecPath) {
    const Top2 bv = top2_wave_ordered(Top2{bm1, bm2, bv1 < 0 ? INT32_MAX : bv1,
                                           bv2 < 0 ? INT32_MAX : bv2});
    int pick = INT32_MAX;                        // the vector this lane rereads from
    if (kStepRecords) {
      // Lanes 0-15 reread the best record's two vectors, lanes 16-31 the
      // second's; a vector past the chunk's last holds nothing.
      const int rec = lane < 2 * kVec ? bv.i1 : (lane < 4 * kVec ? bv.i2 : INT32_MAX);
      if (rec != INT32_MAX) {
        const int v0 = rec / (kUnroll * kThreads) * (kUnroll * kThreads) + rec % kThreads;
        const int vec = v0 + ((lane / kVec) & 1) * kThreads;
        if (vec < nvec) pick = vec;
      }
    } else {
      pick = lane < kVec ? bv.i1 : (lane < 2 * kVec ? bv.i2 : INT32_MAX);
    }
    if (pick != INT32_MAX) {
      mine = pick * kVec + (lane & (kVec - 1));
      const __amdgpu_buffer_rsrc_t r1 = chunk_rsrc(x + begin, (uint32_t)nvec * Raw8<T>::kBytes);
      if (sizeof(T) == 2)
        raw = __builtin_amdgcn_raw_buffer_load_b16(r1, mine * 2, 0, kNonTemporal);
      else
        raw = __builtin_amdgcn_raw_buffer_load_b32(r1, mine * 4, 0, kNonTemporal);
    }
  }
  Lse s = lse_wave_reduce(Lse{ref, sum});
  if (kVecPath && mine != INT32_MAX)
    top2_push(t, sizeof(T) == 2 ? bf16_to_f32((uint16_t)raw) : __uint_as_float(raw), begin + mine);

  // Workgroup reduction.
  t = top2_wave_ordered(t);
  const int wave = tid / kWave;
  if ((tid & (kWave - 1)) == 0) { s_top[wave] = t; s_lse[wave] = s; }
  __syncthreads();

  // Chunk result of this workgroup (thread 0 combines the wave results).
  if (tid == 0) {
    Top2 bt = s_top[0];
    Lse bs = s_lse[0];
#pragma unroll
    for (int w = 1; w < kThreads / kWave; ++w) {
      bt = top2_merge(bt, s_top[w]);
      bs = lse_merge(bs, s_lse[w]);
    }
    if (a.splits > 1) {
      a.partials[(int64_t)row * a.splits + split] =
          Partial{bs.ref, bs.sum, bt.v1, bt.v2, bt.i1, bt.i2, 0, 0};
    } else {
      write_row(a, row, bt, lse_value(bs));
    }
  }
}

// Per sequence: merge each row's chunk results (when rows were split), then
// select the sequence's UFPs from its chain rows' margins.
//
// Eight lanes per row: lane k of a row's group loads chunk results k, k + 8,
// k + 16, k + 24 (all at once, one memory round trip), merges them, and the
// group combines its eight results through VALU lane exchanges. The chain
// rows' margins go to LDS as they are produced, so the gate needs no second
// trip to memory.
constexpr int kFinishGroup = 8;
constexpr int kFinishPerLane = kMaxSplits / kFinishGroup;
static_assert(kMaxSplits % kFinishGroup == 0, "chunk results split evenly over a row's lanes");

__global__ __launch_bounds__(kThreads) void margins_finish(Args a) {
  __shared__ float s_margin[kMaxGateChain];
  __shared__ AcceptLds<kThreads> s_acc;
  const int b = blockIdx.x;
  const bool accept = a.acc.acc_len != nullptr;
  // Chains of up to 64 rows (and trees of up to 64 nodes): after the merge,
  // wave 0 runs the gate and wave 1 the acceptance walk, side by side and
  // without barriers.
  const bool by_waves = a.chain_len <= kWave && (!accept || a.rows <= kWave);
  const int wave = threadIdx.x / kWave;
  // The tree's arrays are loaded before the chunk results are merged, by the
  // thread standing for each node.
  const int node = by_waves ? (int)threadIdx.x - kWave : (int)threadIdx.x;
  int par = -1, tok = 0, nn = 0, root = 0;
  if (accept) {
    const int64_t row = (int64_t)b * a.rows;
    nn = a.n_nodes[b];
    root = a.root_tgt[b];
    if (node >= 0 && node < a.rows) {
      par = a.parent[row + node];
      tok = a.token[row + node];
    }
  }
  if (a.splits > 1) {
    constexpr int kRowsPerPass = kThreads / kFinishGroup;
    const int k = threadIdx.x % kFinishGroup;
    // Every lane runs the same number of passes: the lane exchanges below
    // need all eight lanes of a group active.
    for (int r0 = 0; r0 < a.rows; r0 += kRowsPerPass) {
      const int r = r0 + threadIdx.x / kFinishGroup;
      const bool live = r < a.rows;
      const Partial* p = a.partials + ((int64_t)b * a.rows + (live ? r : 0)) * a.splits;
      Partial q[kFinishPerLane];
#pragma unroll
      for (int u = 0; u < kFinishPerLane; ++u) {
        const int sp = k + u * kFinishGroup;
        q[u] = Partial{kLseEmptyRef, 0.f, -INFINITY, -INFINITY, INT32_MAX, INT32_MAX, 0, 0};
        if (live && sp < a.splits) q[u] = p[sp];
      }
      Top2 t{q[0].v1, q[0].v2, q[0].i1, q[0].i2};
      Lse ls{q[0].ref, q[0].sum};
#pragma unroll
      for (int u = 1; u < kFinishPerLane; ++u) {
        t = top2_merge(t, Top2{q[u].v1, q[u].v2, q[u].i1, q[u].i2});
        ls = lse_merge(ls, Lse{q[u].ref, q[u].sum});
      }
      t = top2_stage<1>(t);
      t = top2_stage<2>(t);
      t = top2_stage<4>(t);
      ls = lse_stage<1>(ls);
      ls = lse_stage<2>(ls);
      ls = lse_stage<4>(ls);
      if (live && k == 0) {
        write_row(a, b * a.rows + r, t, lse_value(ls));
        if (r < a.chain_len) s_margin[r] = t.v1 - t.v2;
        if (accept) s_acc.tgt[r] = t.i1;
      }
    }
  } else {
    if (a.ufp_pos)
      for (int i = threadIdx.x; i < a.chain_len; i += kThreads)
        s_margin[i] = a.margin[(int64_t)b * a.rows + i];
    if (accept)
      for (int i = threadIdx.x; i < a.rows; i += kThreads)
        s_acc.tgt[i] = a.top1_idx[(int64_t)b * a.rows + i];
  }
  if (by_waves) {
    __syncthreads();                     // the margins and argmaxes are in LDS
    if (wave == 0 && a.ufp_pos) select_ufp_wave(a, b, s_margin);
    if (wave == 1 && accept)
      accept_walk<kWave, true>(s_acc, node, b, par, tok, nn, root, a.rows, a.acc_chain, a.acc);
    return;
  }
  if (a.ufp_pos) {
    __syncthreads();
    select_ufp(a, b, s_margin);
  }
  if (accept)
    accept_walk<kThreads, false>(s_acc, node, b, par, tok, nn, root, a.rows, a.acc_chain, a.acc);
}

// Scratch of the allocation-free entry point: the chunk results of one call
// (32 bytes per row and chunk). The library's code object holds one copy per
// GPU it is loaded on, for the life of the process; host code reaches it only
// through the address hipGetSymbolAddress returns for the current device.
constexpr size_t kScratchBytes = 256 * 1024;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

struct Plan {
  int splits, chunk;
};

// Enough workgroups to cover the GPU kTargetWgsPerCu times over, with chunks
// of about kMinChunk entries or more: at most ceil(vocab / kMinChunk) splits,
// so a small batch's chunk fits one loop step of each register set (all its
// loads in flight at once).
Plan make_plan(int64_t nrow, int32_t vocab) {
  int splits = (int)((kTargetWgsPerCu * (int64_t)device_cu_count() + nrow - 1) / nrow);
  splits = std::max(1, std::min(splits, std::min(kMaxSplits, (vocab + kMinChunk - 1) / kMinChunk)));
  int chunk = (vocab + splits - 1) / splits;
  chunk = (chunk + kVec - 1) / kVec * kVec;
  splits = (vocab + chunk - 1) / chunk;
  return Plan{splits, chunk};
}

// Host-side argument checks shared by both entry points.
cure_status check_args(const void* logits, int32_t dtype, int32_t batch, int32_t rows,
                       int32_t vocab, int64_t ld, const float* top1_val,
                       const int32_t* top1_idx, const float* top2_val,
                       const int32_t* top2_idx, const float* lse, const float* margin,
                       int32_t chain_len, int32_t repair_budget, int32_t branch_depth,
                       const int32_t* ufp_pos, const int32_t* ufp_cnt) {
  if (dtype != CURE_F32 && dtype != CURE_BF16) return CURE_ERR_INVALID_ARG;
  if (batch < 0 || rows < 0) return CURE_ERR_INVALID_ARG;
  if (batch == 0 || rows == 0) return CURE_OK;
  if (vocab < 2 || ld < vocab) return CURE_ERR_INVALID_ARG;
  if (!logits || !top1_val || !top1_idx || !top2_val || !top2_idx || !lse || !margin)
    return CURE_ERR_INVALID_ARG;
  const bool gate = ufp_pos != nullptr || ufp_cnt != nullptr;
  if (gate) {
    if (!ufp_pos || !ufp_cnt) return CURE_ERR_INVALID_ARG;
    if (chain_len < 1 || chain_len > rows || branch_depth < 1 || repair_budget < 0)
      return CURE_ERR_INVALID_ARG;
    if (chain_len > kMaxGateChain) return CURE_ERR_UNSUPPORTED;
  }
  if ((int64_t)batch * rows > INT32_MAX / kMaxSplits) return CURE_ERR_UNSUPPORTED;
  return CURE_OK;
}

// The acceptance walk's inputs and outputs (cure_margins_accept).
struct AcceptIn {
  const int32_t* parent;
  const int32_t* token;
  const int32_t* root_tgt;
  const int32_t* n_nodes;
  AcceptOut out;
};

// Launches the pass; `partials` holds the plan's chunk results (nrow * splits
// records) when rows are split; `acc` (or nullptr) adds the acceptance walk.
// The arguments have passed check_args.
cure_status launch(const void* logits, int32_t dtype, int32_t batch, int32_t rows,
                   int32_t vocab, int64_t ld, float* top1_val, int32_t* top1_idx,
                   float* top2_val, int32_t* top2_idx, float* lse, float* margin,
                   int32_t chain_len, float tau, int32_t repair_budget, int32_t branch_depth,
                   int32_t* ufp_pos, int32_t* ufp_cnt, const Plan& pl, void* partials,
                   const AcceptIn* acc, void* stream) {
  const bool gate = ufp_pos != nullptr;
  const int64_t nrow = (int64_t)batch * rows;
  const size_t esize = dtype == CURE_F32 ? 4 : 2;
  const bool vec_ok = (reinterpret_cast<uintptr_t>(logits) % 16 == 0) &&
                      ((size_t)ld * esize) % 16 == 0;

  Args a;
  a.logits = logits;
  a.ld = ld;
  a.rows = rows;
  a.vocab = vocab;
  a.splits = pl.splits;
  a.chunk = pl.chunk;
  const int per_iter = kThreads * kVec * kUnroll;
  a.iters = (pl.chunk + per_iter - 1) / per_iter;
  a.top1_val = top1_val;
  a.top1_idx = top1_idx;
  a.top2_val = top2_val;
  a.top2_idx = top2_idx;
  a.lse = lse;
  a.margin = margin;
  a.chain_len = gate ? chain_len : 0;
  a.max_ufp = gate ? repair_budget / branch_depth : 0;
  a.tau = tau;
  a.ufp_pos = gate ? ufp_pos : nullptr;
  a.ufp_cnt = gate ? ufp_cnt : nullptr;
  a.partials = reinterpret_cast<Partial*>(partials);
  a.parent = acc ? acc->parent : nullptr;
  a.token = acc ? acc->token : nullptr;
  a.root_tgt = acc ? acc->root_tgt : nullptr;
  a.n_nodes = acc ? acc->n_nodes : nullptr;
  a.acc_chain = chain_len;
  a.acc = acc ? acc->out : AcceptOut{nullptr, nullptr, nullptr, nullptr, nullptr};

  const dim3 grid((unsigned)(nrow * pl.splits)), block(kThreads);
  hipStream_t s = as_stream(stream);
  const bool step_records = a.iters >= kStepRecordIters;
  if (dtype == CURE_BF16) {
    if (!vec_ok) hipLaunchKernelGGL((margins_kernel<uint16_t, false, false>), grid, block, 0, s, a);
    else if (step_records) hipLaunchKernelGGL((margins_kernel<uint16_t, true, true>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((margins_kernel<uint16_t, true, false>), grid, block, 0, s, a);
  } else {
    if (!vec_ok) hipLaunchKernelGGL((margins_kernel<float, false, false>), grid, block, 0, s, a);
    else if (step_records) hipLaunchKernelGGL((margins_kernel<float, true, true>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((margins_kernel<float, true, false>), grid, block, 0, s, a);
  }
  if (hipGetLastError() != hipSuccess) return CURE_ERR_HIP;
  if (pl.splits > 1 || gate || acc)
    hipLaunchKernelGGL(margins_finish, dim3(batch), block, 0, s, a);
  return launch_status();
}

// Device address of `scratch` on the current device, looked up once per
// device (each GPU holds its own copy of the array at its own address).
void* scratch_address() {
  static std::mutex mu;
  static void* cached[64] = {nullptr};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  std::lock_guard<std::mutex> lock(mu);
  if (!cached[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
    cached[dev] = p;
  }
  return cached[dev];
}

}  // namespace
}  // namespace cure

using namespace cure;

extern "C" size_t cure_margins_workspace_size(int32_t batch, int32_t rows, int32_t vocab) {
  (void)vocab;
  if (batch <= 0 || rows <= 0) return 0;
  return align_up((size_t)batch * rows * kMaxSplits * sizeof(Partial), 256);
}

extern "C" cure_status cure_margins(const void* logits, int32_t dtype, int32_t batch,
                                    int32_t rows, int32_t vocab, int64_t ld, float* top1_val,
                                    int32_t* top1_idx, float* top2_val, int32_t* top2_idx,
                                    float* lse, float* margin, int32_t chain_len, float tau,
                                    int32_t repair_budget, int32_t branch_depth,
                                    int32_t* ufp_pos, int32_t* ufp_cnt, void* workspace,
                                    size_t workspace_bytes, void* stream) {
  const cure_status st = check_args(logits, dtype, batch, rows, vocab, ld, top1_val, top1_idx,
                                    top2_val, top2_idx, lse, margin, chain_len, repair_budget,
                                    branch_depth, ufp_pos, ufp_cnt);
  if (st != CURE_OK || batch == 0 || rows == 0) return st;
  const Plan pl = make_plan((int64_t)batch * rows, vocab);
  if (pl.splits > 1 &&
      (!workspace || workspace_bytes < cure_margins_workspace_size(batch, rows, vocab)))
    return CURE_ERR_WORKSPACE;
  return launch(logits, dtype, batch, rows, vocab, ld, top1_val, top1_idx, top2_val, top2_idx,
                lse, margin, chain_len, tau, repair_budget, branch_depth, ufp_pos, ufp_cnt, pl,
                workspace, nullptr, stream);
}

extern "C" cure_status cure_margins_accept(
    const void* logits, int32_t dtype, int32_t batch, int32_t rows, int32_t vocab, int64_t ld,
    float* top1_val, int32_t* top1_idx, float* top2_val, int32_t* top2_idx, float* lse,
    float* margin, int32_t chain_len, float tau, int32_t repair_budget, int32_t branch_depth,
    int32_t* ufp_pos, int32_t* ufp_cnt, const int32_t* parent, const int32_t* token,
    const int32_t* root_tgt, const int32_t* n_nodes, int32_t* acc_len, int32_t* path,
    int32_t* best, int32_t* bonus, int32_t* resync, void* workspace, size_t workspace_bytes,
    void* stream) {
  const cure_status st = check_args(logits, dtype, batch, rows, vocab, ld, top1_val, top1_idx,
                                    top2_val, top2_idx, lse, margin, chain_len, repair_budget,
                                    branch_depth, ufp_pos, ufp_cnt);
  if (st != CURE_OK || batch == 0) return st;
  if (chain_len < 0) return CURE_ERR_INVALID_ARG;
  if (!parent || !token || !root_tgt || !n_nodes || !acc_len || !best || !bonus || !resync ||
      (rows > 0 && !path))
    return CURE_ERR_INVALID_ARG;
  if (rows > CURE_MAX_TREE_NODES) return CURE_ERR_UNSUPPORTED;
  if (rows == 0) {
    // No nodes and no rows: nothing is accepted (the walk alone, on empty trees).
    return cure_accept(parent, token, top1_idx, root_tgt, n_nodes, chain_len, batch, 0,
                       acc_len, path, best, bonus, resync, stream);
  }
  const Plan pl = make_plan((int64_t)batch * rows, vocab);
  if (pl.splits > 1 &&
      (!workspace || workspace_bytes < cure_margins_workspace_size(batch, rows, vocab)))
    return CURE_ERR_WORKSPACE;
  const AcceptIn acc{parent, token, root_tgt, n_nodes,
                     AcceptOut{acc_len, path, best, bonus, resync}};
  return launch(logits, dtype, batch, rows, vocab, ld, top1_val, top1_idx, top2_val, top2_idx,
                lse, margin, chain_len, tau, repair_budget, branch_depth, ufp_pos, ufp_cnt, pl,
                workspace, &acc, stream);
}

extern "C" size_t cure_margins_noalloc_scratch_bytes(void) { return kScratchBytes; }

extern "C" cure_status cure_margins_noalloc(const void* logits, int32_t dtype, int32_t batch,
                                            int32_t rows, int32_t vocab, int64_t ld,
                                            float* top1_val, int32_t* top1_idx,
                                            float* top2_val, int32_t* top2_idx, float* lse,
                                            float* margin, int32_t chain_len, float tau,
                                            int32_t repair_budget, int32_t branch_depth,
                                            int32_t* ufp_pos, int32_t* ufp_cnt, void* stream) {
  const cure_status st = check_args(logits, dtype, batch, rows, vocab, ld, top1_val, top1_idx,
                                    top2_val, top2_idx, lse, margin, chain_len, repair_budget,
                                    branch_depth, ufp_pos, ufp_cnt);
  if (st != CURE_OK || batch == 0 || rows == 0) return st;
  const Plan pl = make_plan((int64_t)batch * rows, vocab);
  const size_t need = pl.splits > 1 ? (size_t)batch * rows * pl.splits * sizeof(Partial) : 0;
  if (need > kScratchBytes) return CURE_ERR_UNSUPPORTED;
  void* ws = nullptr;
  if (need > 0) {
    ws = scratch_address();
    if (!ws) return CURE_ERR_HIP;
  }
  return launch(logits, dtype, batch, rows, vocab, ld, top1_val, top1_idx, top2_val, top2_idx,
                lse, margin, chain_len, tau, repair_budget, branch_depth, ufp_pos, ufp_cnt, pl,
                ws, nullptr, stream);
}
