// cure_repair_tree: the budget-aware repair tree of Algorithm 1 and Sec. 3.4,
// with the per-UFP branch budget of Eq. (3).
//
// Two kernels:
//
// topk_chunk -- one 256-thread workgroup per (sequence, UFP slot, 8192-entry
//   chunk of that UFP's logits row). Each lane holds its 32 entries in
//   registers. A lower bound on the chunk's 8th-best value comes almost for
//   free: within a wave, the minimum over eight 8-lane groups of the group
//   maximum is reached by eight distinct entries, so no entry below it can be
//   among the chunk's best eight. The workgroup takes the largest such bound
//   over its waves; each wave appends its entries at or above it to its LDS
//   list (ballot and lane count, no atomics), and every candidate finds its
//   rank by counting the candidates that outrank it. Only when a wave has more
//   than kWaveCap candidates (large runs of equal values) does the workgroup
//   fall back to eight rounds of workgroup-wide selection over the registers.
//   Output: the chunk's best eight (value descending, index ascending) in the
//   workspace.
//
// repair_assemble -- one workgroup per sequence. Eq. (3) on each UFP's margin,
//   then one wave walks the UFPs in order and hands out whole branches while
//   they fit the budget. Each wave takes a UFP row that received branches,
//   writes its branches' suffix nodes, merges the row's chunk results into
//   its best eight and writes the branch roots: the ranked tokens without the
//   draft's own.
//
// The chunk kernel makes the same budget walk up front (from the margins
// alone) and skips the rows of UFPs that the budget leaves without branches.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>

#include "common.hpp"
#include "host_util.hpp"

namespace cure {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kTopK = 8;                 // ranked entries kept per row
constexpr int kVec = 8;                  // entries per 16-byte bf16 vector
constexpr int kLaneVecs = 4;             // vectors per lane per chunk
constexpr int kChunk = kThreads * kVec * kLaneVecs;   // 8192 entries
constexpr int kMaxSplits = 64;
constexpr int kWaveCap = 64;             // LDS candidates per wave
constexpr int kMaxChain = 1024;

// A ranked entry: value and vocabulary index. 8-byte aligned so that one LDS
// access moves a whole record.
struct __attribute__((aligned(8))) Cand {
  float v;
  int i;
};

// (va, ia) ranks before (vb, ib): larger value, or equal value and lower index.
// Written with bitwise operators so that no operand is evaluated lazily (a
// lazy operand becomes a branch around its load).
CURE_DEV bool outranks(float va, int ia, float vb, int ib) {
  return (va > vb) | ((va == vb) & (ia < ib));
}

// Number of set bits of m in lanes below this one.
CURE_DEV int lanes_below(uint64_t m) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                        __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

struct Args {
  const void* logits;
  int64_t ld;
  int32_t batch, rows, vocab, splits, max_slots, chain_len;
  const float* margin;
  const int32_t* ufp_pos;
  const int32_t* ufp_cnt;
  const int32_t* chain_tok;
  const int32_t* suffix;
  int32_t depth, budget, b_min, b_max;
  float scale;
  int32_t n_max;
  int32_t* parent;
  int32_t* token;
  int32_t* n_nodes;
  int32_t* branch_cnt;
  float* part_val;    // [batch][max_slots][splits][kTopK]
  int32_t* part_idx;
};

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
constexpr int kRsrcWord3 = 0x00020000;   // raw (untyped) 32-bit access, gfx9 family

// Range-checked raw buffer over [base, base + bytes): per-lane offsets at or
// past the end read zero without touching memory.
CURE_DEV __amdgpu_buffer_rsrc_t chunk_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, kRsrcWord3);
}

template <typename T>
CURE_DEV float load1(const T* p);
template <>
CURE_DEV float load1<uint16_t>(const uint16_t* p) { return bf16_to_f32(*p); }
template <>
CURE_DEV float load1<float>(const float* p) { return *p; }

// One 8-entry vector at byte offset off of the chunk, widened to float32.
template <typename T>
CURE_DEV void load_vec(__amdgpu_buffer_rsrc_t r, uint32_t off, float (&f)[kVec]);
template <>
CURE_DEV void load_vec<uint16_t>(__amdgpu_buffer_rsrc_t r, uint32_t off, float (&f)[kVec]) {
  const u32x4 w = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0);
  f[0] = bf16_lo(w.x); f[1] = bf16_hi(w.x); f[2] = bf16_lo(w.y); f[3] = bf16_hi(w.y);
  f[4] = bf16_lo(w.z); f[5] = bf16_hi(w.z); f[6] = bf16_lo(w.w); f[7] = bf16_hi(w.w);
}
template <>
CURE_DEV void load_vec<float>(__amdgpu_buffer_rsrc_t r, uint32_t off, float (&f)[kVec]) {
  const u32x4 a = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0);
  const u32x4 b = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off + 16, 0, 0);
  f[0] = __uint_as_float(a.x); f[1] = __uint_as_float(a.y);
  f[2] = __uint_as_float(a.z); f[3] = __uint_as_float(a.w);
  f[4] = __uint_as_float(b.x); f[5] = __uint_as_float(b.y);
  f[6] = __uint_as_float(b.z); f[7] = __uint_as_float(b.w);
}

// The better of (bv, bi) and a partner lane's pair, under (value desc, index asc).
template <int kStage>
CURE_DEV void best_stage(float& bv, int& bi) {
  const float ov = partner<kStage>(bv);
  const int oi = partner<kStage>(bi);
  const bool c = beats(ov, oi, bv, bi);
  bv = c ? ov : bv;
  bi = c ? oi : bi;
}

CURE_DEV void wave_best(float& bv, int& bi) {
  best_stage<1>(bv, bi);
  best_stage<2>(bv, bi);
  best_stage<4>(bv, bi);
  best_stage<8>(bv, bi);
  best_stage<16>(bv, bi);
  best_stage<32>(bv, bi);
}

// Eq. (3): u = clip(1 - m / s, 0, 1), b = clip(round(b_min + u (b_max - b_min)),
// b_min, b_max), each operation rounded once to float32 and round() to the
// nearest even integer. A NaN margin gives u = 0 (fmaxf drops the NaN).
CURE_DEV int branch_budget(float m, float s, int lo, int hi) {
#pragma clang fp contract(off)
  float u = 1.0f - m / s;
  u = fminf(fmaxf(u, 0.0f), 1.0f);
  const float t = (float)lo + u * (float)(hi - lo);
  const int bb = (int)rintf(t);
  return min(max(bb, lo), hi);
}

// Whether the budget walk (the one repair_assemble makes) grants UFP slot
// `slot` of sequence b any branch; false also when this or an earlier slot's
// position lies outside the block (the slot list ends there). Every lane of
// the wave must take part. When even the largest possible grants to the
// earlier slots (b_max branches each) leave room for a branch, and b_min >= 1,
// the answer needs no margins: that saves the dependent read of the margins
// for the first slots. Otherwise each lane evaluates Eq. (3) for one slot and
// the walk reads the results lane by lane.
CURE_DEV bool slot_has_branches(const Args& a, int b, int slot) {
  const int lane = lane_id();
  const int K = a.chain_len;
  const bool sure = a.b_min >= 1 && ((int64_t)slot * a.b_max + 1) * a.depth <= a.budget;
  int remaining = a.budget;
  for (int g0 = 0; g0 <= slot; g0 += kWave) {
    const int s = g0 + lane;
    const int us = s <= slot ? a.ufp_pos[(int64_t)b * K + s] : 0;
    if (__ballot(us < 0 || us >= K)) return false;
    if (sure) continue;
    const int bs = s <= slot ? branch_budget(a.margin[(int64_t)b * a.rows + us], a.scale,
                                             a.b_min, a.b_max)
                             : 0;
    const int last = min(slot - g0, kWave - 1);
    for (int i = 0; i <= last; ++i) {
      const int nb = min(__builtin_amdgcn_readlane(bs, i), remaining / a.depth);
      if (g0 + i == slot) return nb > 0;
      remaining -= nb * a.depth;
    }
  }
  return true;
}

// Rank of the record (mv, mi) among n records in LDS: how many outrank it.
// The records' indices are distinct, so ranks are distinct. All lanes read
// the same record in each step (an LDS broadcast).
CURE_DEV int rank_among(const Cand* c, int n, float mv, int mi) {
  int rank = 0;
#pragma unroll 8
  for (int k = 0; k < n; ++k) {
    const Cand o = c[k];
    rank += outranks(o.v, o.i, mv, mi) ? 1 : 0;
  }
  return rank;
}

// Lane exchanges for merging sorted 8-entry lists held one entry per lane, a
// list in each aligned group of 8 lanes (entry p in lane 8g + p).
//   xor1, xor2     DPP quad permutes
//   xor4           swizzle, lane ^ 4 within 32
//   mirror8        lane 8g + p <-> 8g + 7 - p (DPP half-row mirror)
//   mirror16/32/64 lane i <-> 15 - i / 31 - i / 63 - i within 16 / 32 / 64
//                  (DPP row mirror; swizzle lane ^ 31; that plus permlane32)
enum Xchg { kXor1, kXor2, kXor4, kMirror8, kMirror16, kMirror32, kMirror64 };

template <Xchg kX>
CURE_DEV int xchg(int v) {
  if (kX == kXor1) return __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);
  if (kX == kXor2) return __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);
  if (kX == kXor4) return __builtin_amdgcn_ds_swizzle(v, 0x101F);
  if (kX == kMirror8) return __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false);
  if (kX == kMirror16) return __builtin_amdgcn_update_dpp(0, v, 0x140, 0xF, 0xF, false);
  const int m32 = __builtin_amdgcn_ds_swizzle(v, 0x7C1F);
  if (kX == kMirror32) return m32;
  const auto r = __builtin_amdgcn_permlane32_swap((unsigned)m32, (unsigned)m32, false, false);
  return (int)(lane_id() < 32 ? r[1] : r[0]);
}

// One compare-exchange of a bitonic network: the lane whose position has bit
// kBit clear keeps the better record of itself and its partner, the other
// lane the worse.
template <Xchg kX, int kBit>
CURE_DEV void cmp_xchg(float& v, int& i) {
  const float ov = __int_as_float(xchg<kX>(__float_as_int(v)));
  const int oi = xchg<kX>(i);
  const bool keep_better = (lane_id() & kBit) == 0;
  const bool take = keep_better ? outranks(ov, oi, v, i) : outranks(v, i, ov, oi);
  v = take ? ov : v;
  i = take ? oi : i;
}

// Sorts a bitonic sequence of 8 records held by an 8-lane group, best first.
CURE_DEV void clean8(float& v, int& i) {
  cmp_xchg<kXor4, 4>(v, i);
  cmp_xchg<kXor2, 2>(v, i);
  cmp_xchg<kXor1, 1>(v, i);
}

// The best 8 of two sorted lists, sorted: (v, i) is entry p of one list and
// (ov, oi) entry 7 - p of the other (a mirrored partner), so the better of
// the two forms a bitonic sequence over the group.
CURE_DEV void merge8(float& v, int& i, float ov, int oi) {
  const bool take = outranks(ov, oi, v, i);
  v = take ? ov : v;
  i = take ? oi : i;
  clean8(v, i);
}

// Merges the list of this lane's group with the list of the group mirrored
// across kX; afterwards both groups hold the merged list.
template <Xchg kX>
CURE_DEV void merge_groups(float& v, int& i) {
  merge8(v, i, __int_as_float(xchg<kX>(__float_as_int(v))), xchg<kX>(i));
}

// Appends this lane's record to the wave's LDS list when keep is set, in lane
// order, without atomics: the slot is the wave's running count plus the
// number of keeping lanes below. Records past kWaveCap are dropped but still
// counted. The branch on the ballot is uniform across the wave.
CURE_DEV void wave_append(Cand* list, int& count, bool keep, float v, int i) {
  const uint64_t m = __ballot(keep);
  if (m) {
    const int slot = count + lanes_below(m);
    if (keep && slot < kWaveCap) list[slot] = Cand{v, i};
    count += __popcll(m);
  }
}

template <typename T, bool kVecPath>
__global__ __launch_bounds__(kThreads) void topk_chunk(Args a) {
  __shared__ Cand s_cand[kWaves][kWaveCap];
  __shared__ Cand s_top[kWaves][kTopK];
  __shared__ float s_bound[kWaves];

  // Slot-major order: the budget grants branches to a prefix of each
  // sequence's slots, so the workgroups that find work are dispatched first.
  const int split = blockIdx.x % a.splits;
  const int b = (blockIdx.x / a.splits) % a.batch;
  const int slot = blockIdx.x / (a.splits * a.batch);
  // Unused slots and slots that the budget leaves without branches need no
  // ranking. (Positions below max_slots are always readable.)
  const int listed = a.ufp_cnt[b];
  const bool granted = slot_has_branches(a, b, slot);
  if (slot >= min(listed, a.max_slots) || !granted) return;
  const int u = a.ufp_pos[(int64_t)b * a.chain_len + slot];

  const T* x = reinterpret_cast<const T*>(a.logits) + ((int64_t)b * a.rows + u) * a.ld;
  const int begin = split * kChunk;
  const int n = min(a.vocab, begin + kChunk) - begin;     // entries in this chunk
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;

  // Entry j of the lane's vector w is chunk entry (w * kThreads + tid) * kVec + j.
  float f[kLaneVecs][kVec];
  if (kVecPath) {
    const int nvec = n / kVec;
    const __amdgpu_buffer_rsrc_t rsrc = chunk_rsrc(x + begin, (uint32_t)nvec * kVec * sizeof(T));
#pragma unroll
    for (int w = 0; w < kLaneVecs; ++w)
      load_vec<T>(rsrc, (uint32_t)((w * kThreads + tid) * kVec * sizeof(T)), f[w]);
    // The partial vector at the end of the row (fewer than kVec entries) is
    // read entry by entry by the one lane that owns it.
    const int tail = n - nvec * kVec;
    if (tail > 0 && nvec % kThreads == tid) {
      const int w = nvec / kThreads;
#pragma unroll
      for (int w2 = 0; w2 < kLaneVecs; ++w2)
        if (w2 == w) {
#pragma unroll
          for (int j = 0; j < kVec; ++j)
            f[w2][j] = j < tail ? load1<T>(x + begin + nvec * kVec + j) : 0.f;
        }
    }
  } else {
#pragma unroll
    for (int w = 0; w < kLaneVecs; ++w)
#pragma unroll
      for (int j = 0; j < kVec; ++j) {
        const int e = (w * kThreads + tid) * kVec + j;
        f[w][j] = e < n ? load1<T>(x + begin + e) : 0.f;
      }
  }
  // Entries past the chunk end become -inf; validity is tracked by position.
  float vmax[kLaneVecs];
#pragma unroll
  for (int w = 0; w < kLaneVecs; ++w) {
    const int e0 = (w * kThreads + tid) * kVec;
    float m = -INFINITY;
#pragma unroll
    for (int j = 0; j < kVec; ++j) {
      f[w][j] = e0 + j < n ? f[w][j] : -INFINITY;
      m = fmaxf(m, f[w][j]);
    }
    vmax[w] = m;
  }

  // Lower bound on the chunk's 8th-best value: per wave, the smallest maximum
  // of eight disjoint 8-lane groups (a group without entries gives -inf, no
  // bound); then the largest bound over the waves.
  float g = fmaxf(fmaxf(vmax[0], vmax[1]), fmaxf(vmax[2], vmax[3]));
  g = fmaxf(g, partner<1>(g));
  g = fmaxf(g, partner<2>(g));
  g = fmaxf(g, partner<4>(g));
  g = fminf(g, partner<8>(g));
  g = fminf(g, partner<16>(g));
  g = fminf(g, partner<32>(g));
  if (lane == 0) s_bound[wave] = g;
  __syncthreads();
  const float bound = fmaxf(fmaxf(s_bound[0], s_bound[1]), fmaxf(s_bound[2], s_bound[3]));

  // Candidates: the entries at or above the bound, appended per wave.
  int wcnt = 0;
#pragma unroll
  for (int w = 0; w < kLaneVecs; ++w) {
    const int e0 = (w * kThreads + tid) * kVec;
#pragma unroll
    for (int j = 0; j < kVec; ++j)
      wave_append(s_cand[wave], wcnt, (e0 + j < n) & (f[w][j] >= bound), f[w][j], begin + e0 + j);
  }
  const int64_t out = (((int64_t)b * a.max_slots + slot) * a.splits + split) * kTopK;

  // Each wave's best eight, sorted, into s_top: every candidate finds its rank
  // among the wave's candidates by counting those that outrank it; places
  // beyond the count stay empty. A wave with more candidates than its list
  // holds (long runs of equal values) ranks its registers in eight rounds of
  // a wave-wide best instead.
  if (lane < kTopK) s_top[wave][lane] = Cand{-INFINITY, INT32_MAX};
  __builtin_amdgcn_wave_barrier();
  if (wcnt <= kWaveCap) {
    if (lane < wcnt) {
      const Cand m = s_cand[wave][lane];
      const int rank = rank_among(s_cand[wave], wcnt, m.v, m.i);
      if (rank < kTopK) s_top[wave][rank] = m;
    }
  } else {
    uint32_t taken = 0;
    for (int r = 0; r < kTopK; ++r) {
      float bv = -INFINITY;
      int bi = INT32_MAX;
#pragma unroll
      for (int w = 0; w < kLaneVecs; ++w) {
        const int e0 = (w * kThreads + tid) * kVec;
#pragma unroll
        for (int j = 0; j < kVec; ++j) {
          const bool ok = (e0 + j < n) & !((taken >> (w * kVec + j)) & 1u);
          const bool c = ok & outranks(f[w][j], begin + e0 + j, bv, bi);
          bv = c ? f[w][j] : bv;
          bi = c ? begin + e0 + j : bi;
        }
      }
      wave_best(bv, bi);
      if (lane == 0) s_top[wave][r] = Cand{bv, bi};
      const int rel = bi - begin;                 // chunk entry of the winner
      if (bi != INT32_MAX && (rel / kVec) % kThreads == tid)
        taken |= 1u << ((rel / kVec / kThreads) * kVec + rel % kVec);
    }
  }
  __syncthreads();

  // The four sorted lists, one per 8-lane group of wave 0, merged pairwise.
  if (wave == 0) {
    const Cand m = lane < kWaves * kTopK ? s_top[lane / kTopK][lane % kTopK]
                                         : Cand{-INFINITY, INT32_MAX};
    float v = m.v;
    int i = m.i;
    merge_groups<kMirror16>(v, i);
    merge_groups<kMirror32>(v, i);
    if (lane < kTopK) {
      a.part_val[out + lane] = v;
      a.part_idx[out + lane] = i;
    }
  }
}

// Loads the chunk results of UFP slot s: lane l holds records l + 64 q. The
// loads are unconditional (indices past the end are clamped and their values
// replaced), so no branch forces a wait for them.
CURE_DEV void load_partials(const Args& a, int b, int s, float (&cv)[kMaxSplits * kTopK / kWave],
                            int (&ci)[kMaxSplits * kTopK / kWave]) {
  const int lane = lane_id();
  const int64_t base = (((int64_t)b * a.max_slots + s) * a.splits) * kTopK;
  const int ncand = a.splits * kTopK;
#pragma unroll
  for (int q = 0; q < kMaxSplits * kTopK / kWave; ++q) {
    const int c = lane + q * kWave;
    const int cc = min(c, ncand - 1);
    const float v = a.part_val[base + cc];
    const int i = a.part_idx[base + cc];
    cv[q] = c < ncand ? v : -INFINITY;
    ci[q] = c < ncand ? i : INT32_MAX;
  }
}

// The suffix token of branch node t (t = r * depth + j, j > 0) of the branch
// at block position u, or -1 without suffix tokens.
CURE_DEV int suffix_token(const Args& a, int b, int u, int t) {
  const int r = t / a.depth, j = t - r * a.depth;
  if (!a.suffix || j == 0) return -1;
  return a.suffix[(((int64_t)b * a.chain_len + u) * a.b_max + r) * (a.depth - 1) + (j - 1)];
}

__global__ __launch_bounds__(kThreads) void repair_assemble(Args a) {
  extern __shared__ int s_dyn[];
  int* s_nb = s_dyn;                                // [max_slots] Eq. (3), then granted
  int* s_first = s_nb + a.max_slots;                // [max_slots] first branch number
  int* s_u = s_first + a.max_slots;                 // [max_slots] block position
  int* s_own = s_u + a.max_slots;                   // [max_slots] the draft's token there
  __shared__ int s_slots, s_total;

  const int b = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int K = a.chain_len, d = a.depth;
  int32_t* par = a.parent + (int64_t)b * a.n_max;
  int32_t* tok = a.token + (int64_t)b * a.n_max;
  constexpr int kPer = kMaxSplits * kTopK / kWave;

  // On this GPU one counter tracks loads and stores together, so a wait for a
  // load also waits for every store issued before it: all loads come first,
  // grouped into as few round trips as the dependences allow, and every store
  // is issued after the last wait.
  //
  // First round trip: the UFP count and positions, the draft block, and each
  // wave's first slot's chunk results (read before it is known whether that
  // slot received branches; unused if not). The slots in use are the first
  // min(ufp_cnt, max_slots), cut at the first position outside the block.
  const int listed = a.ufp_cnt[b];
  const int u_first = a.ufp_pos[(int64_t)b * K + min(tid, max(a.max_slots, 1) - 1)];
  const int chain_first = a.chain_tok[(int64_t)b * K + min(tid, K - 1)];
  float cv[kPer];
  int ci[kPer];
  if (a.max_slots > 0) load_partials(a, b, min(wave, a.max_slots - 1), cv, ci);
  if (tid == 0) s_slots = max(0, min(listed, a.max_slots));
  __syncthreads();
  // Second: each slot's margin for Eq. (3) and the draft's token at its position.
  for (int s = tid; s < a.max_slots; s += kThreads) {
    const int u = s == tid ? u_first : a.ufp_pos[(int64_t)b * K + s];
    const bool ok = u >= 0 && u < K;
    if (!ok) atomicMin(&s_slots, s);
    s_u[s] = u;
    s_own[s] = ok ? a.chain_tok[(int64_t)b * K + u] : -1;
    s_nb[s] = ok ? branch_budget(a.margin[(int64_t)b * a.rows + u], a.scale, a.b_min, a.b_max) : 0;
  }
  __syncthreads();
  const int slots = s_slots;

  // The budget walk on wave 0: whole branches of depth nodes, UFP by UFP,
  // while they fit. Lane l holds slot g0 + l; the walk itself runs on scalars.
  if (wave == 0) {
    int remaining = a.budget, granted = 0;
    for (int g0 = 0; g0 < slots; g0 += kWave) {
      const int s = g0 + lane;
      const int want = s < slots ? s_nb[s] : 0;
      int my_nb = 0, my_first = 0;
      const int n = min(slots - g0, kWave);
      for (int i = 0; i < n; ++i) {
        const int nb = min(__builtin_amdgcn_readlane(want, i), remaining / d);
        my_nb = lane == i ? nb : my_nb;
        my_first = lane == i ? granted : my_first;
        granted += nb;
        remaining -= nb * d;
      }
      if (s < slots) {
        s_nb[s] = my_nb;
        s_first[s] = my_first;
      }
    }
    if (lane == 0) s_total = granted;
  }
  __syncthreads();

  // Per slot with branches, one wave: the row's best eight from its chunk
  // results, the branch roots (alternative r, the r-th ranked token other than
  // the draft's own, hangs off chain node u - 1), and the nodes past the roots
  // (suffix tokens, or -1, each hanging off the node before it).
  // The largest 8th entry over the chunk lists bounds the row's 8th best from
  // below, so only the entries at or above it are ranked (by counting, as in
  // the chunk kernel); if ties leave more than a wave's worth of them, eight
  // rounds of a wave-wide best rank all entries instead.
  for (int s = wave; s < slots; s += kWaves) {
    const int nb = s_nb[s];
    if (nb == 0) continue;
    const int u = s_u[s];
    const int first = K + s_first[s] * d;
    const int nodes = nb * d;
    // The first suffix token of this lane (issued now, stored after the merge).
    const int sfx0 = lane < nodes ? suffix_token(a, b, u, lane) : -1;
    if (s != wave) load_partials(a, b, s, cv, ci);
    // Lane l holds entry l % 8 of chunk list l / 8 + 8 q in (cv[q], ci[q]);
    // lists past the chunk count are empty. Fold the register lists
    // pairwise, then the eight lists of the wave across lanes.
    const int nq = (a.splits + kWave / kTopK - 1) / (kWave / kTopK);
#pragma unroll
    for (int step = 1; step < kPer; step *= 2)
#pragma unroll
      for (int q = 0; q + step < kPer; q += 2 * step)
        if (q + step < nq)
          merge8(cv[q], ci[q], __int_as_float(xchg<kMirror8>(__float_as_int(cv[q + step]))),
                 xchg<kMirror8>(ci[q + step]));
    float tv = cv[0];
    int ti = ci[0];
    merge_groups<kMirror16>(tv, ti);
    merge_groups<kMirror32>(tv, ti);
    merge_groups<kMirror64>(tv, ti);
    const int own = s_own[s];
    const bool is_own = lane < kTopK && ti == own;
    const uint64_t own_mask = __ballot(is_own);
    const int own_rank = own_mask ? __builtin_ctzll(own_mask) : kTopK;
    const int alt_rank = lane - (own_rank < lane ? 1 : 0);
    if (lane < kTopK && !is_own && alt_rank < nb) {
      par[first + alt_rank * d] = u - 1;
      tok[first + alt_rank * d] = ti;
    }
    for (int t = lane; t < nodes; t += kWave) {
      if (t % d == 0) continue;
      par[first + t] = first + t - 1;
      tok[first + t] = t == lane ? sfx0 : suffix_token(a, b, u, t);
    }
  }

  // The chain, the per-slot branch counts and the node count.
  for (int i = tid; i < K; i += kThreads) {
    par[i] = i - 1;
    tok[i] = i == tid ? chain_first : a.chain_tok[(int64_t)b * K + i];
    if (a.branch_cnt) a.branch_cnt[(int64_t)b * K + i] = i < slots ? s_nb[i] : 0;
  }
  if (tid == 0) a.n_nodes[b] = K + s_total * d;
}

int max_slots_of(int32_t chain_len, int32_t repair_budget, int32_t depth) {
  return std::min(chain_len, repair_budget / depth);
}

int splits_of(int32_t vocab) { return (vocab + kChunk - 1) / kChunk; }

}  // namespace
}  // namespace cure

using namespace cure;

extern "C" size_t cure_repair_tree_workspace_size(int32_t batch, int32_t chain_len,
                                                  int32_t vocab, int32_t repair_budget,
                                                  int32_t branch_depth) {
  if (batch <= 0 || chain_len <= 0 || vocab <= 0 || repair_budget < 0 || branch_depth < 1)
    return 0;
  const int slots = max_slots_of(chain_len, repair_budget, branch_depth);
  if (slots == 0) return 0;
  const size_t rec = (size_t)batch * slots * splits_of(vocab) * kTopK;
  return align_up(rec * sizeof(float), 256) + align_up(rec * sizeof(int32_t), 256);
}

extern "C" cure_status cure_repair_tree(
    const void* logits, int32_t dtype, int32_t batch, int32_t rows, int32_t vocab, int64_t ld,
    const float* margin, const int32_t* ufp_pos, const int32_t* ufp_cnt,
    const int32_t* chain_tok, int32_t chain_len, int32_t repair_budget, int32_t branch_depth,
    float margin_scale, int32_t b_min, int32_t b_max, const int32_t* suffix, int32_t n_max,
    int32_t* parent, int32_t* token, int32_t* n_nodes, int32_t* branch_cnt, void* workspace,
    size_t workspace_bytes, void* stream) {
  if (dtype != CURE_F32 && dtype != CURE_BF16) return CURE_ERR_INVALID_ARG;
  if (batch < 0) return CURE_ERR_INVALID_ARG;
  if (batch == 0) return CURE_OK;
  if (chain_len < 1 || rows < chain_len || branch_depth < 1 || repair_budget < 0)
    return CURE_ERR_INVALID_ARG;
  if (b_min < 0 || b_max < b_min || b_max < 1 || vocab < b_max + 1 || ld < vocab)
    return CURE_ERR_INVALID_ARG;
  if (!(margin_scale > 0.f) || !std::isfinite(margin_scale)) return CURE_ERR_INVALID_ARG;
  if ((int64_t)n_max < (int64_t)chain_len + repair_budget) return CURE_ERR_INVALID_ARG;
  if (!logits || !margin || !ufp_pos || !ufp_cnt || !chain_tok || !parent || !token || !n_nodes)
    return CURE_ERR_INVALID_ARG;
  if (b_max > kTopK - 1 || chain_len > kMaxChain || splits_of(vocab) > kMaxSplits)
    return CURE_ERR_UNSUPPORTED;

  const int slots = max_slots_of(chain_len, repair_budget, branch_depth);
  const int splits = splits_of(vocab);
  const int64_t grid = (int64_t)batch * slots * splits;
  if (grid > INT32_MAX) return CURE_ERR_UNSUPPORTED;
  const size_t need = cure_repair_tree_workspace_size(batch, chain_len, vocab, repair_budget,
                                                      branch_depth);
  if (need > 0 && (!workspace || workspace_bytes < need)) return CURE_ERR_WORKSPACE;

  const size_t rec = (size_t)batch * slots * splits * kTopK;
  Args a;
  a.logits = logits;
  a.ld = ld;
  a.batch = batch;
  a.rows = rows;
  a.vocab = vocab;
  a.splits = splits;
  a.max_slots = slots;
  a.chain_len = chain_len;
  a.margin = margin;
  a.ufp_pos = ufp_pos;
  a.ufp_cnt = ufp_cnt;
  a.chain_tok = chain_tok;
  a.suffix = branch_depth > 1 ? suffix : nullptr;
  a.depth = branch_depth;
  a.budget = repair_budget;
  a.b_min = b_min;
  a.b_max = b_max;
  a.scale = margin_scale;
  a.n_max = n_max;
  a.parent = parent;
  a.token = token;
  a.n_nodes = n_nodes;
  a.branch_cnt = branch_cnt;
  a.part_val = reinterpret_cast<float*>(workspace);
  a.part_idx = reinterpret_cast<int32_t*>(reinterpret_cast<char*>(workspace) +
                                          align_up(rec * sizeof(float), 256));

  hipStream_t s = as_stream(stream);
  if (grid > 0) {
    const size_t esize = dtype == CURE_F32 ? 4 : 2;
    const bool vec_ok = (reinterpret_cast<uintptr_t>(logits) % 16 == 0) &&
                        ((size_t)ld * esize) % 16 == 0;
    const dim3 g((unsigned)grid), blk(kThreads);
    if (dtype == CURE_BF16) {
      if (vec_ok) hipLaunchKernelGGL((topk_chunk<uint16_t, true>), g, blk, 0, s, a);
      else hipLaunchKernelGGL((topk_chunk<uint16_t, false>), g, blk, 0, s, a);
    } else {
      if (vec_ok) hipLaunchKernelGGL((topk_chunk<float, true>), g, blk, 0, s, a);
      else hipLaunchKernelGGL((topk_chunk<float, false>), g, blk, 0, s, a);
    }
    if (hipGetLastError() != hipSuccess) return CURE_ERR_HIP;
  }
  const size_t lds = (size_t)std::max(slots, 1) * 4 * sizeof(int);
  hipLaunchKernelGGL(repair_assemble, dim3(batch), dim3(kThreads), lds, s, a);
  return launch_status();
}
