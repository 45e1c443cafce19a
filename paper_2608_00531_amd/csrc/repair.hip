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
//   over its waves, appends the few entries at or above it to LDS, and one
//   wave ranks them exactly. Only when more than kCandCap entries pass (large
//   runs of equal values) does the workgroup fall back to eight rounds of
//   workgroup-wide selection over the registers. Output: the chunk's best
//   eight (value descending, index ascending) in the workspace.
//
// repair_assemble -- one workgroup per sequence. Each wave merges the chunk
//   results of a UFP row into the row's best eight, drops the draft's own
//   token to get the ranked alternatives, and evaluates Eq. (3) on the row's
//   margin. One lane then walks the UFPs in order and hands out whole branches
//   while they fit the budget; finally all lanes write the parent/token arrays.
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
constexpr int kCandCap = 256;            // LDS candidates per chunk
constexpr int kMaxChain = 1024;

struct Args {
  const void* logits;
  int64_t ld;
  int32_t rows, vocab, splits, max_slots, chain_len;
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

// Exact best eight over the wave's candidates: lane l holds kPer of them
// (empty = (-inf, INT32_MAX), which every real entry beats; real indices are
// distinct). Eight rounds of a wave-wide best, each removing its winner.
// Lane r < 8 returns the r-th best; every lane must take part.
template <int kPer>
CURE_DEV void wave_top8(float (&v)[kPer], int (&ix)[kPer], float& ov, int& oi) {
  const int lane = lane_id();
  ov = -INFINITY;
  oi = INT32_MAX;
#pragma unroll
  for (int r = 0; r < kTopK; ++r) {
    float bv = v[0];
    int bi = ix[0];
#pragma unroll
    for (int k = 1; k < kPer; ++k) {
      const bool c = beats(v[k], ix[k], bv, bi);
      bv = c ? v[k] : bv;
      bi = c ? ix[k] : bi;
    }
    wave_best(bv, bi);
    ov = lane == r ? bv : ov;
    oi = lane == r ? bi : oi;
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      const bool hit = ix[k] == bi;
      v[k] = hit ? -INFINITY : v[k];
      ix[k] = hit ? INT32_MAX : ix[k];
    }
  }
}

template <typename T, bool kVecPath>
__global__ __launch_bounds__(kThreads) void topk_chunk(Args a) {
  __shared__ float s_cv[kCandCap];
  __shared__ int s_ci[kCandCap];
  __shared__ float s_bound[kWaves];
  __shared__ float s_rv[kWaves];
  __shared__ int s_ri[kWaves];
  __shared__ int s_cnt;

  const int split = blockIdx.x % a.splits;
  const int slot = (blockIdx.x / a.splits) % a.max_slots;
  const int b = blockIdx.x / (a.splits * a.max_slots);
  if (slot >= min(a.ufp_cnt[b], a.max_slots)) return;
  const int u = a.ufp_pos[(int64_t)b * a.chain_len + slot];
  if (u < 0 || u >= a.chain_len) return;

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
  if (tid == 0) s_cnt = 0;
  __syncthreads();
  const float bound = fmaxf(fmaxf(s_bound[0], s_bound[1]), fmaxf(s_bound[2], s_bound[3]));

  // Candidates: the entries at or above the bound.
#pragma unroll
  for (int w = 0; w < kLaneVecs; ++w) {
    if (vmax[w] >= bound) {
      const int e0 = (w * kThreads + tid) * kVec;
#pragma unroll
      for (int j = 0; j < kVec; ++j) {
        if (e0 + j < n && f[w][j] >= bound) {
          const int p = atomicAdd(&s_cnt, 1);
          if (p < kCandCap) {
            s_cv[p] = f[w][j];
            s_ci[p] = begin + e0 + j;
          }
        }
      }
    }
  }
  __syncthreads();
  const int cnt = s_cnt;
  const int64_t out = (((int64_t)b * a.max_slots + slot) * a.splits + split) * kTopK;

  if (cnt <= kCandCap) {
    if (wave == 0) {
      float cv[kCandCap / kWave];
      int ci[kCandCap / kWave];
#pragma unroll
      for (int q = 0; q < kCandCap / kWave; ++q) {
        const int c = lane + q * kWave;
        cv[q] = c < cnt ? s_cv[c] : -INFINITY;
        ci[q] = c < cnt ? s_ci[c] : INT32_MAX;
      }
      float ov;
      int oi;
      wave_top8(cv, ci, ov, oi);
      if (lane < kTopK) {
        a.part_val[out + lane] = ov;
        a.part_idx[out + lane] = oi;
      }
    }
    return;
  }

  // Too many ties at the bound: eight rounds of a workgroup-wide best over the
  // registers, each round removing its winner (taken bits are per entry).
  uint32_t taken = 0;
  float rv = -INFINITY;
  int ri = INT32_MAX;
  for (int r = 0; r < kTopK; ++r) {
    float bv = -INFINITY;
    int bi = INT32_MAX;
#pragma unroll
    for (int w = 0; w < kLaneVecs; ++w) {
      const int e0 = (w * kThreads + tid) * kVec;
#pragma unroll
      for (int j = 0; j < kVec; ++j) {
        const bool ok = e0 + j < n && !((taken >> (w * kVec + j)) & 1u);
        const bool c = ok && beats(f[w][j], begin + e0 + j, bv, bi);
        bv = c ? f[w][j] : bv;
        bi = c ? begin + e0 + j : bi;
      }
    }
    wave_best(bv, bi);
    if (lane == 0) { s_rv[wave] = bv; s_ri[wave] = bi; }
    __syncthreads();
    float gv = s_rv[0];
    int gi = s_ri[0];
#pragma unroll
    for (int k = 1; k < kWaves; ++k) {
      const bool c = beats(s_rv[k], s_ri[k], gv, gi);
      gv = c ? s_rv[k] : gv;
      gi = c ? s_ri[k] : gi;
    }
    __syncthreads();
    const int rel = gi - begin;                 // chunk entry of the winner
    const int owner_w = rel / kVec / kThreads, owner_t = rel / kVec % kThreads;
    if (gi != INT32_MAX && owner_t == tid) taken |= 1u << (owner_w * kVec + rel % kVec);
    rv = tid == r ? gv : rv;
    ri = tid == r ? gi : ri;
  }
  if (tid < kTopK) {
    a.part_val[out + tid] = rv;
    a.part_idx[out + tid] = ri;
  }
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

__global__ __launch_bounds__(kThreads) void repair_assemble(Args a) {
  extern __shared__ int s_dyn[];
  int* s_alt = s_dyn;                               // [max_slots][kTopK]
  int* s_nb = s_alt + a.max_slots * kTopK;          // [max_slots] Eq. (3), then granted
  int* s_first = s_nb + a.max_slots;                // [max_slots] first branch number
  __shared__ int s_slots, s_total;

  const int b = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int K = a.chain_len;
  const int32_t* pos = a.ufp_pos + (int64_t)b * K;

  // UFP slots in use: the first min(ufp_cnt, max_slots), cut at the first
  // position outside the block.
  if (tid == 0) s_slots = max(0, min(a.ufp_cnt[b], a.max_slots));
  __syncthreads();
  const int listed = s_slots;
  __syncthreads();
  for (int s = tid; s < listed; s += kThreads) {
    const int u = pos[s];
    if (u < 0 || u >= K) atomicMin(&s_slots, s);
  }
  __syncthreads();
  const int slots = s_slots;

  // Per slot: the row's best eight from its chunk results, the ranked
  // alternatives (the draft's own token removed) and Eq. (3).
  constexpr int kPer = kMaxSplits * kTopK / kWave;
  for (int s = wave; s < slots; s += kWaves) {
    const int u = pos[s];
    const int64_t base = (((int64_t)b * a.max_slots + s) * a.splits) * kTopK;
    const int ncand = a.splits * kTopK;
    float cv[kPer];
    int ci[kPer];
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
      const int c = lane + q * kWave;
      cv[q] = c < ncand ? a.part_val[base + c] : -INFINITY;
      ci[q] = c < ncand ? a.part_idx[base + c] : INT32_MAX;
    }
    float tv;
    int ti;
    wave_top8(cv, ci, tv, ti);
    const int own = a.chain_tok[(int64_t)b * K + u];
    const bool is_own = lane < kTopK && ti == own;
    const uint64_t own_mask = __ballot(is_own);
    const int own_rank = own_mask ? __builtin_ctzll(own_mask) : kTopK;
    const int alt_rank = lane - (own_rank < lane ? 1 : 0);
    if (lane < kTopK && !is_own && alt_rank < a.b_max) s_alt[s * kTopK + alt_rank] = ti;
    if (lane == 0)
      s_nb[s] = branch_budget(a.margin[(int64_t)b * a.rows + u], a.scale, a.b_min, a.b_max);
  }
  __syncthreads();

  // Whole branches of depth nodes, UFP by UFP, while they fit the budget.
  if (tid == 0) {
    int remaining = a.budget, granted = 0;
    for (int s = 0; s < slots; ++s) {
      const int nb = min(s_nb[s], remaining / a.depth);
      s_nb[s] = nb;
      s_first[s] = granted;
      granted += nb;
      remaining -= nb * a.depth;
    }
    s_total = granted;
  }
  __syncthreads();

  int32_t* par = a.parent + (int64_t)b * a.n_max;
  int32_t* tok = a.token + (int64_t)b * a.n_max;
  for (int i = tid; i < K; i += kThreads) {
    par[i] = i - 1;
    tok[i] = a.chain_tok[(int64_t)b * K + i];
    if (a.branch_cnt) a.branch_cnt[(int64_t)b * K + i] = i < slots ? s_nb[i] : 0;
  }
  const int d = a.depth;
  for (int s = 0; s < slots; ++s) {
    const int u = pos[s];
    const int first = K + s_first[s] * d;
    for (int t = tid; t < s_nb[s] * d; t += kThreads) {
      const int r = t / d, j = t - r * d;
      const int node = first + t;
      par[node] = j == 0 ? u - 1 : node - 1;
      int tk;
      if (j == 0) tk = s_alt[s * kTopK + r];
      else if (a.suffix) tk = a.suffix[(((int64_t)b * K + u) * a.b_max + r) * (d - 1) + (j - 1)];
      else tk = -1;
      tok[node] = tk;
    }
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
  const size_t lds = (size_t)std::max(slots, 1) * (kTopK + 2) * sizeof(int);
  hipLaunchKernelGGL(repair_assemble, dim3(batch), dim3(kThreads), lds, s, a);
  return launch_status();
}
