// cure_tree_attn: tree-masked verification attention (Sec. 3.2 phase 3,
// Sec. 3.4, Sec. 3.5) as a split-KV ("flash-decoding") pass plus a
// log-sum-exp merge of the split partials.
//
// Every node of a sequence's candidate tree attends to the whole cached
// context and to the nodes on its own root path. The context is shared by all
// nodes, so the work is organised around the key/value stream: one workgroup
// owns (sequence, kv-head, row block, context split) and reads each K/V tile
// from HBM exactly once for all query rows of that kv-head -- the G query heads
// of every tree node, packed node-major. Only tiles that reach the tree rows
// at the tail of the sequence apply the ancestor bitmask.
//
// Three kernels compute a split:
//  * tree_attn_m16: bf16, scale > 0, head dim 128 (any row count, in
//    balanced row blocks of up to 256 rows) or 64 (up to 128 rows). Scores
//    are formed transposed, S^T = K Q^T, and the output as O^T = V^T P^T with
//    16x16x32 bf16 MFMAs, 16 query rows per wave. K/V tiles arrive in LDS by
//    DMA; V is read back transposed by the LDS transpose-read instruction in
//    exactly the token order the score MFMA leaves P in registers.
//  * tree_attn_mfma: the same scheme with 32x32x16 MFMAs and 32 rows per
//    wave, for head dim 64 beyond 128 rows.
//  * tree_attn_valu: fp32 or bf16, any supported shape and scale; plain vector
//    ALU code.
// A split writes normalised partial O and its log-sum-exp; attn_merge combines
// the splits of each row (skipped when a sequence has a single split, in which
// case the split kernel writes the final output itself).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <type_traits>
#include <vector>

#include "common.hpp"
#include "host_util.hpp"

namespace cure {
namespace {

constexpr int kTile = 64;            // tokens per K/V tile
constexpr int kStages = 2;           // K/V tile buffers in the MFMA kernel's LDS ring
constexpr int kMaxGridY = 65535;     // largest grid y (the split index)
constexpr int kMinTps = 256;         // tokens per split, at least
constexpr int kAncWords = CURE_MAX_TREE_NODES / 64;

struct Args {
  const void* q;
  const void* k;
  const void* v;
  void* o;
  float* lse;
  int32_t out_bf16;
  int32_t hq, hkv, group, n_max;
  float scale_log2;                  // scale * log2(e): scores live in the log2 domain
  const int64_t* kv_off;
  const int32_t* ctx_len;
  const int32_t* n_nodes;
  const int32_t* parent;
  int32_t tps, max_splits, rows_per_wg;
  int32_t* tree_status;
  float* part_o;                     // [batch][hq][n_max][max_splits][d]
  float* part_lse;                   // [batch][hq][n_max][max_splits]
};

// Number of context splits of a sequence with T = ctx + nodes rows. The last
// split runs to T, so a clamp never drops rows.
CURE_DEV int split_count(int T, int N, int tps, int max_splits) {
  if (N <= 0 || T <= 0) return 0;
  return min((T + tps - 1) / tps, max_splits);
}

CURE_DEV int64_t part_index(const Args& a, int b, int head, int n, int s) {
  return (((int64_t)b * a.hq + head) * a.n_max + n) * a.max_splits + s;
}

// Loads sequence b's parent array, validates it and builds every node's
// ancestor bitmask (its root path, itself included). Returns true if valid.
CURE_DEV bool build_tree(const Args& a, int b, int N, int* s_parent,
                         unsigned long long (*s_anc)[kAncWords], int* s_bad) {
  if (threadIdx.x == 0) *s_bad = 0;
  __syncthreads();
  for (int n = threadIdx.x; n < N; n += blockDim.x) {
    const int p = a.parent[(int64_t)b * a.n_max + n];
    s_parent[n] = p;
    if (p < -1 || p >= n) *s_bad = 1;
  }
  __syncthreads();
  if (*s_bad) return false;
  for (int n = threadIdx.x; n < N; n += blockDim.x) {
    unsigned long long w[kAncWords] = {};
    for (int j = n; j >= 0; j = s_parent[j]) w[j >> 6] |= 1ull << (j & 63);
#pragma unroll
    for (int i = 0; i < kAncWords; ++i) s_anc[n][i] = w[i];
  }
  __syncthreads();
  return true;
}

// As build_tree, for a workgroup of at least N threads where thread n has
// already loaded parent[n] (the load is issued early, off the critical path).
CURE_DEV bool build_tree_loaded(int N, int my_parent, int* s_parent,
                                unsigned long long (*s_anc)[kAncWords], int* s_bad) {
  const int n = threadIdx.x;
  if (n == 0) *s_bad = 0;
  __syncthreads();
  if (n < N) {
    s_parent[n] = my_parent;
    if (my_parent < -1 || my_parent >= n) *s_bad = 1;
  }
  __syncthreads();
  if (*s_bad) return false;
  if (n < N) {
    unsigned long long w[kAncWords] = {};
    for (int j = n; j >= 0; j = s_parent[j]) w[j >> 6] |= 1ull << (j & 63);
#pragma unroll
    for (int i = 0; i < kAncWords; ++i) s_anc[n][i] = w[i];
  }
  __syncthreads();
  return true;
}

CURE_DEV void report_tree(const Args& a, int b, bool ok, bool reporter) {
  if (reporter && threadIdx.x == 0 && a.tree_status) a.tree_status[b] = ok ? CURE_OK : CURE_ERR_BAD_TREE;
}

// Visibility of cache row tok (relative to the sequence) for node n.
CURE_DEV bool visible(int tok, int L, int N, int n, const unsigned long long (*s_anc)[kAncWords]) {
  if (tok < L) return true;
  const int j = tok - L;
  if (j >= N) return false;
  return (s_anc[n][j >> 6] >> (j & 63)) & 1ull;
}

// Additive mask of token tok for node n inside a split that ends at `end`:
// +0 when visible() holds, -inf otherwise. Computed without branches (the
// ancestor word is read for a clamped row index and context rows ignore it;
// tok < end implies tok < ctx + nodes, so a row past the context is a tree
// row), so that adding it to a score leaves no divergent write to a register
// of an MFMA result vector.
CURE_DEV float mask_bias(int tok, int L, int end, int n,
                         const unsigned long long (*s_anc)[kAncWords]) {
  const int j = min(max(tok - L, 0), CURE_MAX_TREE_NODES - 1);
  const uint32_t bit = (uint32_t)(s_anc[n][j >> 6] >> (j & 63)) & 1u;
  const uint32_t vis = (uint32_t)(tok < L) | ((uint32_t)(tok < end) & bit);
  return __uint_as_float((vis ^ 1u) * 0xff800000u);
}

template <typename T>
CURE_DEV float ld_elem(const T* p);
template <>
CURE_DEV float ld_elem<float>(const float* p) { return *p; }
template <>
CURE_DEV float ld_elem<uint16_t>(const uint16_t* p) { return bf16_to_f32(*p); }

CURE_DEV void store_out(const Args& a, int64_t idx, float val) {
  if (a.out_bf16) reinterpret_cast<uint16_t*>(a.o)[idx] = f32_to_bf16(val);
  else reinterpret_cast<float*>(a.o)[idx] = val;
}

// ---------------------------------------------------------------------------
// Vector-ALU split kernel: 4 waves, 8 query rows per wave, one token per lane
// for the scores and D/64 output columns per lane for P V.
constexpr int kValuRowsPerWave = 8;
constexpr int kValuWaves = 4;
constexpr int kValuRows = kValuRowsPerWave * kValuWaves;

template <typename E, int D>
__global__ __launch_bounds__(256) void tree_attn_valu(Args a) {
  __shared__ int s_parent[CURE_MAX_TREE_NODES];
  __shared__ unsigned long long s_anc[CURE_MAX_TREE_NODES][kAncWords];
  __shared__ int s_bad;
  __shared__ float s_q[kValuRows][D];
  __shared__ float s_k[kTile][D + 1];
  __shared__ float s_v[kTile][D];
  __shared__ float s_p[kValuWaves][kValuRowsPerWave][kTile];

  const int b = blockIdx.z;
  const int hk = blockIdx.x % a.hkv;
  const int rb = blockIdx.x / a.hkv;
  const int s = blockIdx.y;
  const int N = min(a.n_nodes[b], a.n_max);
  const int L = a.ctx_len[b];
  const int T = L + N;
  const int S = split_count(T, N, a.tps, a.max_splits);
  const int rows = N * a.group;
  if (S == 0) {                         // no nodes: nothing to compute; the empty tree is valid
    report_tree(a, b, true, s == 0 && hk == 0 && rb == 0);
    return;
  }
  if (s >= S || rb * kValuRows >= rows) return;
  const bool reporter = s == 0 && hk == 0 && rb == 0;
  const bool ok = build_tree(a, b, N, s_parent, s_anc, &s_bad);
  report_tree(a, b, ok, reporter);
  if (!ok) return;

  const int begin = s * a.tps;
  const int end = (s == S - 1) ? T : begin + a.tps;
  const int64_t off = a.kv_off[b];
  const E* qp = reinterpret_cast<const E*>(a.q);
  const E* kp = reinterpret_cast<const E*>(a.k);
  const E* vp = reinterpret_cast<const E*>(a.v);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  for (int i = tid; i < kValuRows * D; i += 256) {
    const int r = i / D, d = i - r * D;
    const int R = rb * kValuRows + r;
    float val = 0.f;
    if (R < rows) {
      const int n = R / a.group, head = hk * a.group + R % a.group;
      val = ld_elem<E>(qp + (((int64_t)b * a.n_max + n) * a.hq + head) * D + d);
    }
    s_q[r][d] = val;
  }

  float m_run[kValuRowsPerWave], l_run[kValuRowsPerWave], acc[kValuRowsPerWave][D / 64];
#pragma unroll
  for (int i = 0; i < kValuRowsPerWave; ++i) {
    m_run[i] = -INFINITY;
    l_run[i] = 0.f;
#pragma unroll
    for (int c = 0; c < D / 64; ++c) acc[i][c] = 0.f;
  }

  for (int t0 = begin; t0 < end; t0 += kTile) {
    __syncthreads();
    for (int i = tid; i < kTile * D; i += 256) {
      const int t = i / D, d = i - t * D;
      const int tok = t0 + t;
      float kv = 0.f, vv = 0.f;
      if (tok < end) {
        const int64_t e = ((off + tok) * a.hkv + hk) * D + d;
        kv = ld_elem<E>(kp + e);
        vv = ld_elem<E>(vp + e);
      }
      s_k[t][d] = kv;
      s_v[t][d] = vv;
    }
    __syncthreads();

    // Scores for this wave's rows: lane = token.
    float sc[kValuRowsPerWave];
#pragma unroll
    for (int i = 0; i < kValuRowsPerWave; ++i) sc[i] = 0.f;
    for (int d = 0; d < D; ++d) {
      const float kd = s_k[lane][d];
#pragma unroll
      for (int i = 0; i < kValuRowsPerWave; ++i)
        sc[i] = fmaf(s_q[wave * kValuRowsPerWave + i][d], kd, sc[i]);
    }
    const int tok = t0 + lane;
#pragma unroll
    for (int i = 0; i < kValuRowsPerWave; ++i) {
      const int R = rb * kValuRows + wave * kValuRowsPerWave + i;
      const int n = min(R / a.group, N - 1);
      const bool vis = tok < end && visible(tok, L, N, n, s_anc);
      const float x = vis ? sc[i] * a.scale_log2 : -INFINITY;
      float mt = x;
      mt = wave_max(mt);
      const float m_new = fmaxf(m_run[i], mt);
      const float m_use = m_new == -INFINITY ? 0.f : m_new;
      const float p = exp2f(x - m_use);
      float ps = p;
      ps = wave_sum(ps);
      const float alpha = exp2f(m_run[i] - m_use);
      l_run[i] = l_run[i] * alpha + ps;
      m_run[i] = m_new;
#pragma unroll
      for (int c = 0; c < D / 64; ++c) acc[i][c] *= alpha;
      s_p[wave][i][lane] = p;
    }
    // P V: lane = output column(s).
    for (int t = 0; t < kTile; ++t) {
      float vv[D / 64];
#pragma unroll
      for (int c = 0; c < D / 64; ++c) vv[c] = s_v[t][lane + 64 * c];
#pragma unroll
      for (int i = 0; i < kValuRowsPerWave; ++i) {
        const float p = s_p[wave][i][t];
#pragma unroll
        for (int c = 0; c < D / 64; ++c) acc[i][c] = fmaf(p, vv[c], acc[i][c]);
      }
    }
  }

#pragma unroll
  for (int i = 0; i < kValuRowsPerWave; ++i) {
    const int R = rb * kValuRows + wave * kValuRowsPerWave + i;
    if (R >= rows) continue;
    const int n = R / a.group, head = hk * a.group + R % a.group;
    const float inv = l_run[i] > 0.f ? 1.f / l_run[i] : 0.f;
    const float lse2 = l_run[i] > 0.f ? m_run[i] + log2f(l_run[i]) : -INFINITY;
    if (S == 1) {
      const int64_t base = (((int64_t)b * a.n_max + n) * a.hq + head) * D;
#pragma unroll
      for (int c = 0; c < D / 64; ++c) store_out(a, base + lane + 64 * c, acc[i][c] * inv);
      if (lane == 0 && a.lse) a.lse[((int64_t)b * a.n_max + n) * a.hq + head] = lse2 * kLn2;
    } else {
      const int64_t pi = part_index(a, b, head, n, s);
#pragma unroll
      for (int c = 0; c < D / 64; ++c) a.part_o[pi * D + lane + 64 * c] = acc[i][c] * inv;
      if (lane == 0) a.part_lse[pi] = lse2 * kLn2;
    }
  }
}

// ---------------------------------------------------------------------------
// MFMA split kernel (bf16 in, fp32 accumulate).
//
// Each of the NW waves owns 32 query rows. Per 64-token tile:
//   S^T = K Q^T  (2 token blocks x D/16 k-steps of 32x32x16 MFMA; lane = query row)
//   online softmax in the log2 domain, rescaling O only when a row's maximum
//   rises by more than 2^8 (values then stay below 2^8, safe in bf16 and fp32)
//   O^T += V^T P^T (D/32 column blocks x 4 k-steps)
// K and V tiles move HBM -> LDS by DMA (buffer loads that write LDS directly)
// through a ring of NBUF tile buffers: while one tile is computed, the next
// NBUF - 1 stream in. Two buffers at head dim 128 leave room for two
// workgroups (eight waves) per CU; a deeper ring trades those waves for more
// bytes in flight, and measured slower. The per-sequence buffer resource
// bounds every read: rows past the sequence end read as zeros, and ring
// slots past the split's end are filled by reads at an offset past the
// resource, which touch no memory. LDS rows are 16-byte-chunk XOR-swizzled so
// that both the K reads (one row per lane) and the transposed V reads (4 rows
// x 16 columns per 16 lanes, ds_read_b64_tr_b16) spread over the banks.
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

typedef int i32x4 __attribute__((ext_vector_type(4)));
constexpr int kRsrcWord3 = 0x00020000;     // raw (untyped) 32-bit access, gfx9 family

// A raw buffer resource over `bytes` bytes at `base`, as four wave-uniform
// dwords (SGPRs): base address (48 bits, stride 0), record count in bytes,
// and the gfx9-family word for untyped 32-bit access. Built from integer
// words rather than converted from the opaque resource type, which the
// compiler would spill through a per-thread memory copy.
CURE_DEV i32x4 raw_rsrc(const void* base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  return i32x4{__builtin_amdgcn_readfirstlane((int)(uint32_t)a),
               __builtin_amdgcn_readfirstlane((int)((uint32_t)(a >> 32) & 0xffffu)),
               __builtin_amdgcn_readfirstlane((int)bytes),
               __builtin_amdgcn_readfirstlane(kRsrcWord3)};
}

CURE_DEV uint32_t lds_addr(const void* p) {
  return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(const lds_void*)p);
}

// 64 lanes x 16 bytes from a buffer resource straight into LDS: lane i's bytes
// land at lds_base + 16 * i (lds_base travels in M0). Out-of-range offsets
// read as zero.
CURE_DEV void dma16(uint32_t lds_base, uint32_t voff, i32x4 rsrc) {
  asm volatile("buffer_load_dwordx4 %0, %1, 0 offen nt lds"
               :
               : "v"(voff), "s"(rsrc), "{m0}"(lds_base)
               : "memory");
}

union Pack8 {
  uint4 u;
  bf16x8 v;
  i16x4 h[2];
};


// Three-input maximum as one v_max3_f32. Written as assembly because fmaxf
// first canonicalises every operand that may be a signalling NaN (an extra
// instruction per score); scores here are finite dot products or -inf.
CURE_DEV float max3_raw(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}
constexpr float kRescaleLog2 = 8.f;       // lazy rescale threshold (log2 units)

template <int D>
struct TileGeo {
  static constexpr int kChunks = D / 8;             // 16-byte chunks per row
  static constexpr int kRowBytes = D * 2;
  static constexpr int kTileBytes = kTile * kRowBytes;
  static constexpr int kBlocks = kTileBytes / 1024;  // 1 KB DMA blocks per tile
  // Swizzle: the chunk index is XORed with a row-dependent value. Any value
  // keeps the layout correct (the DMA and every reader apply the same XOR); it
  // only decides which LDS banks one instruction touches. At head dim 128 the
  // chunk bits are (r1^r2, r1, r2, r0) of the row bits r0..r2: with it neither
  // the K operand reads (16 bytes per lane, 16 rows) nor the transposed V reads
  // (8 bytes per lane, 4 rows per 16 lanes) have bank conflicts, as measured
  // with SQ_LDS_BANK_CONFLICT on gfx950 (the earlier permutation of the row
  // bits cost 4 stall cycles per K read and 2 per V read).
  static CURE_DEV int swz(int row) {
    if (kChunks == 16) {
      const int r0 = row & 1, r1 = (row >> 1) & 1, r2 = (row >> 2) & 1;
      return (r1 ^ r2) | (r1 << 1) | (r2 << 2) | (r0 << 3);
    }
    return ((row & 3) << 1) | ((row >> 2) & 1);
  }
  static CURE_DEV int offset(int row, int chunk) {   // byte offset inside a tile
    return row * kRowBytes + ((chunk ^ swz(row)) << 4);
  }
};

// s_waitcnt immediate: at most `vm` vector-memory operations outstanding, no
// wait on export, all LDS/scalar-memory operations complete (gfx9 encoding:
// vmcnt[3:0] in bits 3:0, vmcnt[5:4] in bits 15:14, expcnt in 6:4).
constexpr int waitcnt_vm(int vm) { return (vm & 15) | ((vm >> 4) << 14) | (7 << 4); }
constexpr uint32_t kOobOffset = 0x80000000u;   // past any sequence's buffer resource

template <int D, int NW, int NBUF>
__global__ __launch_bounds__(64 * NW, NBUF > 2 ? 1 : 2) void tree_attn_mfma(Args a) {
  using G = TileGeo<D>;
  constexpr int kKSteps = D / 16;                  // MFMA k-steps for Q K^T
  constexpr int kDBlk = D / 32;                    // 32-column blocks of O^T
  constexpr int kDmaPerWave = G::kBlocks / NW;     // DMA blocks per wave per tensor
  // Each loop iteration waits until its tile has landed while the NBUF - 2
  // tiles issued after it may still be in flight (2 instructions per block).
  constexpr int kVmWait = waitcnt_vm((NBUF - 2) * 2 * kDmaPerWave);
  static_assert((NBUF - 2) * 2 * kDmaPerWave < 64, "vmcnt holds 6 bits");
  static_assert(G::kBlocks % NW == 0, "tile must split evenly across waves");

  __shared__ int s_parent[CURE_MAX_TREE_NODES];
  __shared__ unsigned long long s_anc[CURE_MAX_TREE_NODES][kAncWords];
  __shared__ int s_bad;
  __shared__ __attribute__((aligned(1024))) unsigned char s_k[NBUF][G::kTileBytes];
  __shared__ __attribute__((aligned(1024))) unsigned char s_v[NBUF][G::kTileBytes];

  const int b = blockIdx.z;
  const int hk = blockIdx.x % a.hkv;
  const int rb = blockIdx.x / a.hkv;
  const int s = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, col = lane & 31;

  // This lane's query row, and its query loads: they need only the launch
  // shape (rows past the sequence's nodes still lie inside q and are zeroed
  // below), so they go out together with the loads of the sequence's sizes,
  // as does each thread's parent entry for the tree.
  const int R = rb * a.rows_per_wg + wave * 32 + col;
  const bool r_in = R < a.n_max * a.group;
  bf16x8 qreg[kKSteps];
  {
    const int qn = r_in ? R / a.group : 0;
    const int qh = hk * a.group + (r_in ? R % a.group : 0);
    const uint16_t* qrow = reinterpret_cast<const uint16_t*>(a.q) +
                           (((int64_t)b * a.n_max + qn) * a.hq + qh) * D;
#pragma unroll
    for (int kk = 0; kk < kKSteps; ++kk) {
      Pack8 p;
      p.u = r_in ? *reinterpret_cast<const uint4*>(qrow + kk * 16 + half * 8)
                 : make_uint4(0, 0, 0, 0);
      qreg[kk] = p.v;
    }
  }
  const int my_parent = tid < a.n_max ? a.parent[(int64_t)b * a.n_max + tid] : -1;

  // The sequence's sizes and cache offset are independent loads: one round
  // trip. The empty asm keeps the compiler from sinking the offset's load
  // below the early exits (a second round trip).
  const int n_raw = a.n_nodes[b];
  const int L = a.ctx_len[b];
  const int64_t off = a.kv_off[b];
  asm volatile("" : : "s"(n_raw), "s"(L), "s"(off));
  const int N = min(n_raw, a.n_max);
  const int T = L + N;
  const int S = split_count(T, N, a.tps, a.max_splits);
  const int rows = N * a.group;
  if (S == 0) {                         // no nodes: nothing to compute; the empty tree is valid
    report_tree(a, b, true, s == 0 && hk == 0 && rb == 0);
    return;
  }
  if (s >= S || rb * a.rows_per_wg >= rows) return;

  const int begin = s * a.tps;
  const int end = (s == S - 1) ? T : begin + a.tps;

  // Buffer resources over this sequence's K and V rows (all kv-heads).
  const uint32_t seq_bytes = (uint32_t)T * (uint32_t)(a.hkv * G::kRowBytes);
  // Per lane and DMA block: byte offset of the source chunk for tile start 0.
  uint32_t src_off[kDmaPerWave];
#pragma unroll
  for (int j = 0; j < kDmaPerWave; ++j) {
    const int byte = (wave * kDmaPerWave + j) * 1024 + lane * 16;   // destination in tile
    const int row = byte / G::kRowBytes;
    const int pchunk = (byte % G::kRowBytes) >> 4;
    const int lchunk = pchunk ^ G::swz(row);
    src_off[j] = (uint32_t)((row * a.hkv + hk) * G::kRowBytes + (lchunk << 4));
  }
  const uint32_t tok_bytes = (uint32_t)(a.hkv * G::kRowBytes);
  // The DMA is issued from inline assembly on purpose: written through the
  // compiler builtin, every later LDS read of the *current* tile gets a wait on
  // the *next* tile's DMA (the compiler cannot tell the buffers apart), which
  // serialises the pipeline. Ordering is explicit instead: each loop iteration
  // starts with s_waitcnt + barrier before any LDS read of the tile it uses.
  // A tile at or past the split's end is still issued (at an out-of-range
  // offset) so that every iteration has the same number of DMAs in flight.
  const i32x4 rk4 = raw_rsrc(reinterpret_cast<const uint16_t*>(a.k) + off * a.hkv * D, seq_bytes);
  const i32x4 rv4 = raw_rsrc(reinterpret_cast<const uint16_t*>(a.v) + off * a.hkv * D, seq_bytes);
  auto dma_tile = [&](int buf, int t0) {
    const bool live = t0 < end;
#pragma unroll
    for (int j = 0; j < kDmaPerWave; ++j) {
      const uint32_t voff = live ? src_off[j] + (uint32_t)t0 * tok_bytes : kOobOffset;
      const int blk = (wave * kDmaPerWave + j) * 1024;
      dma16(lds_addr(&s_k[buf][blk]), voff, rk4);
      dma16(lds_addr(&s_v[buf][blk]), voff, rv4);
    }
  };

  // The first tiles' DMA goes out before anything else this workgroup loads.
#pragma unroll
  for (int i = 0; i < NBUF - 1; ++i) dma_tile(i, begin + i * kTile);

  const bool row_ok = R < rows;
  const int n = row_ok ? R / a.group : 0;
  const int head = hk * a.group + (row_ok ? R % a.group : 0);
  const bool wave_active = rb * a.rows_per_wg + wave * 32 < rows;

  // LDS byte offsets used by this lane, independent of the tile.
  // K rows blk*32 + col, logical chunk 2*kk + half.
  int k_row_base[2], k_swz[2];
#pragma unroll
  for (int blk = 0; blk < 2; ++blk) {
    const int row = blk * 32 + col;
    k_row_base[blk] = row * G::kRowBytes;
    k_swz[blk] = G::swz(row) ^ half;
  }
  // V transposed reads: lane j of each 16-lane group reads 8 bytes at row
  // (4*half + j/4) of a 4-row group, columns 4*(j%4) of a 16-column block.
  const int j16 = lane & 15, g16 = (lane >> 4) & 1;
  const int v_row_lane = 4 * half + (j16 >> 2);          // + 16*ks + 8*r
  const int v_chunk_lane = 2 * g16 + ((j16 & 3) >> 1);   // + 4*i
  const int v_byte_lane = (j16 & 1) * 8;

  // Only a split that reaches the tree's own rows needs the ancestor masks
  // (built while the first tile and the queries are in flight). The last
  // split always does, and it reports the tree's status. With a malformed
  // tree the other splits still run; the sequence's output is unspecified.
  if (end > L) {
    const bool ok = build_tree_loaded(N, my_parent, s_parent, s_anc, &s_bad);
    report_tree(a, b, ok, s == S - 1 && hk == 0 && rb == 0);
    if (!ok) {
      __builtin_amdgcn_s_waitcnt(0);      // no DMA may land after the workgroup ends
      return;
    }
  }

  f32x16 oacc[kDBlk];
#pragma unroll
  for (int i = 0; i < kDBlk; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[i][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  const float c = a.scale_log2;
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};

  // Queries and the first tiles have landed. (This also tells the compiler
  // that no load it issued is pending, so it adds no waits inside the loop.)
  __builtin_amdgcn_s_waitcnt(0);
  if (!row_ok) {
#pragma unroll
    for (int kk = 0; kk < kKSteps; ++kk) qreg[kk] = bf16x8{};
  }
  for (int t0 = begin, buf = 0; t0 < end; t0 += kTile, buf = buf + 1 == NBUF ? 0 : buf + 1) {
    __builtin_amdgcn_s_waitcnt(kVmWait);  // this wave's DMA into `buf` has landed
    __syncthreads();                      // everyone's has; the previous buffer is free
    dma_tile(buf == 0 ? NBUF - 1 : buf - 1, t0 + (NBUF - 1) * kTile);
    if (!wave_active) continue;
    const unsigned char* kt = s_k[buf];
    const unsigned char* vt = s_v[buf];

    // S^T (tokens x query rows), raw dot products; two independent chains.
    f32x16 sacc[2];
#pragma unroll
    for (int blk = 0; blk < 2; ++blk)
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[blk][r] = 0.f;
    // K operands are read one k-step ahead of the MFMAs that consume them.
    Pack8 ka[2][2];
#pragma unroll
    for (int blk = 0; blk < 2; ++blk)
      ka[0][blk].u = *reinterpret_cast<const uint4*>(kt + k_row_base[blk] + (k_swz[blk] << 4));
#pragma unroll
    for (int kk = 0; kk < kKSteps; ++kk) {
      if (kk + 1 < kKSteps) {
#pragma unroll
        for (int blk = 0; blk < 2; ++blk)
          ka[(kk + 1) & 1][blk].u = *reinterpret_cast<const uint4*>(
              kt + k_row_base[blk] + (((2 * (kk + 1)) ^ k_swz[blk]) << 4));
      }
#pragma unroll
      for (int blk = 0; blk < 2; ++blk)
        sacc[blk] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[kk & 1][blk].v, qreg[kk], sacc[blk], 0, 0, 0);
    }
    // Mask the tail, then the tile's row maximum (raw units; the scale is > 0).
    if (t0 + kTile > L) {
#pragma unroll
      for (int blk = 0; blk < 2; ++blk)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          sacc[blk][r] += mask_bias(t0 + blk * 32 + 8 * (r >> 2) + 4 * half + (r & 3), L, end, n, s_anc);
    }
    // Row maximum: one three-input max per two scores, in two chains.
    float mb[2] = {-INFINITY, -INFINITY};
#pragma unroll
    for (int blk = 0; blk < 2; ++blk)
#pragma unroll
      for (int r = 0; r < 16; r += 2) mb[blk] = max3_raw(mb[blk], sacc[blk][r], sacc[blk][r + 1]);
    const float m_tile = max_halves(max3_raw(mb[0], mb[1], mb[1])) * c;
    // Lazy rescale: move the reference only when the maximum rises by > 2^8.
    const bool grow = m_tile > m_run + kRescaleLog2;
    if (__builtin_expect(__ballot(grow) != 0, 0)) {
      if (grow) {
        const float alpha = fast_exp2(m_run - m_tile);
        l_run *= alpha;
#pragma unroll
        for (int i = 0; i < kDBlk; ++i)
#pragma unroll
          for (int r = 0; r < 16; ++r) oacc[i][r] *= alpha;
        m_run = m_tile;
      }
    }
    const float nm = m_run == -INFINITY ? 0.f : -m_run;
    bf16x8 pb[4];
    float l0 = 0.f, l1 = 0.f;
#pragma unroll
    for (int blk = 0; blk < 2; ++blk)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        bf16x8 v8;
#pragma unroll
        for (int e = 0; e < 8; ++e) v8[e] = (__bf16)fast_exp2(fmaf(sacc[blk][8 * j + e], c, nm));
        pb[blk * 2 + j] = v8;
        // Row sums of the probabilities as rounded for the MFMA (bf16 pairs).
#pragma unroll
        for (int e = 0; e < 8; e += 4) {
          l0 = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{v8[e], v8[e + 1]}, ones, l0, false);
          l1 = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{v8[e + 2], v8[e + 3]}, ones, l1, false);
        }
      }
    l_run += l0 + l1;

    // O^T += V^T P^T; the D/32 column blocks are independent chains.
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
#pragma unroll
      for (int i = 0; i < kDBlk; ++i) {
        Pack8 va;
#pragma unroll
        for (int r = 0; r < 2; ++r) {
          const int row = 16 * ks + 8 * r + v_row_lane;
          const int byte = G::offset(row, 4 * i + v_chunk_lane) + v_byte_lane;
          va.h[r] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(vt + byte));
        }
        oacc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va.v, pb[ks], oacc[i], 0, 0, 0);
      }
    }
  }

  __builtin_amdgcn_s_waitcnt(0);          // the ring's trailing DMAs land before exit
  if (!row_ok) return;
  const float l_tot = sum_halves(l_run);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  const float lse_nat = l_tot > 0.f ? (m_run + log2f(l_tot)) * kLn2 : -INFINITY;
  if (S == 1) {
    const int64_t obase = (((int64_t)b * a.n_max + n) * a.hq + head) * D;
#pragma unroll
    for (int i = 0; i < kDBlk; ++i)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int d0 = i * 32 + 8 * g4 + 4 * half;
        const float x0 = oacc[i][4 * g4] * inv, x1 = oacc[i][4 * g4 + 1] * inv;
        const float x2 = oacc[i][4 * g4 + 2] * inv, x3 = oacc[i][4 * g4 + 3] * inv;
        if (a.out_bf16) {
          uint2 pk;
          pk.x = pack_bf16x2(x0, x1);
          pk.y = pack_bf16x2(x2, x3);
          *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(a.o) + obase + d0) = pk;
        } else {
          *reinterpret_cast<float4*>(reinterpret_cast<float*>(a.o) + obase + d0) =
              make_float4(x0, x1, x2, x3);
        }
      }
    if (half == 0 && a.lse) a.lse[((int64_t)b * a.n_max + n) * a.hq + head] = lse_nat;
  } else {
    const int64_t pi = part_index(a, b, head, n, s);
#pragma unroll
    for (int i = 0; i < kDBlk; ++i)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int d0 = i * 32 + 8 * g4 + 4 * half;
        *reinterpret_cast<float4*>(a.part_o + pi * D + d0) =
            make_float4(oacc[i][4 * g4] * inv, oacc[i][4 * g4 + 1] * inv,
                        oacc[i][4 * g4 + 2] * inv, oacc[i][4 * g4 + 3] * inv);
      }
    if (half == 0) a.part_lse[pi] = lse_nat;
  }
}

// ---------------------------------------------------------------------------
// MFMA split kernel with 16 query rows per wave (v_mfma_f32_16x16x32_bf16).
//
// Same tile stream, LDS layout, tree mask and lazily rescaled online softmax
// as the 32-row kernel above (here a tile's row maxima are reduced only when a
// rescale could be due), at half the registers per wave, so that two 8-wave
// workgroups (four waves per SIMD) share a CU, and row blocks of up to 256
// rows fit one 16-wave workgroup with the rows spread evenly over the SIMDs.
// Wider trees take several row blocks of equal size (a multiple of 16 rows).
// The row blocks of one kv-head and split are hkv workgroup ids apart: with
// hkv a multiple of 8 the dispatcher, which deals workgroups to the 8 XCDs in
// turn, puts them on the same XCD, where they share its L2 for the K/V stream.
//
// Lane l = 16 g + c (c = l % 16, g = l / 16) owns query row c of its wave.
//   S^T = K Q^T, per 16-token block tb and 32-wide k-step ks:
//     A = K rows tb*16 + c, columns 32 ks + 8 g .. +7   (one 16-byte LDS read)
//     B = Q row c, columns 32 ks + 8 g .. +7             (registers)
//     D register r = score of token tb*16 + 4 g + r for row c
//   so a row's 64 scores sit in the four lanes c, c+16, c+32, c+48 and its
//   statistics reduce over lane xor 16 and xor 32.
//   O^T += V^T P^T, per 16-wide column block db and 32-token k-step kt, with
//   the k index 8 g + j standing for token 32 kt + 4 g + j (j < 4) or
//   32 kt + 16 + 4 g + (j - 4) (j >= 4): exactly the probabilities lane l
//   already holds from blocks 2 kt and 2 kt + 1, so P needs no exchange.
//     A = V^T: two transposed reads of 4 tokens x 16 columns per 16 lanes
//     D register r = O column 16 db + 4 g + r of row c
// At most 128 VGPRs (four waves per SIMD): two 8-wave workgroups share a CU
// whenever a launch has more workgroups than CUs.
template <int D, int NW>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(4))) void tree_attn_m16(Args a) {
  using G = TileGeo<D>;
  constexpr int kKSteps = D / 32;                  // k-steps for Q K^T
  constexpr int kDBlk = D / 16;                    // 16-column blocks of O^T
  constexpr int kDmaPerWave = G::kBlocks / NW;     // DMA blocks per wave per tensor
  constexpr int kKFrags = 4 * kKSteps;             // K operand fragments per tile
  constexpr int kVFrags = 2 * kDBlk;               // V^T operand fragments per tile
  constexpr int kAheadK = 4;                       // K reads in flight ahead of their MFMA
  constexpr int kAheadV = 4;                       // V^T reads in flight ahead of their MFMA
  static_assert(G::kBlocks % NW == 0, "tile must split evenly across waves");

  __shared__ int s_parent[CURE_MAX_TREE_NODES];
  __shared__ unsigned long long s_anc[CURE_MAX_TREE_NODES][kAncWords];
  __shared__ int s_bad;
  __shared__ __attribute__((aligned(1024))) unsigned char s_k[2][G::kTileBytes];
  __shared__ __attribute__((aligned(1024))) unsigned char s_v[2][G::kTileBytes];

  const int b = blockIdx.z;
  const int hk = blockIdx.x % a.hkv;
  const int rb = blockIdx.x / a.hkv;
  const int s = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int c = lane & 15, g = lane >> 4;

  // Query loads (need only the launch shape) and the parent entry go out with
  // the loads of the sequence's sizes.
  const int R = rb * a.rows_per_wg + wave * 16 + c;
  const bool r_in = R < a.n_max * a.group;
  bf16x8 qreg[kKSteps];
  {
    const int qn = r_in ? R / a.group : 0;
    const int qh = hk * a.group + (r_in ? R % a.group : 0);
    const uint16_t* qrow = reinterpret_cast<const uint16_t*>(a.q) +
                           (((int64_t)b * a.n_max + qn) * a.hq + qh) * D;
#pragma unroll
    for (int ks = 0; ks < kKSteps; ++ks) {
      Pack8 p;
      p.u = r_in ? *reinterpret_cast<const uint4*>(qrow + ks * 32 + g * 8)
                 : make_uint4(0, 0, 0, 0);
      qreg[ks] = p.v;
    }
  }
  const int my_parent = tid < a.n_max ? a.parent[(int64_t)b * a.n_max + tid] : -1;

  const int n_raw = a.n_nodes[b];
  const int L = a.ctx_len[b];
  const int64_t off = a.kv_off[b];
  asm volatile("" : : "s"(n_raw), "s"(L), "s"(off));
  const int N = min(n_raw, a.n_max);
  const int T = L + N;
  const int S = split_count(T, N, a.tps, a.max_splits);
  const int rows = N * a.group;
  if (S == 0) {                         // no nodes: nothing to compute; the empty tree is valid
    report_tree(a, b, true, s == 0 && hk == 0 && rb == 0);
    return;
  }
  if (s >= S || rb * a.rows_per_wg >= rows) return;

  const int begin = s * a.tps;
  const int end = (s == S - 1) ? T : begin + a.tps;

  const uint32_t seq_bytes = (uint32_t)T * (uint32_t)(a.hkv * G::kRowBytes);
  uint32_t src_off[kDmaPerWave];
#pragma unroll
  for (int j = 0; j < kDmaPerWave; ++j) {
    const int byte = (wave * kDmaPerWave + j) * 1024 + lane * 16;
    const int row = byte / G::kRowBytes;
    const int pchunk = (byte % G::kRowBytes) >> 4;
    const int lchunk = pchunk ^ G::swz(row);
    src_off[j] = (uint32_t)((row * a.hkv + hk) * G::kRowBytes + (lchunk << 4));
  }
  const uint32_t tok_bytes = (uint32_t)(a.hkv * G::kRowBytes);
  const i32x4 rk4 = raw_rsrc(reinterpret_cast<const uint16_t*>(a.k) + off * a.hkv * D, seq_bytes);
  const i32x4 rv4 = raw_rsrc(reinterpret_cast<const uint16_t*>(a.v) + off * a.hkv * D, seq_bytes);
  auto dma_tile = [&](int buf, int t0) {
    const bool live = t0 < end;
#pragma unroll
    for (int j = 0; j < kDmaPerWave; ++j) {
      const uint32_t voff = live ? src_off[j] + (uint32_t)t0 * tok_bytes : kOobOffset;
      const int blk = (wave * kDmaPerWave + j) * 1024;
      dma16(lds_addr(&s_k[buf][blk]), voff, rk4);
      dma16(lds_addr(&s_v[buf][blk]), voff, rv4);
    }
  };
  dma_tile(0, begin);

  // A row block may hold fewer rows than the workgroup has row waves.
  const bool own = wave * 16 < a.rows_per_wg;
  const bool row_ok = own && R < rows;
  const int n = row_ok ? R / a.group : 0;
  const int head = hk * a.group + (row_ok ? R % a.group : 0);
  const bool wave_active = own && rb * a.rows_per_wg + wave * 16 < rows;

  // LDS byte offsets of this lane's operands inside a tile.
  int k_off[4][kKSteps];                           // K: row tb*16 + c, chunk 4 ks + g
#pragma unroll
  for (int tb = 0; tb < 4; ++tb)
#pragma unroll
    for (int ks = 0; ks < kKSteps; ++ks) k_off[tb][ks] = G::offset(tb * 16 + c, 4 * ks + g);
  // V: within a 16-lane group, lane j = c addresses row 4 g + j / 4 (+16) of
  // the k-step's 32 tokens, columns 16 db + 4 (j % 4) .. +3.
  const int v_row = 4 * g + (c >> 2);
  const int v_chunk = (c & 3) >> 1;                // + 2 db
  const int v_byte = (c & 1) * 8;

  if (end > L) {
    const bool ok = build_tree_loaded(N, my_parent, s_parent, s_anc, &s_bad);
    report_tree(a, b, ok, s == S - 1 && hk == 0 && rb == 0);
    if (!ok) {
      __builtin_amdgcn_s_waitcnt(0);
      return;
    }
  }

  f32x4 oacc[kDBlk];
#pragma unroll
  for (int i = 0; i < kDBlk; ++i) oacc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;            // l_run: this lane's share of the row sum
  const float cs = a.scale_log2;
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};

  __builtin_amdgcn_s_waitcnt(0);
  if (!row_ok) {
#pragma unroll
    for (int ks = 0; ks < kKSteps; ++ks) qreg[ks] = bf16x8{};
  }
  for (int t0 = begin, buf = 0; t0 < end; t0 += kTile, buf ^= 1) {
    __builtin_amdgcn_s_waitcnt(0);        // this wave's DMA into `buf` has landed
    __syncthreads();                      // everyone's has; the other buffer is free
    dma_tile(buf ^ 1, t0 + kTile);
    if (!wave_active) continue;
    const unsigned char* kt = s_k[buf];
    const unsigned char* vt = s_v[buf];

    // Scores: four 16-token blocks, each a chain of kKSteps MFMAs. The K
    // operand reads run kAheadK fragments ahead of the MFMA that takes them,
    // so LDS latency overlaps the matrix core instead of stalling each MFMA.
    f32x4 sacc[4];
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) sacc[tb] = f32x4{0.f, 0.f, 0.f, 0.f};
    Pack8 kf[kKFrags];
#pragma unroll
    for (int i = 0; i < kAheadK; ++i) kf[i].u = *reinterpret_cast<const uint4*>(kt + k_off[i & 3][i >> 2]);
#pragma unroll
    for (int i = 0; i < kKFrags; ++i) {
      if (i + kAheadK < kKFrags) {
        const int j = i + kAheadK;
        kf[j].u = *reinterpret_cast<const uint4*>(kt + k_off[j & 3][j >> 2]);
      }
      sacc[i & 3] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[i].v, qreg[i >> 2], sacc[i & 3], 0, 0, 0);
    }
    // Left alone, the scheduler sinks each read back next to its MFMA; pin the
    // order: kAheadK reads, then alternate one MFMA (0x008) and one LDS read
    // (0x100), then the last kAheadK MFMAs.
    __builtin_amdgcn_sched_group_barrier(0x100, kAheadK, 0);
#pragma unroll
    for (int i = 0; i < kKFrags - kAheadK; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, kAheadK, 0);
    if (t0 + kTile > L) {
#pragma unroll
      for (int tb = 0; tb < 4; ++tb)
#pragma unroll
        for (int r = 0; r < 4; ++r) sacc[tb][r] += mask_bias(t0 + tb * 16 + 4 * g + r, L, end, n, s_anc);
    }
    // V^T fragment i: k-step i / kDBlk, column block i % kDBlk. The first
    // kAheadV go out before the exponentials, which then hide their latency.
    Pack8 vf[kVFrags];
    auto load_v = [&](Pack8& f, int i) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int row = 32 * (i / kDBlk) + 16 * h + v_row;
        const int byte = G::offset(row, 2 * (i % kDBlk) + v_chunk) + v_byte;
        f.h[h] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(vt + byte));
      }
    };
#pragma unroll
    for (int i = 0; i < kAheadV; ++i) load_v(vf[i], i);
    // Probabilities against the running reference m_run, bf16 for the P V
    // product, and the lane's share of the row sums from the same bf16 values.
    bf16x8 pb[2];                                  // k-steps kt = 0, 1 (blocks 2 kt, 2 kt + 1)
    float l0 = 0.f, l1 = 0.f;
    auto exps = [&](float nm) {
      l0 = 0.f;
      l1 = 0.f;
#pragma unroll
      for (int kt2 = 0; kt2 < 2; ++kt2) {
        bf16x8 v8;
#pragma unroll
        for (int j = 0; j < 8; ++j)
          v8[j] = (__bf16)fast_exp2(fmaf(sacc[2 * kt2 + (j >> 2)][j & 3], cs, nm));
        pb[kt2] = v8;
        l0 = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{v8[0], v8[1]}, ones, l0, false);
        l1 = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{v8[2], v8[3]}, ones, l1, false);
        l0 = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{v8[4], v8[5]}, ones, l0, false);
        l1 = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{v8[6], v8[7]}, ones, l1, false);
      }
    };
    // The reference moves lazily, when a row's maximum rises by more than 2^8.
    // The tile's row maxima are reduced only when that can happen: when a row
    // has no reference yet, or when some lane's probabilities sum to more than
    // 2^8 (otherwise none of them exceeds 2^8, so no row's maximum rose that
    // far). Up to rounding at the threshold the probabilities are those of
    // reducing the maximum on every tile.
    bool have = false, check = true;
    if (__ballot(m_run == -INFINITY) == 0) {
      exps(-m_run);
      have = true;
      check = __ballot(!(l0 + l1 <= 256.f)) != 0;
    }
    if (__builtin_expect(check, 0)) {
      // Row maximum over the lane's 16 scores (eight v_max3), then its 3 partners.
      float mb = max3_raw(sacc[0][0], sacc[0][1], sacc[0][2]);
#pragma unroll
      for (int i = 3; i < 15; i += 2)
        mb = max3_raw(mb, sacc[i >> 2][i & 3], sacc[(i + 1) >> 2][(i + 1) & 3]);
      mb = max3_raw(mb, sacc[3][3], sacc[3][3]);
      mb = max3_raw(mb, partner<16>(mb), mb);
      const float m_tile = max_halves(mb) * cs;
      const bool grow = m_tile > m_run + kRescaleLog2;
      const bool grew = __ballot(grow) != 0;
      if (grow) {
        const float alpha = fast_exp2(m_run - m_tile);
        l_run *= alpha;
#pragma unroll
        for (int i = 0; i < kDBlk; ++i) oacc[i] *= alpha;
        m_run = m_tile;
      }
      if (!have || grew) exps(m_run == -INFINITY ? 0.f : -m_run);
    }
    l_run += l0 + l1;

#pragma unroll
    for (int i = 0; i < kVFrags; ++i) {
      if (i + kAheadV < kVFrags) load_v(vf[i + kAheadV], i + kAheadV);
      oacc[i % kDBlk] =
          __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[i].v, pb[i / kDBlk], oacc[i % kDBlk], 0, 0, 0);
    }
  }

  __builtin_amdgcn_s_waitcnt(0);          // the trailing out-of-range DMA lands before exit
  if (!row_ok) return;
  float l_tot = l_run + partner<16>(l_run);
  l_tot = sum_halves(l_tot);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  const float lse_nat = l_tot > 0.f ? (m_run + log2f(l_tot)) * kLn2 : -INFINITY;
  if (S == 1) {
    const int64_t obase = (((int64_t)b * a.n_max + n) * a.hq + head) * D;
#pragma unroll
    for (int db = 0; db < kDBlk; ++db) {
      const int d0 = db * 16 + 4 * g;
      const float x0 = oacc[db][0] * inv, x1 = oacc[db][1] * inv;
      const float x2 = oacc[db][2] * inv, x3 = oacc[db][3] * inv;
      if (a.out_bf16) {
        uint2 pk;
        pk.x = pack_bf16x2(x0, x1);
        pk.y = pack_bf16x2(x2, x3);
        *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(a.o) + obase + d0) = pk;
      } else {
        *reinterpret_cast<float4*>(reinterpret_cast<float*>(a.o) + obase + d0) =
            make_float4(x0, x1, x2, x3);
      }
    }
    if (g == 0 && a.lse) a.lse[((int64_t)b * a.n_max + n) * a.hq + head] = lse_nat;
  } else {
    const int64_t pi = part_index(a, b, head, n, s);
#pragma unroll
    for (int db = 0; db < kDBlk; ++db)
      *reinterpret_cast<float4*>(a.part_o + pi * D + db * 16 + 4 * g) =
          make_float4(oacc[db][0] * inv, oacc[db][1] * inv, oacc[db][2] * inv, oacc[db][3] * inv);
    if (g == 0) a.part_lse[pi] = lse_nat;
  }
}

// ---------------------------------------------------------------------------
// MFMA split kernel with RG 16-row groups per wave (v_mfma_f32_16x16x32_bf16).
//
// The 16-row kernel's operand layout, tile stream, tree mask and online
// softmax, with two changes:
//  * each wave owns RG groups of 16 query rows, and every K fragment and V^T
//    fragment it reads from LDS feeds the MFMAs of all RG groups, so a tile's
//    LDS reads serve 16 RG rows per wave instead of 16 (LDS read bandwidth
//    co-bounds the K/V stream once a kv-head has more than ~128 rows);
//  * the K/V ring holds NBUF tiles, so NBUF - 1 tiles (32 KB each at head dim
//    128) are in flight while one is computed; only the first NDMA waves
//    issue the tile DMA (G::kBlocks / NDMA blocks per tensor each), and the
//    barrier after their wait releases the others.
// The block's ceil(rows_per_wg / 16) row groups are dealt so that the first
// n_full waves own RG groups each and the others RG - 1: waves w and w + 4
// share a SIMD, so with 8 waves every SIMD carries the same number of groups
// whenever the count allows (320 rows: 3 + 2 groups on each SIMD, where seven
// 3-group waves put 6 groups on three SIMDs and 3 on the fourth). A wave
// runs the tile loop's body instantiated for its own group count. Row r of a
// wave's group rg is query row rb * rows_per_wg + 16 (first + rg) + c, with
// first the wave's first group (lane l = 16 g + c as in the 16-row kernel).
template <int D, int NW, int RG, int NBUF, int NDMA, int HT, int WPE>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(WPE, WPE)))
void tree_attn_rg(Args a) {
  using G = TileGeo<D>;
  constexpr int kKSteps = D / 32;                  // k-steps for Q K^T
  constexpr int kDBlk = D / 16;                    // 16-column blocks of O^T
  constexpr int kDmaBlocks = G::kBlocks / NDMA;    // DMA blocks per DMA wave per tensor
  // The tile's 64 tokens are taken in HT steps of online softmax, each of
  // kTB 16-token blocks (scores) and kPV 32-token k-steps (P V).
  constexpr int kTB = 4 / HT;
  constexpr int kPV = 2 / HT;
  constexpr int kKFrags = kTB * kKSteps;           // K operand fragments per step
  constexpr int kVFrags = kPV * kDBlk;             // V^T operand fragments per step
  constexpr int kAheadK = 4;                       // K reads in flight ahead of their MFMAs
  constexpr int kAheadV = 4;                       // V^T reads in flight ahead of their MFMAs
  // Each iteration waits until its tile has landed while the NBUF - 2 tiles
  // issued after it may still be in flight (2 instructions per block).
  constexpr int kVmWait = waitcnt_vm((NBUF - 2) * 2 * kDmaBlocks);
  static_assert(G::kBlocks % NDMA == 0 && NDMA <= NW, "DMA blocks split evenly over DMA waves");
  static_assert((NBUF - 2) * 2 * kDmaBlocks < 64, "vmcnt holds 6 bits");
  static_assert(NBUF >= 2, "a ring of at least two tiles");
  static_assert(HT == 1 || HT == 2, "one or two softmax steps per tile");

  __shared__ int s_parent[CURE_MAX_TREE_NODES];
  __shared__ unsigned long long s_anc[CURE_MAX_TREE_NODES][kAncWords];
  __shared__ int s_bad;
  __shared__ __attribute__((aligned(1024))) unsigned char s_k[NBUF][G::kTileBytes];
  __shared__ __attribute__((aligned(1024))) unsigned char s_v[NBUF][G::kTileBytes];

  const int b = blockIdx.z;
  const int hk = blockIdx.x % a.hkv;
  const int rb = blockIdx.x / a.hkv;
  const int s = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int c = lane & 15, g = lane >> 4;
  const int groups_wg = (a.rows_per_wg + 15) / 16;
  const int n_full = min(NW, max(0, groups_wg - (RG - 1) * NW));
  const int my_groups = wave < n_full ? RG : RG - 1;
  const int first = wave < n_full ? RG * wave : RG * n_full + (RG - 1) * (wave - n_full);
  const int wrow = rb * a.rows_per_wg + 16 * first;        // this wave's first row

  // Query loads (they need only the launch shape) and the parent entry go out
  // with the loads of the sequence's sizes.
  bf16x8 qreg[RG][kKSteps];
#pragma unroll
  for (int rg = 0; rg < RG; ++rg) {
    const int R = wrow + 16 * rg + c;
    const bool r_in = rg < my_groups && R < a.n_max * a.group;
    const int qn = r_in ? R / a.group : 0;
    const int qh = hk * a.group + (r_in ? R % a.group : 0);
    const uint16_t* qrow = reinterpret_cast<const uint16_t*>(a.q) +
                           (((int64_t)b * a.n_max + qn) * a.hq + qh) * D;
#pragma unroll
    for (int ks = 0; ks < kKSteps; ++ks) {
      Pack8 p;
      p.u = r_in ? *reinterpret_cast<const uint4*>(qrow + ks * 32 + g * 8)
                 : make_uint4(0, 0, 0, 0);
      qreg[rg][ks] = p.v;
    }
  }
  const int my_parent = tid < a.n_max ? a.parent[(int64_t)b * a.n_max + tid] : -1;

  const int n_raw = a.n_nodes[b];
  const int L = a.ctx_len[b];
  const int64_t off = a.kv_off[b];
  asm volatile("" : : "s"(n_raw), "s"(L), "s"(off));
  const int N = min(n_raw, a.n_max);
  const int T = L + N;
  const int S = split_count(T, N, a.tps, a.max_splits);
  const int rows = N * a.group;
  if (S == 0) {                         // no nodes: nothing to compute; the empty tree is valid
    report_tree(a, b, true, s == 0 && hk == 0 && rb == 0);
    return;
  }
  if (s >= S || rb * a.rows_per_wg >= rows) return;

  const int begin = s * a.tps;
  const int end = (s == S - 1) ? T : begin + a.tps;

  const uint32_t seq_bytes = (uint32_t)T * (uint32_t)(a.hkv * G::kRowBytes);
  const bool dma_wave = wave < NDMA;
  uint32_t src_off[kDmaBlocks];
#pragma unroll
  for (int j = 0; j < kDmaBlocks; ++j) {
    const int byte = ((dma_wave ? wave : 0) * kDmaBlocks + j) * 1024 + lane * 16;
    const int row = byte / G::kRowBytes;
    const int pchunk = (byte % G::kRowBytes) >> 4;
    const int lchunk = pchunk ^ G::swz(row);
    src_off[j] = (uint32_t)((row * a.hkv + hk) * G::kRowBytes + (lchunk << 4));
  }
  const uint32_t tok_bytes = (uint32_t)(a.hkv * G::kRowBytes);
  const i32x4 rk4 = raw_rsrc(reinterpret_cast<const uint16_t*>(a.k) + off * a.hkv * D, seq_bytes);
  const i32x4 rv4 = raw_rsrc(reinterpret_cast<const uint16_t*>(a.v) + off * a.hkv * D, seq_bytes);
  // Tiles at or past the split's end are still issued (at an out-of-range
  // offset, which reads nothing) so that every iteration of a DMA wave has
  // the same number of DMAs in flight.
  auto dma_tile = [&](int buf, int t0) {
    if (!dma_wave) return;
    const bool live = t0 < end;
#pragma unroll
    for (int j = 0; j < kDmaBlocks; ++j) {
      const uint32_t voff = live ? src_off[j] + (uint32_t)t0 * tok_bytes : kOobOffset;
      const int blk = (wave * kDmaBlocks + j) * 1024;
      dma16(lds_addr(&s_k[buf][blk]), voff, rk4);
      dma16(lds_addr(&s_v[buf][blk]), voff, rv4);
    }
  };
#pragma unroll
  for (int i = 0; i < NBUF - 1; ++i) dma_tile(i, begin + i * kTile);

  // A row block may hold fewer rows than the workgroup has row waves.
  bool row_ok[RG];
  int n_of[RG], head_of[RG];
#pragma unroll
  for (int rg = 0; rg < RG; ++rg) {
    const int R = wrow + 16 * rg + c;
    row_ok[rg] = rg < my_groups && 16 * (first + rg) < a.rows_per_wg && R < rows;
    n_of[rg] = row_ok[rg] ? R / a.group : 0;
    head_of[rg] = hk * a.group + (row_ok[rg] ? R % a.group : 0);
  }
  const bool wave_active = my_groups > 0 && 16 * first < a.rows_per_wg && wrow < rows;

  // LDS byte offsets of this lane's operands inside a tile. The swizzle takes
  // only the row's low three bits, so a 16-row block's offset is a constant
  // (an instruction immediate) away from the first block's.
  int k_off[kKSteps];                              // K: row tb*16 + c, chunk 4 ks + g
#pragma unroll
  for (int ks = 0; ks < kKSteps; ++ks) k_off[ks] = G::offset(c, 4 * ks + g);
  const int v_row = 4 * g + (c >> 2);
  int v_off[kDBlk];                                // V^T: rows v_row (+16 h, +32 kt), 16-col block db
#pragma unroll
  for (int db = 0; db < kDBlk; ++db) v_off[db] = G::offset(v_row, 2 * db + ((c & 3) >> 1)) + (c & 1) * 8;

  if (end > L) {
    const bool ok = build_tree_loaded(N, my_parent, s_parent, s_anc, &s_bad);
    report_tree(a, b, ok, s == S - 1 && hk == 0 && rb == 0);
    if (!ok) {
      __builtin_amdgcn_s_waitcnt(0);
      return;
    }
  }

  f32x4 oacc[RG][kDBlk];
#pragma unroll
  for (int rg = 0; rg < RG; ++rg)
#pragma unroll
    for (int i = 0; i < kDBlk; ++i) oacc[rg][i] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run[RG], l_run[RG];
#pragma unroll
  for (int rg = 0; rg < RG; ++rg) {
    m_run[rg] = -INFINITY;
    l_run[rg] = 0.f;
  }
  const float cs = a.scale_log2;
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};

  // Queries and the first tiles have landed. (This also tells the compiler
  // that no load it issued is pending, so it adds no waits inside the loop.)
  __builtin_amdgcn_s_waitcnt(0);
#pragma unroll
  for (int rg = 0; rg < RG; ++rg)
    if (!row_ok[rg]) {
#pragma unroll
      for (int ks = 0; ks < kKSteps; ++ks) qreg[rg][ks] = bf16x8{};
    }
  for (int t0 = begin, buf = 0; t0 < end; t0 += kTile, buf = buf + 1 == NBUF ? 0 : buf + 1) {
    __builtin_amdgcn_s_waitcnt(kVmWait);  // this wave's DMA into `buf` has landed
    __syncthreads();                      // everyone's has; the previous buffer is free
    dma_tile(buf == 0 ? NBUF - 1 : buf - 1, t0 + (NBUF - 1) * kTile);
    if (!wave_active) continue;
    const unsigned char* kt = s_k[buf];
    const unsigned char* vt = s_v[buf];
    // The tile's work for NG row groups (NG = RG or RG - 1, this wave's count).
    auto tile_body = [&](auto ng) {
      constexpr int NG = decltype(ng)::value;
#pragma unroll
      for (int hs = 0; hs < HT; ++hs) {
        // Scores of this step's kTB 16-token blocks x NG row groups, each a
        // chain of kKSteps MFMAs; every K fragment feeds all NG groups.
        f32x4 sacc[NG][kTB];
#pragma unroll
        for (int rg = 0; rg < NG; ++rg)
#pragma unroll
          for (int tb = 0; tb < kTB; ++tb) sacc[rg][tb] = f32x4{0.f, 0.f, 0.f, 0.f};
        Pack8 kf[kKFrags];
        auto load_k = [&](Pack8& f, int i) {
          f.u = *reinterpret_cast<const uint4*>(kt + (hs * kTB + i % kTB) * 16 * G::kRowBytes +
                                                k_off[i / kTB]);
        };
#pragma unroll
        for (int i = 0; i < kAheadK; ++i) load_k(kf[i], i);
#pragma unroll
        for (int i = 0; i < kKFrags; ++i) {
          if (i + kAheadK < kKFrags) load_k(kf[i + kAheadK], i + kAheadK);
#pragma unroll
          for (int rg = 0; rg < NG; ++rg)
            sacc[rg][i % kTB] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[i].v, qreg[rg][i / kTB],
                                                                       sacc[rg][i % kTB], 0, 0, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x100, kAheadK, 0);
#pragma unroll
        for (int i = 0; i < kKFrags - kAheadK; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, NG, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, NG * kAheadK, 0);
        const int s0 = t0 + hs * 16 * kTB;             // first token of this step
        if (s0 + 16 * kTB > L) {
#pragma unroll
          for (int rg = 0; rg < NG; ++rg)
#pragma unroll
            for (int tb = 0; tb < kTB; ++tb)
#pragma unroll
              for (int r = 0; r < 4; ++r) {
                const int tok = s0 + tb * 16 + 4 * g + r;
                sacc[rg][tb][r] += mask_bias(tok, L, end, n_of[rg], s_anc);
              }
        }
        // V^T fragment i: k-step hs * kPV + i / kDBlk, column block i % kDBlk.
        Pack8 vf[kVFrags];
        auto load_v = [&](Pack8& f, int i) {
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int rows0 = 32 * (hs * kPV + i / kDBlk) + 16 * h;   // multiple of 8: swizzle-free
            f.h[h] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (lds_i16x4*)(vt + rows0 * G::kRowBytes + v_off[i % kDBlk]));
          }
        };
#pragma unroll
        for (int i = 0; i < kAheadV; ++i) load_v(vf[i], i);
        // Probabilities of group rg against its running reference, bf16 for
        // the P V product, and the lane's share of the row sum from them.
        bf16x8 pb[NG][kPV];
        float lsum[NG];
        auto exps = [&](int rg, float nm) {
          float l0 = 0.f, l1 = 0.f;
#pragma unroll
          for (int kt2 = 0; kt2 < kPV; ++kt2) {
            bf16x8 v8;
#pragma unroll
            for (int j = 0; j < 8; ++j)
              v8[j] = (__bf16)fast_exp2(fmaf(sacc[rg][2 * kt2 + (j >> 2)][j & 3], cs, nm));
            pb[rg][kt2] = v8;
            l0 = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{v8[0], v8[1]}, ones, l0, false);
            l1 = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{v8[2], v8[3]}, ones, l1, false);
            l0 = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{v8[4], v8[5]}, ones, l0, false);
            l1 = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{v8[6], v8[7]}, ones, l1, false);
          }
          lsum[rg] = l0 + l1;
        };
        // The lazy rescale of the 16-row kernel: each group's reference moves
        // when its row maximum rises by more than 2^8, and the maxima are
        // reduced only when that can happen (a row without a reference, or a
        // lane whose probabilities sum to more than 2^8).
        bool no_ref = false;
#pragma unroll
        for (int rg = 0; rg < NG; ++rg) no_ref |= m_run[rg] == -INFINITY;
        bool have = false, check = true;
        if (__ballot(no_ref) == 0) {
          bool big = false;
#pragma unroll
          for (int rg = 0; rg < NG; ++rg) {
            exps(rg, -m_run[rg]);
            big |= !(lsum[rg] <= 256.f);
          }
          have = true;
          check = __ballot(big) != 0;
        }
        if (__builtin_expect(check, 0)) {
          // Row maxima (the lane's 4 kTB scores, then its 3 partners).
          float m_tile[NG];
          bool grow_any = false;
#pragma unroll
          for (int rg = 0; rg < NG; ++rg) {
            float mb = max3_raw(sacc[rg][0][0], sacc[rg][0][1], sacc[rg][0][2]);
#pragma unroll
            for (int i = 3; i + 1 < 4 * kTB; i += 2)
              mb = max3_raw(mb, sacc[rg][i >> 2][i & 3], sacc[rg][(i + 1) >> 2][(i + 1) & 3]);
            mb = max3_raw(mb, sacc[rg][kTB - 1][3], sacc[rg][kTB - 1][3]);
            mb = max3_raw(mb, partner<16>(mb), mb);
            m_tile[rg] = max_halves(mb) * cs;
            grow_any |= m_tile[rg] > m_run[rg] + kRescaleLog2;
          }
          const bool grew = __ballot(grow_any) != 0;
          if (grew) {
#pragma unroll
            for (int rg = 0; rg < NG; ++rg) {
              if (m_tile[rg] > m_run[rg] + kRescaleLog2) {
                const float alpha = fast_exp2(m_run[rg] - m_tile[rg]);
                l_run[rg] *= alpha;
#pragma unroll
                for (int i = 0; i < kDBlk; ++i) oacc[rg][i] *= alpha;
                m_run[rg] = m_tile[rg];
              }
            }
          }
          if (!have || grew) {
#pragma unroll
            for (int rg = 0; rg < NG; ++rg) exps(rg, m_run[rg] == -INFINITY ? 0.f : -m_run[rg]);
          }
        }
#pragma unroll
        for (int rg = 0; rg < NG; ++rg) l_run[rg] += lsum[rg];
#pragma unroll
        for (int i = 0; i < kVFrags; ++i) {
          if (i + kAheadV < kVFrags) load_v(vf[i + kAheadV], i + kAheadV);
#pragma unroll
          for (int rg = 0; rg < NG; ++rg)
            oacc[rg][i % kDBlk] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                vf[i].v, pb[rg][i / kDBlk], oacc[rg][i % kDBlk], 0, 0, 0);
        }
      }
    };
    if (my_groups == RG) tile_body(std::integral_constant<int, RG>{});
    else tile_body(std::integral_constant<int, (RG > 1 ? RG - 1 : 1)>{});
  }

  __builtin_amdgcn_s_waitcnt(0);          // the ring's trailing DMAs land before exit
#pragma unroll
  for (int rg = 0; rg < RG; ++rg) {
    if (!row_ok[rg]) continue;
    const int n = n_of[rg], head = head_of[rg];
    float l_tot = l_run[rg] + partner<16>(l_run[rg]);
    l_tot = sum_halves(l_tot);
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    const float lse_nat = l_tot > 0.f ? (m_run[rg] + log2f(l_tot)) * kLn2 : -INFINITY;
    if (S == 1) {
      const int64_t obase = (((int64_t)b * a.n_max + n) * a.hq + head) * D;
#pragma unroll
      for (int db = 0; db < kDBlk; ++db) {
        const int d0 = db * 16 + 4 * g;
        const float x0 = oacc[rg][db][0] * inv, x1 = oacc[rg][db][1] * inv;
        const float x2 = oacc[rg][db][2] * inv, x3 = oacc[rg][db][3] * inv;
        if (a.out_bf16) {
          uint2 pk;
          pk.x = pack_bf16x2(x0, x1);
          pk.y = pack_bf16x2(x2, x3);
          *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(a.o) + obase + d0) = pk;
        } else {
          *reinterpret_cast<float4*>(reinterpret_cast<float*>(a.o) + obase + d0) =
              make_float4(x0, x1, x2, x3);
        }
      }
      if (g == 0 && a.lse) a.lse[((int64_t)b * a.n_max + n) * a.hq + head] = lse_nat;
    } else {
      const int64_t pi = part_index(a, b, head, n, s);
#pragma unroll
      for (int db = 0; db < kDBlk; ++db)
        *reinterpret_cast<float4*>(a.part_o + pi * D + db * 16 + 4 * g) =
            make_float4(oacc[rg][db][0] * inv, oacc[rg][db][1] * inv, oacc[rg][db][2] * inv,
                        oacc[rg][db][3] * inv);
      if (g == 0) a.part_lse[pi] = lse_nat;
    }
  }
}

// ---------------------------------------------------------------------------
// LSE merge: one wave per output row (b, n, head).
//
// A split's partial row is D floats = D/4 lanes of float4, so one load
// instruction covers 64/(D/4) splits (2 at D=128, 4 at D=64). A batch of NB
// such loads, with each split's LSE alongside, is issued before anything is
// reduced, and NB is the smallest of 2, 4, 8 that covers the launch's largest
// split count when it can: the partials then take one memory round trip,
// with no more registers held than that needs. When every sequence has the
// launch's largest split count that batch goes out with the loads of the
// sequence's sizes; otherwise (kOwnSplits, a ragged batch) the sizes come
// first and each row reads only its own splits' slots, instead of fetching
// slots it would discard. The lane groups holding different splits are
// combined with xor shuffles at the end.
template <int D, int NB, bool kOwnSplits>
__global__ __launch_bounds__(256) void attn_merge(Args a) {
  constexpr int kLanesPerSplit = D / 4;
  constexpr int kSplitsPerLoad = kWave / kLanesPerSplit;
  constexpr int kSplitsPerBatch = kSplitsPerLoad * NB;
  // Grid (heads / 4, n_max, batch): the row's coordinates come straight from
  // the block index (no 64-bit divisions).
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int head = blockIdx.x * 4 + wave;
  const int n = blockIdx.y;
  const int b = blockIdx.z;
  if (head >= a.hq) return;
  const int64_t p0 = part_index(a, b, head, n, 0);
  const int sub = lane / kLanesPerSplit;            // which split of a load this lane holds
  const int col = (lane % kLanesPerSplit) * 4;      // its four output columns

  // The first batch of partials is loaded together with the sequence's sizes
  // (its addresses need neither): one memory round trip. Slots past the
  // sequence's own split count hold stale data and are masked out below.
  float4 v[NB];
  float l[NB];
  auto load_batch = [&](int s0, int limit) {
#pragma unroll
    for (int u = 0; u < NB; ++u) {
      const int sp = s0 + u * kSplitsPerLoad + sub;
      const bool ok = sp < limit;
      v[u] = ok ? *reinterpret_cast<const float4*>(a.part_o + (p0 + sp) * D + col)
                : make_float4(0.f, 0.f, 0.f, 0.f);
      l[u] = ok ? a.part_lse[p0 + sp] : -INFINITY;
    }
  };
  if (!kOwnSplits) load_batch(0, a.max_splits);
  const int n_raw = a.n_nodes[b];
  const int L = a.ctx_len[b];
  const int N = min(n_raw, a.n_max);
  if (n >= N) return;
  const int S = split_count(L + N, N, a.tps, a.max_splits);
  if (S <= 1) return;
  if (kOwnSplits) {
    load_batch(0, S);
  } else {
    // Slots past this sequence's own split count get zero weight (the plan
    // comes from host copies of the sizes, so this cannot be taken for granted).
#pragma unroll
    for (int u = 0; u < NB; ++u) {
      if (u * kSplitsPerLoad + sub >= S) {
        v[u] = make_float4(0.f, 0.f, 0.f, 0.f);
        l[u] = -INFINITY;
      }
    }
  }
  // Reference maximum: from the loaded batch when it holds every split, else
  // from all of the row's LSEs.
  float m = -INFINITY;
  if (S <= kSplitsPerBatch) {
#pragma unroll
    for (int u = 0; u < NB; ++u) m = fmaxf(m, l[u]);
  } else {
    for (int sp = lane; sp < S; sp += kWave) m = fmaxf(m, a.part_lse[p0 + sp]);
  }
  m = wave_max(m);
  const float ms = m == -INFINITY ? 0.f : m;     // empty splits (lse = -inf) weigh 0

  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  float wsum = 0.f;
  for (int s0 = 0;;) {
#pragma unroll
    for (int u = 0; u < NB; ++u) {
      const float w = fast_exp2((l[u] - ms) * kLog2e);
      wsum += w;
      acc.x = fmaf(w, v[u].x, acc.x);
      acc.y = fmaf(w, v[u].y, acc.y);
      acc.z = fmaf(w, v[u].z, acc.z);
      acc.w = fmaf(w, v[u].w, acc.w);
    }
    s0 += kSplitsPerBatch;
    if (s0 >= S) break;
    load_batch(s0, S);
  }
  if (kLanesPerSplit == 16) {                       // lane groups 16 apart
    acc.x += partner<16>(acc.x);
    acc.y += partner<16>(acc.y);
    acc.z += partner<16>(acc.z);
    acc.w += partner<16>(acc.w);
    wsum += partner<16>(wsum);
  }
  acc.x = sum_halves(acc.x);                        // and 32 apart
  acc.y = sum_halves(acc.y);
  acc.z = sum_halves(acc.z);
  acc.w = sum_halves(acc.w);
  wsum = sum_halves(wsum);
  if (sub != 0) return;
  const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
  const int64_t obase = (((int64_t)b * a.n_max + n) * a.hq + head) * D + col;
  store_out(a, obase, acc.x * inv);
  store_out(a, obase + 1, acc.y * inv);
  store_out(a, obase + 2, acc.z * inv);
  store_out(a, obase + 3, acc.w * inv);
  if (lane == 0 && a.lse) a.lse[((int64_t)b * a.n_max + n) * a.hq + head] =
      wsum > 0.f ? m + logf(wsum) : -INFINITY;
}

// Status of a launch with no tree nodes at all: every sequence's (empty)
// tree is valid. A fill kernel rather than a memset, so that the call stays
// capturable in a graph.
__global__ __launch_bounds__(256) void tree_status_ok(int32_t* status, int batch) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < batch) status[i] = CURE_OK;
}

// ---------------------------------------------------------------------------
// Host-side plan: tokens per split and the launch shape.
struct Plan {
  bool mfma;
  bool rows16;        // MFMA kernel with 16 query rows per wave
  bool rows48;        // MFMA kernel with three 16-row groups per wave (tree_attn_rg)
  int nw;             // waves per workgroup (MFMA kernel)
  int rows_per_wg;
  int row_blocks;
  int tps;
  int max_splits;
  bool uniform_splits;  // every sequence with nodes has max_splits splits (host sizes)
};

// The three-row-group kernel as instantiated: 8 waves of up to 48 query rows
// (one workgroup per CU, a two-tile ring), two 32-token softmax steps per
// tile; planned for 257 - 384 rows.
constexpr int kRg3Waves = 8;
constexpr int kRg3Rows = kRg3Waves * 48;

// MFMA workgroups one CU holds at once: bounded by LDS (the K/V ring plus the
// tree masks) and by registers (about 220 VGPRs per lane at head dim 128, so
// two waves per SIMD; about 120 at head dim 64, four waves per SIMD).
int mfma_wgs_per_cu(int d, int nw, bool rows16, bool rows48) {
  if (rows48) return 1;
  constexpr int kLdsPerCu = 160 * 1024;
  const int stages = rows16 ? 2 : kStages;
  const int lds = 2 * stages * kTile * d * 2 +
                  CURE_MAX_TREE_NODES * (4 + kAncWords * 8) + 64;
  const int by_lds = kLdsPerCu / lds;
  // 16-row waves hold about half the registers: four waves per SIMD. The
  // 8-wave 16-row kernel is planned at one workgroup per CU all the same:
  // the longer splits halve the partial rows the merge reads, and a second
  // workgroup per CU measured no faster.
  const int by_regs = rows16 ? 8 / nw : (d == 128 ? 8 : 16) / nw;
  return std::max(1, std::min(by_lds, by_regs));
}

Plan make_plan(int32_t batch, int32_t hq, int32_t hkv, int32_t d, int32_t n_max,
               const int32_t* host_ctx_len, const int32_t* host_n_nodes, int32_t kv_split,
               bool mfma) {
  Plan p{};
  p.mfma = mfma;
  const int group = hq / hkv;
  const int rows = n_max * group;
  // Head dim 128: the 16-row kernel, in balanced row blocks of at most 256
  // rows (8 waves up to 128 rows, else 16), except for 257 - 384 rows, which
  // one workgroup of the three-row-group kernel covers. Per call at 8k
  // context x 8 sequences: 320 rows 126 µs against 144 for two 160-row
  // blocks of the 16-row kernel, 352 rows 139 against 151; at 224 and 256
  // rows the 16-row kernel's single block is ahead (103 vs 106, 109 vs 113).
  // Head dim 64: the 16-row kernel up to 128 rows, else the 32-row kernel.
  p.rows48 = mfma && d == 128 && rows > 256 && rows <= kRg3Rows;
  p.rows16 = mfma && !p.rows48 && (d == 128 || rows <= 128);
  if (p.rows48) {
    // 257 - 384 rows: one block of eight waves of two or three 16-row groups,
    // so each K/V tile is streamed once per kv-head (two 16-row blocks would
    // stream it twice) and every LDS operand read feeds two or three row
    // groups. The block holds exactly the launch's row groups, so the kernel
    // deals them evenly over the SIMDs.
    p.row_blocks = 1;
    p.rows_per_wg = (rows + 15) / 16 * 16;
    p.nw = kRg3Waves;
  } else if (p.rows16) {
    // Row blocks of at most 256 rows, balanced, in multiples of 16.
    p.row_blocks = (rows + 255) / 256;
    p.rows_per_wg = ((rows + p.row_blocks - 1) / p.row_blocks + 15) / 16 * 16;
    p.nw = p.rows_per_wg > 128 ? 16 : 8;
  } else {
    if (mfma) {
      p.nw = 8;
      p.rows_per_wg = 32 * p.nw;
    } else {
      p.nw = kValuWaves;
      p.rows_per_wg = kValuRows;
    }
    p.row_blocks = std::max(1, (rows + p.rows_per_wg - 1) / p.rows_per_wg);
  }
  int64_t t_max = 0, t_sum = 0;
  for (int b = 0; b < batch; ++b) {
    const int N = std::min(host_n_nodes[b], n_max);
    if (N <= 0) continue;
    const int64_t T = (int64_t)host_ctx_len[b] + N;
    t_max = std::max(t_max, T);
    t_sum += T;
  }
  const auto round_tile = [](int64_t t) {
    return std::max<int64_t>(kTile, (t + kTile - 1) / kTile * kTile);
  };
  // Workgroups of one launch: splits of every sequence x kv-heads x row blocks.
  const auto workgroups = [&](int64_t tps) {
    int64_t c = 0;
    for (int b = 0; b < batch; ++b) {
      const int N = std::min(host_n_nodes[b], n_max);
      if (N > 0) c += ((int64_t)host_ctx_len[b] + N + tps - 1) / tps;
    }
    return c * hkv * p.row_blocks;
  };
  const int64_t slots =
      (int64_t)(mfma ? mfma_wgs_per_cu(d, p.nw, p.rows16, p.rows48) : 2) * device_cu_count();
  // The shortest split (at least kMinTps tokens) whose workgroups are all
  // resident at once, so no workgroup waits for a second round. A batch with
  // more sequence x head pairs than that gets a single split per sequence.
  const auto shortest_resident_split = [&]() {
    const int64_t hi = round_tile(t_max);
    const int64_t lo = round_tile(std::max<int64_t>(
        kMinTps, (t_sum * hkv * p.row_blocks + slots - 1) / std::max<int64_t>(1, slots)));
    if (lo >= hi || workgroups(hi) > slots) return hi;
    // workgroups() falls as tps grows: bisect over multiples of the tile.
    int64_t a = lo / kTile, z = hi / kTile;         // workgroups(z * kTile) <= slots
    while (a < z) {
      const int64_t m = (a + z) / 2;
      if (workgroups(m * kTile) <= slots) z = m;
      else a = m + 1;
    }
    return z * kTile;
  };
  int64_t tps;
  if (kv_split > 0) {
    tps = round_tile((t_max + kv_split - 1) / kv_split);
  } else {
    tps = shortest_resident_split();
    // A small launch (even the shortest splits leave most CUs idle, as for one
    // sequence) cuts the 16-row kernel's rows into more blocks, of at least 32
    // rows: the blocks of one kv-head and split are hkv workgroup ids apart,
    // so they share an XCD's L2 for the K/V stream, and more CUs stream it
    // (one sequence at 128 rows: 72 -> 216 workgroups).
    const int64_t fits = slots / std::max<int64_t>(1, workgroups(tps));
    if (p.rows16 && fits >= 2 && rows >= 64) {
      const int blocks = (int)std::min<int64_t>((int64_t)p.row_blocks * fits, rows / 32);
      if (blocks > p.row_blocks) {
        p.rows_per_wg = ((rows + blocks - 1) / blocks + 15) / 16 * 16;
        p.row_blocks = (rows + p.rows_per_wg - 1) / p.rows_per_wg;
        p.nw = p.rows_per_wg > 128 ? 16 : 8;
        tps = shortest_resident_split();
      }
    }
  }
  // Splits index the grid's y dimension (at most kMaxGridY).
  tps = std::max<int64_t>(tps, round_tile((t_max + kMaxGridY - 1) / kMaxGridY));
  p.tps = (int)std::min<int64_t>(tps, INT32_MAX / 2);
  p.max_splits = t_max > 0 ? (int)((t_max + p.tps - 1) / p.tps) : 0;
  p.uniform_splits = true;
  for (int b = 0; b < batch; ++b) {
    const int N = std::min(host_n_nodes[b], n_max);
    if (N <= 0) continue;
    const int64_t T = (int64_t)host_ctx_len[b] + N;
    if ((T + p.tps - 1) / p.tps < p.max_splits) p.uniform_splits = false;
  }
  return p;
}

size_t plan_workspace(const Plan& p, int32_t batch, int32_t hq, int32_t d, int32_t n_max) {
  if (p.max_splits <= 1) return 0;
  const size_t parts = (size_t)batch * hq * n_max * p.max_splits;
  return align_up(parts * d * sizeof(float), 256) + align_up(parts * sizeof(float), 256);
}

bool use_mfma(int32_t dtype, int32_t d, uint32_t flags) {
  return dtype == CURE_BF16 && (d == 64 || d == 128) && !(flags & CURE_ATTN_FORCE_VALU);
}

}  // namespace
}  // namespace cure

using namespace cure;

extern "C" size_t cure_tree_attn_workspace_size(int32_t batch, int32_t hq, int32_t hkv,
                                                int32_t d, int32_t n_max,
                                                const int32_t* host_ctx_len,
                                                const int32_t* host_n_nodes,
                                                int32_t kv_split) {
  if (batch <= 0 || hq <= 0 || hkv <= 0 || hq % hkv || n_max <= 0 || !host_ctx_len ||
      !host_n_nodes)
    return 0;
  // The MFMA and VALU plans may differ in row blocking; report the larger need.
  const Plan pm = make_plan(batch, hq, hkv, d, n_max, host_ctx_len, host_n_nodes, kv_split, true);
  const Plan pv = make_plan(batch, hq, hkv, d, n_max, host_ctx_len, host_n_nodes, kv_split, false);
  return std::max(plan_workspace(pm, batch, hq, d, n_max), plan_workspace(pv, batch, hq, d, n_max));
}

extern "C" cure_status cure_tree_attn(const void* q, const void* k, const void* v, void* o,
                                      float* lse, int32_t dtype, int32_t out_dtype,
                                      int32_t batch, int32_t hq, int32_t hkv, int32_t d,
                                      float scale, const int64_t* kv_off,
                                      const int32_t* ctx_len, const int32_t* n_nodes,
                                      const int32_t* parent, int32_t n_max,
                                      const int32_t* host_ctx_len,
                                      const int32_t* host_n_nodes, int32_t kv_split,
                                      uint32_t flags, int32_t* tree_status, void* workspace,
                                      size_t workspace_bytes, void* stream) {
  if (dtype != CURE_F32 && dtype != CURE_BF16) return CURE_ERR_INVALID_ARG;
  if (out_dtype != CURE_F32 && out_dtype != CURE_BF16) return CURE_ERR_INVALID_ARG;
  if (batch < 0 || hq <= 0 || hkv <= 0 || n_max < 0 || kv_split < 0) return CURE_ERR_INVALID_ARG;
  if (hq % hkv != 0) return CURE_ERR_INVALID_ARG;
  if (d != 64 && d != 128) return CURE_ERR_UNSUPPORTED;
  if (n_max > CURE_MAX_TREE_NODES) return CURE_ERR_UNSUPPORTED;
  if (batch == 0) return CURE_OK;
  if (n_max == 0) {                     // no sequence can have nodes
    if (tree_status) {
      hipLaunchKernelGGL(tree_status_ok, dim3((unsigned)((batch + 255) / 256)), dim3(256), 0,
                         as_stream(stream), tree_status, batch);
      return launch_status();
    }
    return CURE_OK;
  }
  if (!q || !k || !v || !o || !kv_off || !ctx_len || !n_nodes || !parent || !host_ctx_len ||
      !host_n_nodes)
    return CURE_ERR_INVALID_ARG;
  for (int b = 0; b < batch; ++b)
    if (host_ctx_len[b] < 0 || host_n_nodes[b] < 0 || host_n_nodes[b] > n_max)
      return CURE_ERR_INVALID_ARG;
  // The MFMA kernel takes the row maximum on raw scores (valid for scale > 0)
  // and addresses a sequence's K/V rows with 32-bit byte offsets.
  bool mfma = use_mfma(dtype, d, flags) && scale > 0.f && std::isfinite(scale);
  if (mfma) {
    int64_t t_max = 0;
    for (int b = 0; b < batch; ++b)
      t_max = std::max<int64_t>(t_max, (int64_t)host_ctx_len[b] + host_n_nodes[b]);
    if ((t_max + kTile) * hkv * d * 2 >= (int64_t(1) << 31)) mfma = false;
  }
  const Plan p = make_plan(batch, hq, hkv, d, n_max, host_ctx_len, host_n_nodes, kv_split, mfma);
  if (p.max_splits == 0) {              // no sequence has tree nodes
    if (tree_status) {
      hipLaunchKernelGGL(tree_status_ok, dim3((unsigned)((batch + 255) / 256)), dim3(256), 0,
                         as_stream(stream), tree_status, batch);
      return launch_status();
    }
    return CURE_OK;
  }
  const size_t need = plan_workspace(p, batch, hq, d, n_max);
  if (need > 0 && (!workspace || workspace_bytes < need)) return CURE_ERR_WORKSPACE;
  if ((size_t)p.row_blocks * hkv > 65535 || batch > 65535) return CURE_ERR_UNSUPPORTED;

  Args a{};
  a.q = q;
  a.k = k;
  a.v = v;
  a.o = o;
  a.lse = lse;
  a.out_bf16 = out_dtype == CURE_BF16;
  a.hq = hq;
  a.hkv = hkv;
  a.group = hq / hkv;
  a.n_max = n_max;
  a.scale_log2 = scale * kLog2e;
  a.kv_off = kv_off;
  a.ctx_len = ctx_len;
  a.n_nodes = n_nodes;
  a.parent = parent;
  a.tps = p.tps;
  a.max_splits = p.max_splits;
  a.rows_per_wg = p.rows_per_wg;
  a.tree_status = tree_status;
  if (need > 0) {
    const size_t parts = (size_t)batch * hq * n_max * p.max_splits;
    a.part_o = reinterpret_cast<float*>(workspace);
    a.part_lse = reinterpret_cast<float*>(reinterpret_cast<char*>(workspace) +
                                          align_up(parts * d * sizeof(float), 256));
  }
  if (mfma) {
    // The MFMA kernel reads q, k and v as 16-byte vectors.
    const uintptr_t mis = reinterpret_cast<uintptr_t>(q) | reinterpret_cast<uintptr_t>(k) |
                          reinterpret_cast<uintptr_t>(v);
    if (mis % 16 != 0) return CURE_ERR_INVALID_ARG;
    if (a.out_bf16 ? reinterpret_cast<uintptr_t>(o) % 8 : reinterpret_cast<uintptr_t>(o) % 16)
      return CURE_ERR_INVALID_ARG;
  }
  // Split partials are written and read as 16-byte vectors.
  if (need > 0 && reinterpret_cast<uintptr_t>(workspace) % 16 != 0) return CURE_ERR_INVALID_ARG;

  hipStream_t st = as_stream(stream);
  // KV heads (and row blocks) vary fastest: consecutive workgroups, which the
  // dispatcher spreads over the XCDs and starts together, read the heads of
  // the same token range, so concurrent reads cover whole cache rows.
  const dim3 grid(hkv * p.row_blocks, p.max_splits, batch);
  if (p.rows48) {
    hipLaunchKernelGGL((tree_attn_rg<128, kRg3Waves, 3, 2, 4, 2, 2>), grid, dim3(64 * kRg3Waves), 0,
                       st, a);
  } else if (p.rows16) {
    if (d == 128) {
      if (p.nw == 8) hipLaunchKernelGGL((tree_attn_m16<128, 8>), grid, dim3(512), 0, st, a);
      else hipLaunchKernelGGL((tree_attn_m16<128, 16>), grid, dim3(1024), 0, st, a);
    } else {
      hipLaunchKernelGGL((tree_attn_m16<64, 8>), grid, dim3(512), 0, st, a);
    }
  } else if (mfma) {
    hipLaunchKernelGGL((tree_attn_mfma<64, 8, kStages>), grid, dim3(512), 0, st, a);
  } else {
    if (dtype == CURE_BF16) {
      if (d == 128) hipLaunchKernelGGL((tree_attn_valu<uint16_t, 128>), grid, dim3(256), 0, st, a);
      else hipLaunchKernelGGL((tree_attn_valu<uint16_t, 64>), grid, dim3(256), 0, st, a);
    } else {
      if (d == 128) hipLaunchKernelGGL((tree_attn_valu<float, 128>), grid, dim3(256), 0, st, a);
      else hipLaunchKernelGGL((tree_attn_valu<float, 64>), grid, dim3(256), 0, st, a);
    }
  }
  if (hipGetLastError() != hipSuccess) return CURE_ERR_HIP;
  if (p.max_splits > 1) {
    const dim3 mgrid((unsigned)((hq + 3) / 4), (unsigned)n_max, (unsigned)batch);
    const int per_load = 256 / d;                       // splits per merge load
    const int nb = p.max_splits <= 2 * per_load ? 2 : p.max_splits <= 4 * per_load ? 4 : 8;
    const bool own = !p.uniform_splits;
#define CURE_MERGE(DD, NN)                                                                   \
    do {                                                                                     \
      if (own) hipLaunchKernelGGL((attn_merge<DD, NN, true>), mgrid, dim3(256), 0, st, a);   \
      else hipLaunchKernelGGL((attn_merge<DD, NN, false>), mgrid, dim3(256), 0, st, a);      \
    } while (0)
    if (d == 128) {
      if (nb == 2) CURE_MERGE(128, 2);
      else if (nb == 4) CURE_MERGE(128, 4);
      else CURE_MERGE(128, 8);
    } else {
      if (nb == 2) CURE_MERGE(64, 2);
      else if (nb == 4) CURE_MERGE(64, 4);
      else CURE_MERGE(64, 8);
    }
#undef CURE_MERGE
  }
  return launch_status();
}
