/*
 * libcure -- MI355X (gfx950) verify-and-repair hot path of CURE
 * (local uncertainty repair for block-parallel speculative decoding).
 *
 * Stream-ordered entry points cover one decoding iteration's data-parallel
 * work on the device:
 *
 *   cure_margins    top-1/top-2 margin and log-sum-exp per logits row, plus the
 *                   Uncertainty Focal Point (UFP) selection      (Sec. 3.3, Eq. 2)
 *   cure_tree_attn  tree-masked verification attention over the KV cache and
 *                   each node's own tree ancestors           (Sec. 3.2, 3.4, 3.5)
 *   cure_accept     accepted prefix per path and the best path     (Eq. 1, Eq. 4)
 *   cure_margins_accept  cure_margins over a tree's node logits followed by
 *                   cure_accept on their argmaxes, in the margin pass's launches
 *   cure_repair_tree  the budget-aware repair tree: ranked alternatives at the
 *                   UFPs, the Eq. 3 branch budget and the parent/token arrays
 *                                                       (Sec. 3.3, 3.4, Alg. 1)
 *   cure_commit     the winning path committed: its cache rows moved after the
 *                   context in every layer, the emitted tokens, the new context
 *                   length and the draft-cache replay start   (Sec. 3.5, Alg. 1)
 *   cure_margins_noalloc  cure_margins for callers that cannot allocate: its
 *                   scratch is a fixed array inside the library
 *   cure_read_ceiling  not a step of the method: a plain streaming read, the
 *                   practical HBM read rate the other calls are compared with
 *
 * Conventions shared by every entry point
 *  - All array arguments are DEVICE pointers (memory the caller allocated with
 *    hipMalloc or equivalent), except those whose name starts with host_.
 *    The library allocates no device memory and keeps no state beyond a cached
 *    device-property query (and the static scratch array of
 *    cure_margins_noalloc, part of its code object); the caller owns every
 *    buffer.
 *  - stream is a hipStream_t passed as void* (NULL = the legacy default stream).
 *    Calls only enqueue work: they return before the work runs, and the outputs
 *    are valid once the stream reaches that point.
 *  - The return value reports errors the host can see: invalid arguments,
 *    unsupported shapes, a too-small workspace and HIP launch failures. Errors
 *    in device data (a malformed tree) are reported through device status words.
 *    No C++ exception crosses this interface.
 *  - Workspaces: a call that takes a workspace needs at least the size its
 *    *_workspace_size function returns for the same arguments (0 means none is
 *    needed and the pointer may be NULL). A workspace holds scratch data only
 *    while the call's kernels run: it needs no initialisation and may be reused
 *    by any later call on the same stream. Two calls whose work may overlap on
 *    the GPU must not share a workspace.
 *  - bf16 values are raw IEEE bfloat16 bit patterns (uint16 storage).
 */
#ifndef CURE_H
#define CURE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum cure_status {
  CURE_OK = 0,
  CURE_ERR_INVALID_ARG = 1,   /* null pointer, negative size, inconsistent shapes   */
  CURE_ERR_UNSUPPORTED = 2,   /* shape outside what the kernels implement            */
  CURE_ERR_BAD_TREE = 3,      /* device status word only: parent[n] not in [-1, n-1] */
  CURE_ERR_HIP = 4,           /* a HIP runtime call or kernel launch failed          */
  CURE_ERR_WORKSPACE = 5      /* workspace null or smaller than required             */
} cure_status;

typedef enum cure_dtype { CURE_F32 = 0, CURE_BF16 = 1 } cure_dtype;

/* Flags for cure_tree_attn. */
#define CURE_ATTN_FORCE_VALU 1u   /* use the vector-ALU kernel even where MFMA applies */

#define CURE_MAX_TREE_NODES 256   /* largest tree (nodes per sequence) supported       */

/* Human-readable name of a status code (static storage, never NULL). */
const char* cure_status_string(int status);

/* Library version as 10000*major + 100*minor + patch. */
int cure_version(void);

/* ------------------------------------------------------------------------- */
/* Margin pass and UFP gate -- Sec. 3.3 Eq. (2) and Algorithm 1.
 *
 * For every row r of logits (batch*rows rows of vocab entries; row r of
 * sequence b starts at element (b*rows + r)*ld):
 *   top1_idx/top1_val  the largest entry,
 *   top2_idx/top2_val  the next entry in the order (value descending, index
 *                      ascending) -- ties go to the lowest index, so a maximum
 *                      that occurs twice gives top2 = its second index,
 *   margin             top1_val - top2_val, computed in float32,
 *   lse                log(sum_v exp(x_v)), natural log, float32.
 * Entries are widened exactly to float32; values must be finite or -inf.
 *
 * UFP gate (skipped when ufp_pos and ufp_cnt are both NULL): over the first
 * chain_len rows of each sequence, the positions with margin < tau (strict),
 * ordered by (margin ascending, position ascending), at most
 * floor(repair_budget / branch_depth) of them, so that branches of branch_depth
 * nodes never exceed the repair budget. ufp_pos is [batch][chain_len] int32,
 * filled with the selected positions in that order and padded with -1;
 * ufp_cnt is [batch] int32.
 *
 * Layout: logits row-major, ld >= vocab elements between rows; every per-row
 * output has batch*rows entries. Requires vocab >= 2, 0 <= chain_len <= rows
 * (chain_len >= 1 when the gate runs), branch_depth >= 1, repair_budget >= 0.
 * workspace: cure_margins_workspace_size(batch, rows, vocab) bytes.
 */
size_t cure_margins_workspace_size(int32_t batch, int32_t rows, int32_t vocab);

cure_status cure_margins(const void* logits, int32_t dtype, int32_t batch, int32_t rows,
                         int32_t vocab, int64_t ld,
                         float* top1_val, int32_t* top1_idx, float* top2_val,
                         int32_t* top2_idx, float* lse, float* margin,
                         int32_t chain_len, float tau, int32_t repair_budget,
                         int32_t branch_depth, int32_t* ufp_pos, int32_t* ufp_cnt,
                         void* workspace, size_t workspace_bytes, void* stream);

/* Margin pass with the acceptance walk as its epilogue -- Sec. 3.3 Eq. (2),
 * Algorithm 1, Sec. 3.1 Eq. (1), Sec. 3.5 Eq. (4).
 *
 * For logits whose rows are the nodes of each sequence's candidate tree (row
 * n of sequence b = node n, so rows is the tree arrays' n_max): exactly
 * cure_margins(...) followed by cure_accept(parent, token, top1_idx, root_tgt,
 * n_nodes, chain_len, batch, rows, ...), with every output of both, bit for
 * bit. The walk runs in the workgroup that finishes each sequence's rows, so
 * the pair costs the margin pass's launches only (no separate acceptance
 * launch). chain_len serves the UFP gate (when ufp_pos/ufp_cnt are given) and
 * the walk's resync flag.
 *   parent, token  [batch][rows] int32;  root_tgt, n_nodes  [batch] int32
 *   acc_len, best, bonus, resync  [batch] int32;  path  [batch][rows] int32
 * Requires everything cure_margins requires, chain_len >= 0 and rows <= 256
 * (CURE_ERR_UNSUPPORTED otherwise). workspace: cure_margins_workspace_size(
 * batch, rows, vocab) bytes.
 */
cure_status cure_margins_accept(const void* logits, int32_t dtype, int32_t batch, int32_t rows,
                                int32_t vocab, int64_t ld,
                                float* top1_val, int32_t* top1_idx, float* top2_val,
                                int32_t* top2_idx, float* lse, float* margin,
                                int32_t chain_len, float tau, int32_t repair_budget,
                                int32_t branch_depth, int32_t* ufp_pos, int32_t* ufp_cnt,
                                const int32_t* parent, const int32_t* token,
                                const int32_t* root_tgt, const int32_t* n_nodes,
                                int32_t* acc_len, int32_t* path, int32_t* best,
                                int32_t* bonus, int32_t* resync,
                                void* workspace, size_t workspace_bytes, void* stream);

/* Allocation-free margin pass, for callers that cannot allocate device memory
 * (code under HIP stream capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same pass, outputs and UFP gate as cure_margins, with no
 * workspace argument. Its scratch (the chunk results of rows split across
 * workgroups, 32 bytes per row and chunk) lives in a fixed device array of
 * cure_margins_noalloc_scratch_bytes() bytes (256 KiB) inside the library,
 * one per GPU the library runs on, held until the process ends. The call
 * itself allocates nothing; its first use on a device looks up that device's
 * copy of the array (hipGetSymbolAddress).
 * Returns CURE_ERR_UNSUPPORTED when the call would need more scratch than the
 * array holds (never on a 256-CU MI355X, whose plans need at most 32 KiB),
 * CURE_ERR_HIP when the array cannot be found on the current device, else as
 * cure_margins. Every call on one GPU shares that GPU's array and leaves its
 * contents behind: calls whose work may overlap on the GPU (different streams
 * without ordering between them) race and must not be issued. */
size_t cure_margins_noalloc_scratch_bytes(void);

cure_status cure_margins_noalloc(const void* logits, int32_t dtype, int32_t batch,
                                 int32_t rows, int32_t vocab, int64_t ld,
                                 float* top1_val, int32_t* top1_idx, float* top2_val,
                                 int32_t* top2_idx, float* lse, float* margin,
                                 int32_t chain_len, float tau, int32_t repair_budget,
                                 int32_t branch_depth, int32_t* ufp_pos, int32_t* ufp_cnt,
                                 void* stream);

/* ------------------------------------------------------------------------- */
/* Tree-attention verification -- Sec. 3.2 (phase 3), Sec. 3.4, Sec. 3.5.
 *
 * One forward attention layer of the target over every node of each
 * sequence's candidate tree. Node n of sequence b, query head h (key/value head
 * h / (hq/hkv)) attends to
 *   - the ctx_len[b] cached context rows, and
 *   - the tree rows of the nodes on its own root path, itself included,
 * with scores scale * <q, k>, natural-base softmax:
 *   o[b][n][h]   = sum_j softmax_j * v_j            (normalised)
 *   lse[b][n][h] = log sum_j exp(scale * <q, k_j>)
 *
 * Layout:
 *   q       [batch][n_max][hq][d]          dtype
 *   k, v    token rows of [hkv][d]         dtype; sequence b owns rows
 *           kv_off[b] .. kv_off[b] + ctx_len[b] + n_nodes[b] - 1: its context,
 *           then its tree nodes in node order
 *   o       [batch][n_max][hq][d]          out_dtype (CURE_F32 or CURE_BF16)
 *   lse     [batch][n_max][hq]             float32 (may be NULL)
 *   parent  [batch][n_max]                 int32, parent[n] in [-1, n-1]: the
 *           tree in topological order, -1 = attached to the context
 *   kv_off  [batch] int64, ctx_len/n_nodes [batch] int32 (device)
 *   host_ctx_len/host_n_nodes: host copies of ctx_len/n_nodes, used only to
 *           plan the split of each context across workgroups.
 * Rows n >= n_nodes[b] of o and lse are not written.
 * tree_status [batch] int32 (may be NULL): CURE_OK (also for a sequence with
 * no nodes), or CURE_ERR_BAD_TREE when sequence b's parent array is malformed
 * (that sequence's o/lse are then unspecified).
 * Supports d in {64, 128}, hq % hkv == 0, 0 <= n_nodes[b] <= min(n_max, 256)
 * (a sequence with no nodes is skipped).
 * kv_split: 0 = automatic, else the number of context splits per sequence.
 * flags: CURE_ATTN_FORCE_VALU or 0.
 * workspace: cure_tree_attn_workspace_size(...) bytes for the same arguments.
 *   It holds each context split's fp32 partial rows and their log-sum-exps;
 *   the splits are combined by a log-sum-exp merge.
 * Alignment (else CURE_ERR_INVALID_ARG): workspace 16 bytes; on the bf16
 * matrix-core path (bf16 inputs, d 64 or 128, scale > 0, no FORCE_VALU) also
 * q, k, v 16 bytes and o 8 bytes (bf16 out) or 16 bytes (fp32 out).
 */
size_t cure_tree_attn_workspace_size(int32_t batch, int32_t hq, int32_t hkv, int32_t d,
                                     int32_t n_max, const int32_t* host_ctx_len,
                                     const int32_t* host_n_nodes, int32_t kv_split);

cure_status cure_tree_attn(const void* q, const void* k, const void* v, void* o, float* lse,
                           int32_t dtype, int32_t out_dtype, int32_t batch, int32_t hq,
                           int32_t hkv, int32_t d, float scale, const int64_t* kv_off,
                           const int32_t* ctx_len, const int32_t* n_nodes,
                           const int32_t* parent, int32_t n_max,
                           const int32_t* host_ctx_len, const int32_t* host_n_nodes,
                           int32_t kv_split, uint32_t flags, int32_t* tree_status,
                           void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------- */
/* Acceptance walk -- Sec. 3.1 Eq. (1), Sec. 3.5 Eq. (4), greedy decoding.
 *
 * Per sequence b with n_nodes[b] nodes (all arrays [batch][n_max] int32 unless
 * noted):
 *   node n is accepted when its token equals the target's argmax before it --
 *   root_tgt[b] for parent[n] == -1, else tgt[parent[n]] -- and its parent is
 *   accepted. The winner is the accepted node of greatest depth, lowest index
 *   on ties (so branch 0, numbered first, wins ties).
 *   acc_len [batch]  depth(winner)+1, or 0 when nothing is accepted
 *   best    [batch]  the winner, or -1
 *   path    [batch][n_max] root->winner node indices, padded with -1
 *   bonus   [batch]  tgt[winner], or root_tgt[b] when nothing is accepted
 *   resync  [batch]  1 when the winning path holds a node >= chain_len (a repair
 *                    node, so the draft cache must be resynchronised), else 0;
 *                    -1 together with acc_len = -1 when the parent array is
 *                    malformed.
 * tgt is typically cure_margins' top1_idx over the target's node logits.
 * Supports 0 <= n_nodes[b] <= min(n_max, 256); with no nodes, acc_len = 0
 * and bonus = root_tgt.
 */
cure_status cure_accept(const int32_t* parent, const int32_t* token, const int32_t* tgt,
                        const int32_t* root_tgt, const int32_t* n_nodes, int32_t chain_len,
                        int32_t batch, int32_t n_max, int32_t* acc_len, int32_t* path,
                        int32_t* best, int32_t* bonus, int32_t* resync, void* stream);

/* ------------------------------------------------------------------------- */
/* Repair-tree construction -- Sec. 3.3 Eq. (3), Sec. 3.4, Algorithm 1.
 *
 * Builds each sequence's candidate tree from its draft block (branch 0) and
 * the UFPs that cure_margins selected. For UFP slot s (in the given,
 * ascending-margin order) at block position u = ufp_pos[b][s]:
 *   ranked      the draft row's entries in the order (value descending, index
 *               ascending), read from logits row u of sequence b;
 *   alternatives the ranked tokens other than chain_tok[b][u], best first;
 *   b_s         Eq. (3) on margin m = margin[b*rows + u]:
 *                 t = b_min + clip(1 - m / margin_scale, 0, 1) * (b_max - b_min)
 *                 b_s = clip(round_half_even(t), b_min, b_max)
 *               in float32, every operation rounded once; a NaN margin counts
 *               as certain (b_s = b_min);
 *   granted     min(b_s, remaining / branch_depth): whole branches only,
 *               remaining starting at repair_budget, slots taken in order.
 * Branch r of slot s is a chain of branch_depth nodes: its root carries
 * alternative r and hangs off chain node u - 1 (-1, the context, when u = 0);
 * node j > 0 carries suffix[b][u][r][j-1] (the token the drafter proposed
 * after that substitution) or -1 when suffix is NULL, and hangs off node j - 1.
 *
 * Node numbering (the tree is in topological order): nodes 0 .. chain_len-1 are
 * the chain (parent[i] = i - 1, token = chain_tok); then the branches, slot by
 * slot and within a slot by alternative rank, each branch's nodes consecutive.
 *
 * Layout:
 *   logits     [batch][rows][ld] dtype (the draft block's rows; the first
 *              chain_len rows of each sequence are the chain positions)
 *   margin     [batch][rows] float32, as cure_margins wrote it
 *   ufp_pos    [batch][chain_len] int32, ufp_cnt [batch] int32, as cure_margins
 *              wrote them (the slots used are the first min(ufp_cnt,
 *              repair_budget / branch_depth), cut at the first position
 *              outside [0, chain_len))
 *   chain_tok  [batch][chain_len] int32, the draft block
 *   suffix     [batch][chain_len][b_max][branch_depth-1] int32, or NULL
 *   parent, token  [batch][n_max] int32 outputs; entries at or past
 *              n_nodes[b] are not written
 *   n_nodes    [batch] int32 output: chain_len + branch_depth * (branches)
 *   branch_cnt [batch][chain_len] int32 output (may be NULL): branches granted
 *              per slot, 0 for unused slots
 * Requires 1 <= chain_len <= min(rows, 1024), branch_depth >= 1,
 * repair_budget >= 0, 0 <= b_min <= b_max <= 7, b_max >= 1,
 * vocab >= b_max + 1, vocab <= 524288, ld >= vocab, margin_scale > 0 and
 * finite, n_max >= chain_len + repair_budget (so every tree fits).
 * workspace: cure_repair_tree_workspace_size(...) bytes for the same arguments.
 */
size_t cure_repair_tree_workspace_size(int32_t batch, int32_t chain_len, int32_t vocab,
                                       int32_t repair_budget, int32_t branch_depth);

cure_status cure_repair_tree(const void* logits, int32_t dtype, int32_t batch, int32_t rows,
                             int32_t vocab, int64_t ld, const float* margin,
                             const int32_t* ufp_pos, const int32_t* ufp_cnt,
                             const int32_t* chain_tok, int32_t chain_len,
                             int32_t repair_budget, int32_t branch_depth, float margin_scale,
                             int32_t b_min, int32_t b_max, const int32_t* suffix,
                             int32_t n_max, int32_t* parent, int32_t* token, int32_t* n_nodes,
                             int32_t* branch_cnt, void* workspace, size_t workspace_bytes,
                             void* stream);

/* ------------------------------------------------------------------------- */
/* Committing the winning path -- Sec. 3.5 (cache resynchronisation), Alg. 1.
 *
 * The accepted tokens become context for the next step. For each sequence b
 * with a = acc_len[b] accepted nodes and winning path path[b][0 .. a-1] (node
 * indices, root first, as cure_accept writes them):
 *   cache       in every layer, cache row kv_off[b] + ctx_len[b] + j takes
 *               the contents of row kv_off[b] + ctx_len[b] + path[b][j], for
 *               j < a (tree node n's rows sit at ctx_len + n, as for
 *               cure_tree_attn), in K and in V. The move is in place; rows from
 *               ctx_len + a on keep whatever they held.
 *   new_ctx_len [batch] ctx_len[b] + a
 *   emit        [batch][n_max + 1] the a accepted tokens token[b][path[b][j]],
 *               then bonus[b], padded with -1
 *   emit_cnt    [batch] a + 1
 *   replay_start [batch] depth of the path's first node numbered >= chain_len
 *               (a repair node), else a: the emitted tokens from there to a-1
 *               are the ones to replay into the draft model's cache
 *   commit_status [batch] CURE_OK, or CURE_ERR_BAD_TREE when the sequence is
 *               not committable: acc_len < 0 (cure_accept's mark of a malformed
 *               tree), acc_len > n_nodes, n_nodes outside [0, n_max], a
 *               negative ctx_len or kv_off, or a path entry outside
 *               [0, n_nodes) or not above its predecessor. Such a sequence's
 *               cache is left untouched, new_ctx_len = ctx_len, emit_cnt = 0,
 *               replay_start = 0 and its emit row is all -1.
 *
 * Layout:
 *   k, v       n_layers caches; layer l's starts at element l * layer_stride
 *              of k and of v and holds token rows of [hkv][d] dtype elements
 *              (layer_stride is ignored when n_layers <= 1)
 *   kv_off [batch] int64, ctx_len, n_nodes, acc_len, bonus [batch] int32,
 *   path, token [batch][n_max] int32 -- all device memory
 * Requires hkv * d * sizeof(dtype) to be a multiple of 16 bytes, n_max <= 256,
 * batch <= 65535. Outputs must not overlap the inputs (new_ctx_len may not be
 * ctx_len itself: other workgroups still read ctx_len while it is written).
 * Every cache row kv_off[b] .. kv_off[b] + ctx_len[b] + n_nodes[b] - 1 of
 * every layer must exist. No workspace.
 */
cure_status cure_commit(void* k, void* v, int32_t dtype, int32_t n_layers, int64_t layer_stride,
                        int32_t hkv, int32_t d, int32_t batch, const int64_t* kv_off,
                        const int32_t* ctx_len, const int32_t* n_nodes, const int32_t* path,
                        const int32_t* acc_len, const int32_t* token, const int32_t* bonus,
                        int32_t chain_len, int32_t n_max, int32_t* new_ctx_len, int32_t* emit,
                        int32_t* emit_cnt, int32_t* replay_start, int32_t* commit_status,
                        void* stream);

/* ------------------------------------------------------------------------- */
/* Read ceiling -- a measurement aid, not a step of the method.
 *
 * Streams `bytes` of device memory (a multiple of 16) the way the margin pass
 * streams its rows: one workgroup per 256 KB chunk, 16-byte non-temporal
 * loads. Writes the XOR of each chunk's 32-bit words to chunk_xor[i] (device,
 * cure_read_ceiling_chunks(bytes) entries), so the read is needed and can be
 * checked. Its time is the practical HBM read rate the hot path's bandwidth is
 * compared against.
 */
size_t cure_read_ceiling_chunks(size_t bytes);

cure_status cure_read_ceiling(const void* buf, size_t bytes, uint32_t* chunk_xor, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* CURE_H */
