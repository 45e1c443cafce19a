"""Oracle: candidate-tree encoding and tree-attention verification.

Test infrastructure only (see the package docstring).

Paper passages followed:

* Sec. 3.4: repair paths keep the original prefix and substitute the fragile
  token; paths sharing a prefix merge into shared parent nodes, so the
  candidate set is a tree rooted at the context. It is given here as a parent
  array in topological order: parent[n] in {-1, 0, ..., n-1}, where -1 attaches
  node n directly after the cached context.
* Sec. 3.2 (phase 3) and Sec. 3.5: one forward pass of the target evaluates
  every tree node at once with tree attention. A node may see the whole cached
  context and the tree nodes on its own root-to-node path (itself included),
  and nothing else.

Readings where the paper is silent:

* Scores are scale * <q, k> with the scale given by the caller (1/sqrt(D) in
  every workload), natural exp and log, output normalised by the softmax sum.
* The tree's own keys and values sit in the cache right after the context, in
  node order (rows ctx_len .. ctx_len + n_nodes - 1 of the sequence).
* Grouped-query attention: query head h reads key/value head h // (hq // hkv).
* Rotary position encoding happens before this step; q and k arrive rotated.
"""

import numpy as np

from .margins import as_float32


def ancestors(parent, n_nodes):
    """Ancestor sets and depths of a parent-array tree.

    Returns (anc, depth): anc[n] is the sorted list of nodes on the path from the
    tree root down to n, n included; depth[n] is len(anc[n]) - 1.
    Raises ValueError if some parent[n] is outside [-1, n-1].
    """
    parent = [int(p) for p in parent[:n_nodes]]
    for n, p in enumerate(parent):
        if p < -1 or p >= n:
            raise ValueError("parent[%d] = %d is not in [-1, %d]" % (n, p, n - 1))
    anc, depth = [], []
    for n in range(n_nodes):
        path, j = [], n
        while j >= 0:
            path.append(j)
            j = parent[j]
        anc.append(sorted(path))
        depth.append(len(path) - 1)
    return anc, depth


def tree_attention(q, k, v, dtype, kv_off, ctx_len, n_nodes, parent, hq, hkv, scale,
                   sample=None):
    """Tree-masked verification attention for a batch of sequences.

    q:      [batch, n_max, hq, d]    query of every tree node
    k, v:   [rows, hkv, d]           token-major cache; sequence b occupies rows
                                     kv_off[b] .. kv_off[b] + ctx_len[b] + n_nodes[b] - 1
    parent: [batch, n_max]           parent array of each sequence's tree
    dtype:  'f32' or 'bf16' (raw uint16 bits) for q, k and v

    sample: optional collection of (b, n) pairs; when given, only those nodes
            are computed (for spot checks of very large workloads).

    Returns (o, lse): o [batch, n_max, hq, d] float64 and lse [batch, n_max, hq]
    float64; entries for nodes n >= n_nodes[b], or outside the sample, are zero.
    """
    wanted = None if sample is None else {(int(b), int(n)) for b, n in sample}
    qf = as_float32(q, dtype).astype(np.float64)
    kf = as_float32(k, dtype)
    vf = as_float32(v, dtype)
    batch, n_max, hq_, d = qf.shape
    if hq_ != hq or hq % hkv != 0:
        raise ValueError("bad head counts")
    group = hq // hkv
    o = np.zeros((batch, n_max, hq, d), np.float64)
    lse = np.zeros((batch, n_max, hq), np.float64)
    for b in range(batch):
        if wanted is not None and not any(wb == b for wb, _ in wanted):
            continue
        L, N, off = int(ctx_len[b]), int(n_nodes[b]), int(kv_off[b])
        anc, _ = ancestors(parent[b], N)
        for g in range(hkv):
            heads = list(range(g * group, (g + 1) * group))
            # Visible keys of node n: every context row, then the tree rows of
            # the nodes on n's root path (rows L + j for j in anc[n]).
            k_ctx = kf[off: off + L, g, :].astype(np.float64)          # [L, d]
            v_ctx = vf[off: off + L, g, :].astype(np.float64)
            k_tree = kf[off + L: off + L + N, g, :].astype(np.float64)  # [N, d]
            v_tree = vf[off + L: off + L + N, g, :].astype(np.float64)
            for n in range(N):
                if wanted is not None and (b, n) not in wanted:
                    continue
                k_vis = np.concatenate([k_ctx, k_tree[anc[n]]], axis=0)   # [|visible|, d]
                v_vis = np.concatenate([v_ctx, v_tree[anc[n]]], axis=0)
                for h in heads:
                    s = scale * (k_vis @ qf[b, n, h])                      # [|visible|]
                    m = np.max(s)
                    p = np.exp(s - m)
                    den = np.sum(p)
                    o[b, n, h] = (p @ v_vis) / den
                    lse[b, n, h] = m + np.log(den)
    return o, lse
