"""Pins for the tree-attention oracle (Sec. 3.2 phase 3, Sec. 3.4, Sec. 3.5).

The oracle builds each node's visible set by walking parent pointers and runs a
two-pass softmax per (node, head). These tests compare it with torch's
scaled_dot_product_attention on the CPU, fed a mask built by a different
construction (a boolean transitive closure, or a plain causal triangle), and
with closed forms (zero queries, single-node trees).
"""

import json
import math
import os

import numpy as np
import pytest
import scipy.special
import torch
import torch.nn.functional as F

import oracle
from synth import make_workload

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def closure_mask(parent, n):
    """Visibility among tree nodes via transitive closure of the parent relation.

    A[i, j] = 1 when j is i's parent; reach = I + A + A^2 + ... by repeated
    boolean squaring of (I + A). No parent-pointer walking is involved.
    """
    a = torch.zeros(n, n, dtype=torch.bool)
    for i in range(n):
        if parent[i] >= 0:
            a[i, parent[i]] = True
    reach = a | torch.eye(n, dtype=torch.bool)
    for _ in range(max(1, math.ceil(math.log2(max(n, 2))) + 1)):
        reach = reach | ((reach.float() @ reach.float()) > 0)
    return reach


def sdpa_reference(w, b):
    """torch SDPA (float64, CPU) over the context plus the tree, masked by closure."""
    L, N, off = int(w.ctx_len[b]), int(w.n_nodes[b]), int(w.kv_off[b])
    q = torch.from_numpy(oracle.as_float32(w.q[b, :N], w.dtype).astype(np.float64))
    k = torch.from_numpy(oracle.as_float32(w.k[off:off + L + N], w.dtype).astype(np.float64))
    v = torch.from_numpy(oracle.as_float32(w.v[off:off + L + N], w.dtype).astype(np.float64))
    group = w.hq // w.hkv
    qh = q.permute(1, 0, 2)                                        # [hq, N, d]
    kh = k.permute(1, 0, 2).repeat_interleave(group, dim=0)        # [hq, L+N, d]
    vh = v.permute(1, 0, 2).repeat_interleave(group, dim=0)
    mask = torch.ones(N, L + N, dtype=torch.bool)
    mask[:, L:] = closure_mask(w.parent[b], N)
    o = F.scaled_dot_product_attention(qh, kh, vh, attn_mask=mask, scale=w.scale)
    s = (qh @ kh.transpose(1, 2)) * w.scale
    s = s.masked_fill(~mask, float("-inf"))
    lse = torch.logsumexp(s, dim=-1)                               # [hq, N]
    return o.permute(1, 0, 2).numpy(), lse.permute(1, 0).numpy()


def run_oracle(w):
    return oracle.tree_attention(w.q, w.k, w.v, w.dtype, w.kv_off, w.ctx_len, w.n_nodes,
                                 w.parent, w.hq, w.hkv, w.scale)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_random_trees_against_sdpa_with_closure_mask(dtype):
    w = make_workload("t", dtype=dtype, batch=3, hq=8, hkv=2, d=32, vocab=64,
                      ctx_lens=[5, 17, 40], chain_len=6, n_ufp=3, branch_depth=2, seed=21)
    o, lse = run_oracle(w)
    for b in range(w.batch):
        ro, rl = sdpa_reference(w, b)
        N = int(w.n_nodes[b])
        assert np.allclose(o[b, :N], ro, atol=1e-12, rtol=0)
        assert np.allclose(lse[b, :N], rl, atol=1e-12, rtol=0)


def test_arbitrary_parent_arrays_against_sdpa():
    rng = np.random.default_rng(7)
    w = make_workload("t", dtype="f32", batch=2, hq=4, hkv=4, d=16, vocab=64,
                      ctx_lens=[3, 9], chain_len=8, n_ufp=2, branch_depth=2, seed=3)
    for b in range(w.batch):      # replace the trees by random topologically ordered ones
        N = int(w.n_nodes[b])
        w.parent[b, :N] = [int(rng.integers(-1, n)) if n else -1 for n in range(N)]
    o, lse = run_oracle(w)
    for b in range(w.batch):
        ro, rl = sdpa_reference(w, b)
        N = int(w.n_nodes[b])
        assert np.allclose(o[b, :N], ro, atol=1e-12) and np.allclose(lse[b, :N], rl, atol=1e-12)


def test_pure_chain_is_causal_attention():
    w = make_workload("t", dtype="f32", batch=1, hq=4, hkv=2, d=32, vocab=64,
                      ctx_lens=[23], chain_len=10, n_ufp=0, branch_depth=1, seed=5)
    o, lse = run_oracle(w)
    L, N = 23, 10
    q = torch.from_numpy(w.q[0, :N].astype(np.float64)).permute(1, 0, 2)
    k = torch.from_numpy(w.k[:L + N].astype(np.float64)).permute(1, 0, 2).repeat_interleave(2, 0)
    v = torch.from_numpy(w.v[:L + N].astype(np.float64)).permute(1, 0, 2).repeat_interleave(2, 0)
    # Query i sits at position L + i; a causal (lower-right aligned) triangle.
    mask = torch.ones(L + N, L + N, dtype=torch.bool).tril()[L:]
    ref = F.scaled_dot_product_attention(q, k, v, attn_mask=mask, scale=w.scale)
    assert np.allclose(o[0, :N], ref.permute(1, 0, 2).numpy(), atol=1e-12)


def test_each_root_to_leaf_path_is_independent_causal_attention():
    w = make_workload("t", dtype="f32", batch=1, hq=2, hkv=1, d=16, vocab=64,
                      ctx_lens=[12], chain_len=6, n_ufp=3, branch_depth=3, seed=9)
    o, lse = run_oracle(w)
    L, N = 12, int(w.n_nodes[0])
    par = list(w.parent[0, :N])
    leaves = [n for n in range(N) if n not in par]
    assert len(leaves) >= 3
    for leaf in leaves:
        path, j = [], leaf
        while j >= 0:
            path.append(j)
            j = par[j]
        path.reverse()
        rows = list(range(L)) + [L + j for j in path]
        q = torch.from_numpy(w.q[0, path].astype(np.float64)).permute(1, 0, 2)
        k = torch.from_numpy(w.k[rows].astype(np.float64)).permute(1, 0, 2).repeat_interleave(2, 0)
        v = torch.from_numpy(w.v[rows].astype(np.float64)).permute(1, 0, 2).repeat_interleave(2, 0)
        mask = torch.ones(len(rows), len(rows), dtype=torch.bool).tril()[L:]
        ref = F.scaled_dot_product_attention(q, k, v, attn_mask=mask, scale=w.scale)
        assert np.allclose(o[0, path], ref.permute(1, 0, 2).numpy(), atol=1e-12)


def test_zero_query_gives_mean_of_visible_values():
    w = make_workload("t", dtype="f32", batch=2, hq=4, hkv=2, d=8, vocab=64,
                      ctx_lens=[7, 0], chain_len=5, n_ufp=2, branch_depth=2, seed=13)
    w.q[...] = 0.0
    o, lse = run_oracle(w)
    for b in range(w.batch):
        L, N, off = int(w.ctx_len[b]), int(w.n_nodes[b]), int(w.kv_off[b])
        for n in range(N):
            depth = int(w.depth[b, n])
            # |visible| = L + depth + 1, and O is the plain mean of those rows.
            anc, j = [], n
            while j >= 0:
                anc.append(j)
                j = int(w.parent[b, j])
            rows = list(range(off, off + L)) + [off + L + a for a in anc]
            assert len(rows) == L + depth + 1
            for h in range(w.hq):
                mean = w.v[rows, h // 2].astype(np.float64).mean(axis=0)
                assert np.allclose(o[b, n, h], mean, atol=1e-12)
                assert lse[b, n, h] == pytest.approx(math.log(L + depth + 1), abs=1e-12)


def test_single_node_is_decode_attention():
    w = make_workload("t", dtype="f32", batch=1, hq=3, hkv=1, d=8, vocab=64,
                      ctx_lens=[30], chain_len=1, n_ufp=0, branch_depth=1, seed=17)
    o, lse = run_oracle(w)
    k = w.k[:31, 0].astype(np.float64)
    v = w.v[:31, 0].astype(np.float64)
    for h in range(3):
        s = w.scale * (k @ w.q[0, 0, h].astype(np.float64))
        assert np.allclose(o[0, 0, h], scipy.special.softmax(s) @ v, atol=1e-12)
        assert lse[0, 0, h] == pytest.approx(scipy.special.logsumexp(s), abs=1e-12)


def test_packed_sequences_match_separate_calls():
    w = make_workload("t", dtype="f32", batch=3, hq=4, hkv=2, d=16, vocab=64,
                      ctx_lens=[4, 11, 6], chain_len=5, n_ufp=1, branch_depth=3, seed=19)
    o, lse = run_oracle(w)
    for b in range(w.batch):
        off, rows = int(w.kv_off[b]), int(w.ctx_len[b] + w.n_nodes[b])
        ob, lb = oracle.tree_attention(w.q[b:b + 1], w.k[off:off + rows], w.v[off:off + rows],
                                       "f32", [0], w.ctx_len[b:b + 1], w.n_nodes[b:b + 1],
                                       w.parent[b:b + 1], w.hq, w.hkv, w.scale)
        assert np.array_equal(o[b], ob[0]) and np.array_equal(lse[b], lb[0])


def test_sample_option_computes_only_requested_nodes():
    w = make_workload("t", dtype="f32", batch=2, hq=2, hkv=1, d=8, vocab=64,
                      ctx_lens=[5, 6], chain_len=4, n_ufp=1, branch_depth=2, seed=23)
    full_o, full_l = run_oracle(w)
    o, l = oracle.tree_attention(w.q, w.k, w.v, "f32", w.kv_off, w.ctx_len, w.n_nodes,
                                 w.parent, w.hq, w.hkv, w.scale, sample=[(1, 3), (0, 0)])
    assert np.array_equal(o[1, 3], full_o[1, 3]) and np.array_equal(o[0, 0], full_o[0, 0])
    assert not o[1, 2].any() and not o[0, 1].any()


def test_ancestors_worked_tree_and_invalid_parents():
    with open(os.path.join(GOLDEN, "tree_worked.json")) as f:
        doc = json.load(f)
    anc, depth = oracle.ancestors(doc["parent"], len(doc["parent"]))
    assert anc == doc["ancestors"] and depth == doc["depth"]
    for bad in ([0], [-1, 1], [-1, 0, -2], [-1, 5, 0]):
        with pytest.raises(ValueError):
            oracle.ancestors(bad, len(bad))
