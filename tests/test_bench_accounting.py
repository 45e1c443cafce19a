"""The bench's work accounting (no GPU): algorithmic bytes and attention flops
against closed forms on small synthetic workloads."""

import os
import sys

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import bench  # noqa: E402
from synth import algorithmic_bytes, make_workload  # noqa: E402


def test_attention_flops_of_a_pure_chain():
    # No branches: node i of a chain sees the L context rows and nodes 0 .. i,
    # so the visible pairs per head are N L + N (N + 1) / 2.
    L, N, hq, d = 100, 16, 8, 64
    w = make_workload("chain", batch=1, hq=hq, hkv=2, d=d, ctx_lens=[L], chain_len=N,
                      n_ufp=0, branch_depth=4, seed=3, vocab=64)
    assert int(w.n_nodes[0]) == N
    assert bench.attention_flops(w) == 4 * hq * d * (N * L + N * (N + 1) // 2)


def test_attention_flops_count_each_branch_node_at_its_depth():
    # One depth-3 branch at UFP position u: its nodes sit at depths u .. u + 2
    # (root parent = chain node u - 1), so they see u + 1, u + 2, u + 3 tree rows.
    L, K, hq, d, depth = 50, 8, 4, 32, 3
    w = make_workload("branch", batch=1, hq=hq, hkv=4, d=d, ctx_lens=[L], chain_len=K,
                      n_ufp=1, branch_depth=depth, seed=5, vocab=64)
    par = np.asarray(w.parent[0][:int(w.n_nodes[0])])
    root = K
    u = int(par[root]) + 1                       # the branch replaces chain token u
    chain = K * L + K * (K + 1) // 2
    branch = depth * L + sum(u + 1 + j for j in range(depth))
    assert bench.attention_flops(w) == 4 * hq * d * (chain + branch)


def test_attention_flops_of_the_widest_sweep_tree():
    # Batch 8, context 8192, 16-node chain plus 16 depth-4 branches (80 nodes):
    # about 86 GFLOP, the figure the budget-64 sweep point is priced against.
    w = make_workload("w", batch=8, ctx_lens=[8192] * 8, chain_len=16, n_ufp=16,
                      branch_depth=4, seed=564, vocab=64)
    f = bench.attention_flops(w)
    per_seq = 4 * 32 * 128 * (80 * 8192)
    assert per_seq * 8 < f < per_seq * 8 * 1.01
    b = algorithmic_bytes(w)
    assert b["attention_kv"] == 8 * (8192 + 80) * 8 * 128 * 2 * 2
