"""GPU parity: cure_accept (Eq. 1, Eq. 4) against the oracle, bit-exact."""

import numpy as np
import pytest
import torch

import oracle
import paper_2608_00531_amd as pc
from synth import preset, make_workload
from parity_util import say, upload, check_accept

pytestmark = pytest.mark.gpu


def _run(parent, token, tgt, root_tgt, n_nodes, chain_len):
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()
    return pc.cure_accept(t(parent), t(token), t(tgt), t(root_tgt), t(n_nodes), chain_len)


@pytest.mark.parametrize("name", ["tiny_fp32", "llama3_8b_ctx2k_b1"])
def test_preset_trees_with_planted_targets(name):
    say("accept", name)
    w = preset(name)
    got = _run(w.parent, w.token, w.tgt_planted, w.root_tgt, w.n_nodes, w.chain_len)
    check_accept(w, got, w.tgt_planted)


def test_budget_sweep_trees():
    say("accept budget sweep")
    for budget in (0, 8, 16, 32, 64):
        w = make_workload("s", batch=8, hq=4, hkv=1, d=64, vocab=50, ctx_lens=[4] * 8,
                          chain_len=16, n_ufp=budget // 4, branch_depth=4, seed=500 + budget)
        got = _run(w.parent, w.token, w.tgt_planted, w.root_tgt, w.n_nodes, w.chain_len)
        check_accept(w, got, w.tgt_planted)


def test_random_trees_small_vocab():
    say("accept random trees")
    rng = np.random.default_rng(77)
    B, n_max = 64, 256
    parent = np.full((B, n_max), -1, np.int32)
    token = rng.integers(0, 3, (B, n_max)).astype(np.int32)
    tgt = rng.integers(0, 3, (B, n_max)).astype(np.int32)
    root = rng.integers(0, 3, B).astype(np.int32)
    n_nodes = rng.integers(0, n_max + 1, B).astype(np.int32)
    n_nodes[:4] = [0, 1, 255, 256]
    for b in range(B):
        for n in range(1, int(n_nodes[b])):
            # Deep trees: mostly extend a recent node.
            parent[b, n] = int(rng.integers(max(-1, n - 4), n))
    chain = 16
    got = _run(parent, token, tgt, root, n_nodes, chain)
    for b in range(B):
        ref = oracle.accept(parent[b], token[b], tgt[b], int(root[b]), int(n_nodes[b]), chain)
        assert int(got["acc_len"][b]) == ref["acc_len"], b
        assert int(got["best"][b]) == ref["best"]
        assert int(got["bonus"][b]) == ref["bonus"]
        assert int(got["resync"][b]) == ref["resync"]
        p = got["path"][b].tolist()
        assert p[: ref["acc_len"]] == ref["path"] and all(x == -1 for x in p[ref["acc_len"]:])


def test_malformed_tree_reports_minus_one():
    say("accept malformed tree")
    parent = np.array([[-1, 0, 5, 1], [-1, 0, 1, 2]], np.int32)   # seq 0: parent[2] = 5 >= 2
    token = np.zeros((2, 4), np.int32)
    tgt = np.zeros((2, 4), np.int32)
    got = _run(parent, token, tgt, np.array([0, 0], np.int32), np.array([4, 4], np.int32), 4)
    assert int(got["acc_len"][0]) == -1 and int(got["resync"][0]) == -1
    assert got["path"][0].tolist() == [-1] * 4
    assert int(got["acc_len"][1]) == 4 and got["path"][1].tolist() == [0, 1, 2, 3]


@pytest.mark.parametrize("seed", range(16))
def test_random_batches(seed):
    # Seeded random batches: up to 32 sequences, n_max 1 .. 256, alphabets of
    # 2 .. 1000 tokens, chain lengths 1 .. 32 and trees that mostly extend a
    # chain then attach within a random span of recent nodes.
    rng = np.random.default_rng(9500 + seed)
    B = int(rng.integers(1, 33))
    n_max = int(rng.integers(1, 257))
    alpha = int(rng.choice([2, 3, 5, 50, 1000]))
    chain = int(rng.integers(1, 33))
    say("accept random", seed, B, n_max, alpha, chain)
    parent = np.full((B, n_max), -1, np.int32)
    n_nodes = rng.integers(0, n_max + 1, B).astype(np.int32)
    span = int(rng.integers(1, 10))
    for b in range(B):
        for n in range(1, int(n_nodes[b])):
            parent[b, n] = (n - 1 if (n < chain and rng.random() < 0.8)
                            else int(rng.integers(max(-1, n - span), n)))
    token = rng.integers(0, alpha, (B, n_max)).astype(np.int32)
    tgt = rng.integers(0, alpha, (B, n_max)).astype(np.int32)
    root = rng.integers(0, alpha, B).astype(np.int32)
    got = _run(parent, token, tgt, root, n_nodes, chain)
    for b in range(B):
        ref = oracle.accept(parent[b], token[b], tgt[b], int(root[b]), int(n_nodes[b]), chain)
        assert int(got["acc_len"][b]) == ref["acc_len"], b
        assert int(got["best"][b]) == ref["best"]
        assert int(got["bonus"][b]) == ref["bonus"]
        assert int(got["resync"][b]) == ref["resync"]
        p = got["path"][b].tolist()
        assert p[: ref["acc_len"]] == ref["path"] and all(x == -1 for x in p[ref["acc_len"]:])


def test_sweep_mean_accepted_chain_closed_form():
    # The sweep's E[a] estimate (cure_accept over 2048 seeded trees) at budget
    # 0, a pure 16-node chain agreeing i.i.d. with probability 0.8: the
    # accepted length is the run of leading agreements, E[a] = sum_k 0.8^k.
    import os
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    if root not in sys.path:
        sys.path.insert(0, root)
    import bench
    say("accept sweep E[a] closed form")
    mean, se, resync = bench.mean_accepted(pc, torch, 0, 2048, 0)
    closed = sum(0.8 ** k for k in range(1, 17))
    assert abs(mean - closed) < 4 * se, (mean, se, closed)
    assert resync == 0.0                 # a chain has no repair node to resync
