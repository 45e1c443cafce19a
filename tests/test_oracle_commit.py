"""Pins for the commit oracle (Sec. 3.5, Algorithm 1: accepted path and resync).

Checked against hand-worked commits, against the tree-attention oracle (the
committed cache gives the winner's query exactly the attention it had in the
tree), and against path facts derived independently from the parent array.
"""

import json
import math
import os

import numpy as np
import pytest

import oracle
from oracle import commit
from synth import make_workload

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def load_fixture():
    with open(os.path.join(GOLDEN, "commit_worked.json")) as f:
        return json.load(f)


def test_worked_commits():
    g = load_fixture()
    rows = np.array([[r, -r] for r in range(22)], np.int64)
    paths = [p + [0] * (8 - len(p)) for p in g["path"]]
    after = commit.commit_kv(rows, g["kv_off"], g["ctx_len"], paths, g["acc_len"])
    for b, c in enumerate(g["cases"]):
        lo = g["kv_off"][b]
        hi = lo + g["ctx_len"][b] + g["n_nodes"][b]
        assert after[lo:hi, 0].tolist() == c["rows_after"][0], c["why"]
        assert np.array_equal(after[lo:hi, 1], -after[lo:hi, 0])
        t = commit.commit_tokens(g["token"][b], paths[b], g["acc_len"][b], g["bonus"][b],
                                 g["chain_len"][b])
        assert t["emit"] == c["emit"], c["why"]
        assert t["replay_start"] == c["replay_start"], c["why"]
        assert t["new_ctx_add"] == c["new_ctx_add"], c["why"]
    # The input array is not modified.
    assert rows[:, 0].tolist() == list(range(22))


def _accept_all(w):
    return [oracle.accept(w.parent[b], w.token[b], w.tgt_planted[b], int(w.root_tgt[b]),
                          int(w.n_nodes[b]), w.chain_len) for b in range(w.batch)]


@pytest.mark.parametrize("seed", [2, 8, 13, 16, 18])
def test_committed_cache_reproduces_tree_attention_of_the_winner(seed):
    # Sec. 3.5: the accepted tokens become context. After the commit, plain
    # attention of the winner's query over the first ctx_len + a cache rows
    # must equal its tree attention over context plus ancestors. Each seed has
    # a sequence whose winning path runs through a repair branch.
    w = make_workload("commit", dtype="f32", batch=3, hq=4, hkv=2, d=16, vocab=64,
                      ctx_lens=[5, 9, 0], chain_len=6, n_ufp=2, branch_depth=3, seed=seed,
                      p_agree=0.9, scale=0.25)
    acc = _accept_all(w)
    paths = [r["path"] + [0] * (w.n_max - len(r["path"])) for r in acc]
    alen = [r["acc_len"] for r in acc]
    k2 = commit.commit_kv(w.k, w.kv_off, w.ctx_len, paths, alen)
    v2 = commit.commit_kv(w.v, w.kv_off, w.ctx_len, paths, alen)
    o_tree, lse_tree = oracle.tree_attention(w.q, w.k, w.v, "f32", w.kv_off, w.ctx_len,
                                             w.n_nodes, w.parent, w.hq, w.hkv, w.scale)
    checked = 0
    for b in range(w.batch):
        a = alen[b]
        if a <= 0:
            continue
        win = acc[b]["best"]
        lo = int(w.kv_off[b])
        hi = lo + int(w.ctx_len[b]) + a
        for h in range(w.hq):
            kh = h // (w.hq // w.hkv)
            q = w.q[b, win, h].astype(np.float64)
            s = (k2[lo:hi, kh].astype(np.float64) @ q) * w.scale
            m = s.max()
            p = np.exp(s - m)
            o = (p / p.sum()) @ v2[lo:hi, kh].astype(np.float64)
            assert np.allclose(o, o_tree[b, win, h], atol=1e-12, rtol=0)
            assert math.isclose(m + math.log(p.sum()), lse_tree[b, win, h], abs_tol=1e-12)
            checked += 1
    assert checked > 0
    assert any(r["resync"] for r in acc)


@pytest.mark.parametrize("seed", range(6))
def test_path_facts(seed):
    w = make_workload("commit", dtype="f32", batch=4, hq=2, hkv=1, d=4, vocab=16,
                      ctx_lens=[3, 0, 7, 2], chain_len=8, n_ufp=3, branch_depth=2,
                      seed=100 + seed, p_agree=0.85)
    acc = _accept_all(w)
    paths = [r["path"] + [0] * (w.n_max - len(r["path"])) for r in acc]
    alen = [r["acc_len"] for r in acc]
    k2 = commit.commit_kv(w.k, w.kv_off, w.ctx_len, paths, alen)
    for b in range(w.batch):
        a = alen[b]
        base = int(w.kv_off[b]) + int(w.ctx_len[b])
        end = base + int(w.n_nodes[b])
        # Rows outside [base, base + a) are untouched: the context, and the
        # tree rows past the accepted length.
        off = int(w.kv_off[b])
        assert np.array_equal(k2[off:base], w.k[off:base])
        assert np.array_equal(k2[base + a:end], w.k[base + a:end])
        # The winner's root path, walked up through the parent array.
        chain, n = [], acc[b]["best"]
        while n >= 0:
            chain.append(n)
            n = int(w.parent[b][n])
        chain.reverse()
        assert len(chain) == a
        for j, node in enumerate(chain):
            assert np.array_equal(k2[base + j], w.k[base + node])
        t = commit.commit_tokens(w.token[b], paths[b], a, acc[b]["bonus"], w.chain_len)
        assert t["emit"] == [int(w.token[b][n]) for n in chain] + [acc[b]["bonus"]]
        # Before the replay start the path runs along the draft chain (node j
        # at depth j); the node at the start, if any, is a repair node.
        rs = t["replay_start"]
        assert all(chain[j] == j for j in range(rs))
        assert rs == a or chain[rs] >= w.chain_len
        assert (rs < a) == bool(acc[b]["resync"])
