"""Pins for the repair-tree oracle (Eq. (3), Algorithm 1, Sec. 3.4).

The oracle is checked against hand-derived values of Eq. (3), a pairwise brute
force for the ranked alternatives, hand-worked trees, and structural
invariants that any correct construction satisfies.
"""

import json
import math
import os

import numpy as np
import pytest

import oracle
from oracle import repair

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# Eq. (3) at s = 1, b_min = 1, b_max = 5, so t = 1 + 4 u with u = 1 - m, worked
# by hand; 0.125, 0.375, 0.625 and 0.875 land exactly on halves and round to
# the even neighbour.
EQ3_TABLE = [
    (0.0, 5), (0.125, 4), (0.25, 4), (0.375, 4), (0.5, 3), (0.625, 2),
    (0.75, 2), (0.875, 2), (1.0, 1), (2.0, 1), (math.inf, 1), (-1.0, 5),
    (math.nan, 1),
]


@pytest.mark.parametrize("m,b", EQ3_TABLE)
def test_branch_budget_table(m, b):
    assert repair.branch_budget(np.float32(m), 1.0, 1, 5) == b


def test_branch_budget_scale_and_range():
    # u depends on m / s only: scaling both leaves b unchanged.
    for m in (0.0, 0.3, 0.5, 0.9, 1.7):
        assert repair.branch_budget(np.float32(m), 1.0) == repair.branch_budget(np.float32(4 * m), 4.0)
    # b_min == b_max pins the result; the output always lies in [b_min, b_max]
    # and never increases with the margin.
    rng = np.random.default_rng(3)
    ms = np.sort(rng.uniform(0, 3, 500).astype(np.float32))
    for lo, hi in ((1, 5), (0, 4), (2, 2), (0, 7)):
        bs = [repair.branch_budget(m, 1.5, lo, hi) for m in ms]
        assert all(lo <= x <= hi for x in bs)
        assert all(x >= y for x, y in zip(bs, bs[1:]))
        assert bs[0] == hi or ms[0] > 0
    assert repair.branch_budget(np.float32(0), 1.0, 0, 4) == 4
    assert repair.branch_budget(np.float32(10), 1.0, 0, 4) == 0


def brute_ranked(row, k):
    """The k best entries by pairwise wins: i beats j if x_i > x_j or equal and i < j."""
    n = len(row)
    wins = [sum(1 for j in range(n) if j != i and (row[i] > row[j] or (row[i] == row[j] and i < j)))
            for i in range(n)]
    order = sorted(range(n), key=lambda i: -wins[i])
    return order[:k]


@pytest.mark.parametrize("seed", range(6))
def test_topk_brute_force(seed):
    rng = np.random.default_rng(seed)
    vocab = int(rng.integers(6, 40))
    x = rng.integers(-4, 4, size=(5, vocab)).astype(np.float32)   # many ties
    x[rng.random(x.shape) < 0.15] = -np.inf
    k = min(6, vocab)
    vals, idx = repair.topk(x, "f32", k)
    for r in range(x.shape[0]):
        ref = brute_ranked(list(x[r]), k)
        assert list(idx[r]) == ref
        assert np.array_equal(vals[r], x[r][ref])


def test_topk_bf16_matches_margins():
    # The first two ranked entries are the margin pass's top-1 and top-2.
    rng = np.random.default_rng(11)
    bits = (rng.integers(0x3000, 0x4100, size=(7, 300))).astype(np.uint16)
    vals, idx = repair.topk(bits, "bf16", 6)
    m = oracle.margins(bits, "bf16")
    assert np.array_equal(idx[:, 0], m["top1_idx"]) and np.array_equal(idx[:, 1], m["top2_idx"])
    assert np.all(np.diff(vals, axis=1) <= 0)


def _case_args(c):
    K = len(c["chain_tok"])
    kk = c["b_max"] + 1
    ranked = np.zeros((K, kk), np.int64)
    for u, lst in c["ranked"].items():
        ranked[int(u)] = lst
    suffix = None
    if c["suffix"] is not None:
        suffix = np.zeros((K, c["b_max"], c["depth"] - 1), np.int64)
        for u, lst in c["suffix"].items():
            suffix[int(u)] = lst
    return dict(chain_tok=c["chain_tok"], margin_f32=np.asarray(c["margin"], np.float32),
                ufp_pos=c["ufp_pos"], topk_idx=ranked, suffix=suffix,
                repair_budget=c["repair_budget"], depth=c["depth"], scale=c["scale"],
                b_min=c["b_min"], b_max=c["b_max"])


def test_worked_trees():
    with open(os.path.join(GOLDEN, "repair_worked.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        t = repair.repair_tree(**_case_args(c))
        assert t["branches"] == c["branches"], c["why"]
        assert t["parent"] == c["parent"], c["why"]
        assert t["token"] == c["token"], c["why"]
        assert t["n_nodes"] == len(c["parent"])


def test_placeholder_suffix():
    with open(os.path.join(GOLDEN, "repair_worked.json")) as f:
        c = json.load(f)["cases"][0]
    args = _case_args(c)
    args["suffix"] = None
    t = repair.repair_tree(**args)
    assert t["parent"] == c["parent"]
    want = [tok if n < 4 or n % 2 == 0 else -1 for n, tok in enumerate(c["token"])]
    assert t["token"] == want


def random_case(rng, K=16, vocab=50, b_min=1, b_max=5, depth=4, budget=40, n_ufp=6):
    chain = rng.integers(0, vocab, K)
    margin = rng.uniform(0, 2, K).astype(np.float32)
    ufp = [int(i) for i in np.argsort(margin, kind="stable")[:n_ufp]]
    ranked = np.stack([rng.permutation(vocab)[:b_max + 1] for _ in range(K)])
    greedy = rng.random(K) < 0.7
    ranked[greedy, 0] = chain[greedy]               # greedy draft: own token ranks first
    for u in range(K):                              # keep each list free of duplicates
        if greedy[u]:
            rest = [t for t in rng.permutation(vocab) if t != chain[u]][:b_max]
            ranked[u, 1:] = rest
    suffix = rng.integers(0, vocab, (K, b_max, max(depth - 1, 0)))
    return dict(chain_tok=chain, margin_f32=margin, ufp_pos=ufp, topk_idx=ranked,
                suffix=suffix, repair_budget=budget, depth=depth, scale=1.0,
                b_min=b_min, b_max=b_max)


@pytest.mark.parametrize("seed", range(12))
def test_tree_invariants(seed):
    rng = np.random.default_rng(100 + seed)
    depth = int(rng.integers(1, 6))
    args = random_case(rng, depth=depth, budget=int(rng.integers(0, 60)),
                       b_min=int(rng.integers(0, 2)), n_ufp=int(rng.integers(0, 9)))
    t = repair.repair_tree(**args)
    K = len(args["chain_tok"])
    parent, token, src = t["parent"], t["token"], t["src"]
    # The chain comes first, unchanged.
    assert parent[:K] == list(range(-1, K - 1)) and token[:K] == [int(x) for x in args["chain_tok"]]
    # Topological order, and the node count adds up to whole branches within budget.
    assert all(-1 <= p < n for n, p in enumerate(parent))
    assert t["n_nodes"] == K + depth * sum(t["branches"]) <= K + args["repair_budget"]
    # The walk stops only when the next UFP's branches no longer fit.
    used = depth * sum(t["branches"])
    if len(t["branches"]) < len(args["ufp_pos"]):
        assert args["repair_budget"] - used < depth
    # Each UFP receives min(Eq. (3), what fits) branches.
    remaining = args["repair_budget"]
    for s, nb in enumerate(t["branches"]):
        u = args["ufp_pos"][s]
        b = repair.branch_budget(args["margin_f32"][u], args["scale"], args["b_min"], args["b_max"])
        assert nb == min(b, remaining // depth)
        remaining -= nb * depth
    # Branch structure: roots hang off the chain node before their position and
    # carry alternatives (ranked tokens other than the draft's own), in rank order.
    n = K
    for s, nb in enumerate(t["branches"]):
        u = args["ufp_pos"][s]
        alts = [int(x) for x in args["topk_idx"][u] if x != args["chain_tok"][u]]
        for r in range(nb):
            assert parent[n] == u - 1 and token[n] == alts[r] and src[n] == u * args["b_max"] + r
            for j in range(1, depth):
                assert parent[n + j] == n + j - 1
                assert token[n + j] == args["suffix"][u][r][j - 1]
            n += depth
    assert n == t["n_nodes"]
    # Position semantics: a branch substitutes block position u, so its node j
    # sits at depth u + j and sees exactly the chain prefix 0 .. u-1.
    anc, dep = oracle.ancestors(parent, t["n_nodes"])
    n = K
    for s, nb in enumerate(t["branches"]):
        u = args["ufp_pos"][s]
        for r in range(nb):
            for j in range(depth):
                assert dep[n + j] == u + j
                assert [a for a in anc[n + j] if a < K] == list(range(u))
            n += depth
