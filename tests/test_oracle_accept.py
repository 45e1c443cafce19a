"""Pins for the acceptance oracle (Sec. 3.1 Eq. (1), Sec. 3.5 Eq. (4)).

The oracle walks nodes in index order with a per-node recursion. These tests
compare it with an enumeration of every root-to-leaf path, which computes
a(pi) for each path directly and takes Eq. (4)'s argmax, over every tree of up
to four nodes with every token/target assignment on a two-symbol vocabulary,
and over random larger trees; plus closed cases and a hand-worked fixture.
"""

import itertools
import json
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def brute_accept(parent, token, tgt, root_tgt, chain_len):
    """Enumerate root-to-leaf paths; a(pi) = longest prefix whose every token equals
    the target's argmax at the previous position; pick the longest, ties to the
    path whose last accepted node has the lowest index."""
    n = len(parent)
    kids = {p: [c for c in range(n) if parent[c] == p] for p in range(-1, n)}
    paths = []

    def walk(node, prefix):
        prefix = prefix + [node]
        if not kids[node]:
            paths.append(prefix)
        for c in kids[node]:
            walk(c, prefix)

    for r in kids[-1]:
        walk(r, [])
    best_a, best_end = 0, None
    for p in paths:
        a, prev = 0, root_tgt
        for node in p:
            if token[node] != prev:
                break
            a += 1
            prev = tgt[node]
        end = p[a - 1] if a else None
        if a > best_a or (a == best_a and a > 0 and end < best_end):
            best_a, best_end = a, end
    if best_a == 0:
        return 0, [], root_tgt, 0
    path = next(p[:best_a] for p in paths if len(p) >= best_a and p[best_a - 1] == best_end)
    return best_a, path, tgt[best_end], int(any(x >= chain_len for x in path))


def all_parent_arrays(n):
    return itertools.product(*[range(-1, i) for i in range(n)])


def check(parent, token, tgt, root_tgt, chain_len):
    got = oracle.accept(parent, token, tgt, root_tgt, len(parent), chain_len)
    a, path, bonus, resync = brute_accept(list(parent), list(token), list(tgt), root_tgt,
                                          chain_len)
    assert (got["acc_len"], got["path"], got["bonus"], got["resync"]) == (a, path, bonus, resync)
    assert got["best"] == (path[-1] if path else -1)


def test_exhaustive_small_trees_two_symbol_vocab():
    cases = 0
    for n in range(1, 5):
        for parent in all_parent_arrays(n):
            for token in itertools.product((0, 1), repeat=n):
                for tgts in itertools.product((0, 1), repeat=n + 1):
                    check(parent, token, tgts[1:], tgts[0], chain_len=min(2, n))
                    cases += 1
    assert cases > 10000


def test_random_larger_trees():
    rng = np.random.default_rng(31)
    for _ in range(3000):
        n = int(rng.integers(5, 13))
        parent = [int(rng.integers(-1, i)) if i else -1 for i in range(n)]
        token = [int(t) for t in rng.integers(0, 3, n)]
        tgt = [int(t) for t in rng.integers(0, 3, n)]
        check(parent, token, tgt, int(rng.integers(0, 3)), chain_len=int(rng.integers(1, n + 1)))


def test_pure_chain_is_prefix_matching():
    token = [5, 6, 7, 8, 9]
    tgt = [6, 7, 1, 9, 4]      # target agrees after nodes 0 and 1, then diverges
    out = oracle.accept([-1, 0, 1, 2, 3], token, tgt, 5, 5, 5)
    assert (out["acc_len"], out["path"], out["bonus"], out["resync"]) == (3, [0, 1, 2], 1, 0)


def test_all_agree_and_none_agree():
    parent = [-1, 0, 1, 0, 3, 4]
    token = [1, 2, 3, 9, 9, 9]
    # Every node's target names its first child's token; all depth-0 nodes match.
    tgt = [2, 3, 0, 9, 9, 0]
    out = oracle.accept(parent, token, tgt, 1, 6, 3)
    assert out["acc_len"] == 3 and out["path"] == [0, 1, 2] and out["resync"] == 0
    out = oracle.accept(parent, token, tgt, 7, 6, 3)
    assert (out["acc_len"], out["path"], out["best"], out["bonus"]) == (0, [], -1, 7)


def test_repair_branch_win_sets_resync():
    # chain 0-1-2; repair branch 3-4 replaces position 1 (parent 0).
    parent = [-1, 0, 1, 0, 3]
    token = [10, 11, 12, 21, 22]
    tgt = [21, 99, 99, 22, 5]
    out = oracle.accept(parent, token, tgt, 10, 5, 3)
    assert (out["acc_len"], out["path"], out["bonus"], out["resync"]) == (3, [0, 3, 4], 5, 1)


def test_equal_length_tie_prefers_branch_zero():
    parent = [-1, 0, 0]            # node 2 is a sibling of node 1 with the same token
    out = oracle.accept(parent, [4, 6, 6], [6, 8, 9], 4, 3, 2)
    assert out["path"] == [0, 1] and out["resync"] == 0 and out["bonus"] == 8


def test_golden_accept_fixture():
    with open(os.path.join(GOLDEN, "accept_worked.json")) as f:
        doc = json.load(f)
    for c in doc["cases"]:
        out = oracle.accept(c["parent"], c["token"], c["tgt"], c["root_tgt"],
                            len(c["parent"]), c["chain_len"])
        for key in ("acc_len", "path", "best", "bonus", "resync"):
            assert out[key] == c[key], (c["why"], key)


def test_invalid_tree_rejected():
    with pytest.raises(ValueError):
        oracle.accept([-1, 2, 0], [0, 0, 0], [0, 0, 0], 0, 3, 3)
