"""Pins for the margin and UFP oracle (Sec. 3.3 Eq. (2), Algorithm 1).

Every check here compares the oracle with something other than itself: a
pairwise brute force, scipy's logsumexp, torch's own bf16 widening, closed
forms, hand-worked fixtures, or the structure the generator planted.
"""

import itertools
import json
import math
import os

import numpy as np
import pytest
import scipy.special
import torch

import oracle
from synth import make_workload, bf16_round

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def brute_top2(row):
    """Top-2 by pairwise comparison: entry i beats j if x_i > x_j, or equal and i < j."""
    def beats(i, j):
        return row[i] > row[j] or (row[i] == row[j] and i < j)
    idx = list(range(len(row)))
    first = [i for i in idx if all(beats(i, j) for j in idx if j != i)][0]
    rest = [i for i in idx if i != first]
    second = [i for i in rest if all(beats(i, j) for j in rest if j != i)][0]
    return first, second


def test_bf16_widening_matches_torch():
    bits = np.array([0x3F80, 0xC000, 0x7F80, 0xFF80, 0x0001, 0x8001, 0x7F7F, 0x4049, 0],
                    np.uint16)
    mine = oracle.widen_bf16(bits)
    ref = torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).float().numpy()
    assert np.array_equal(mine.view(np.uint32), ref.view(np.uint32))
    rnd = np.random.default_rng(3).integers(0, 2 ** 16, 4096).astype(np.uint16)
    rnd = rnd[(rnd & 0x7F80) != 0x7F80]          # drop inf/NaN patterns
    ref = torch.from_numpy(rnd.view(np.int16).copy()).view(torch.bfloat16).float().numpy()
    assert np.array_equal(oracle.widen_bf16(rnd), ref)


def test_tiny_rows_against_pairwise_brute_force():
    values = [-np.inf, -1.5, 0.0, 0.25, 2.0, 2.0, 7.0]
    rng = np.random.default_rng(0)
    checked = 0
    for vocab in range(2, 7):
        for _ in range(150):
            row = rng.choice(values, size=vocab).astype(np.float32)
            if np.all(row == -np.inf):
                continue
            out = oracle.margins(row[None, :], "f32")
            i1, i2 = brute_top2(list(row))
            assert (out["top1_idx"][0], out["top2_idx"][0]) == (i1, i2)
            assert out["margin"][0] == float(row[i1]) - float(row[i2])
            ref_lse = scipy.special.logsumexp(row.astype(np.float64))
            assert out["lse"][0] == pytest.approx(ref_lse, abs=1e-12)
            checked += 1
    assert checked > 500


def test_exhaustive_small_value_set():
    # Every row of length 4 over {-inf, 0, 1, 1.5}: all tie patterns appear.
    vals = [-np.inf, 0.0, 1.0, 1.5]
    for row in itertools.product(vals, repeat=4):
        row = np.array(row, np.float32)
        if np.all(row == -np.inf):
            continue
        out = oracle.margins(row[None, :], "f32")
        assert (out["top1_idx"][0], out["top2_idx"][0]) == brute_top2(list(row))


def test_lse_against_scipy_and_log_softmax_order():
    rng = np.random.default_rng(1)
    x = (rng.standard_normal((6, 5000)) * 3).astype(np.float32)
    out = oracle.margins(x, "f32")
    lse = scipy.special.logsumexp(x.astype(np.float64), axis=1)
    assert np.allclose(out["lse"], lse, rtol=0, atol=1e-10)
    # Full softmax sort: the log-softmax has the same top-2 and the same margin.
    lp = x.astype(np.float64) - lse[:, None]
    for r in range(x.shape[0]):
        order = sorted(range(x.shape[1]), key=lambda v: (-lp[r, v], v))
        assert order[0] == out["top1_idx"][r] and order[1] == out["top2_idx"][r]
        assert lp[r, order[0]] - lp[r, order[1]] == pytest.approx(out["margin"][r], abs=1e-12)


def test_bf16_rows_against_torch_topk_and_logsumexp():
    rng = np.random.default_rng(2)
    vals = (rng.standard_normal((4, 20000)) * 3).astype(np.float32)
    bits = bf16_round(vals)
    out = oracle.margins(bits, "bf16")
    t = torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).double()
    assert np.allclose(out["lse"], torch.logsumexp(t, dim=1).numpy(), atol=1e-10, rtol=0)
    # torch.sort(stable=True) of the negated values gives the same lowest-index tie rule.
    order = torch.sort(-t, dim=1, stable=True).indices.numpy()
    assert np.array_equal(out["top1_idx"], order[:, 0])
    assert np.array_equal(out["top2_idx"], order[:, 1])


def test_closed_forms_and_degenerate_rows():
    out = oracle.margins(np.full((1, 1000), 2.5, np.float32), "f32")
    assert (out["top1_idx"][0], out["top2_idx"][0], out["margin"][0]) == (0, 1, 0.0)
    assert out["lse"][0] == pytest.approx(2.5 + math.log(1000), abs=1e-12)
    # A large shift must not overflow: lse(x + c) = lse(x) + c.
    base = np.array([[0.0, 1.0, -2.0, 0.5]], np.float32)
    big = base + np.float32(1000.0)
    assert oracle.margins(big, "f32")["lse"][0] == pytest.approx(
        oracle.margins(base, "f32")["lse"][0] + 1000.0, abs=1e-9)
    # -inf entries contribute nothing; two finite entries decide.
    out = oracle.margins(np.array([[-np.inf, 3.0, -np.inf, 1.0]], np.float32), "f32")
    assert (out["top1_idx"][0], out["top2_idx"][0], out["margin"][0]) == (1, 3, 2.0)
    assert out["lse"][0] == pytest.approx(math.log(math.exp(3) + math.exp(1)), abs=1e-12)
    # A single finite entry: the top-2 is the first -inf, the margin is +inf.
    out = oracle.margins(np.array([[-np.inf, -np.inf, 4.0]], np.float32), "f32")
    assert (out["top1_idx"][0], out["top2_idx"][0]) == (2, 0)
    assert out["margin"][0] == np.inf and out["lse"][0] == pytest.approx(4.0)
    # All -inf: lse is -inf, indices 0 and 1, margin undefined (NaN).
    out = oracle.margins(np.full((1, 3), -np.inf, np.float32), "f32")
    assert (out["top1_idx"][0], out["top2_idx"][0]) == (0, 1)
    assert out["lse"][0] == -np.inf and np.isnan(out["margin"][0])


def test_golden_margin_fixture():
    with open(os.path.join(GOLDEN, "margins_worked.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        row = np.array([-np.inf if v == "-inf" else v for v in c["row"]], np.float32)
        out = oracle.margins(row[None, :], "f32")
        assert out["top1_idx"][0] == c["top1_idx"]
        assert out["top2_idx"][0] == c["top2_idx"]
        assert out["margin"][0] == pytest.approx(c["margin"], abs=1e-12)
        lse = math.log(math.fsum(cnt * math.exp(val) for cnt, val in c["lse_terms"]))
        assert out["lse"][0] == pytest.approx(lse, abs=1e-12)


def test_planted_argmax_and_gap_recovered():
    w = make_workload("t", batch=2, hq=4, hkv=1, d=64, vocab=3000, ctx_lens=[16, 16],
                      chain_len=16, n_ufp=4, branch_depth=2, seed=11)
    for b in range(w.batch):
        out = oracle.margins(w.logits[b], "bf16")
        assert np.array_equal(out["top1_idx"], w.tgt_planted[b])
        assert np.all(out["margin"] >= 0.02)
        m = out["margin_f32"][: w.chain_len]
        ufp = set(w.ufp_planted[b])
        assert all(m[i] < 0.53 for i in ufp)
        assert all(m[i] > 0.69 for i in range(w.chain_len) if i not in ufp)


# ---- UFP selection (Sec. 3.3, Algorithm 1) ----

def brute_ufp(m, tau, budget, depth):
    """Rank-based: position i is kept iff it is a candidate and fewer than
    floor(budget/depth) candidates precede it in (margin, position) order; the
    output is the kept positions listed by rank."""
    cand = [i for i in range(len(m)) if m[i] < tau]
    cap = budget // depth
    ranked = {}
    for i in cand:
        rank = sum(1 for j in cand if (m[j] < m[i]) or (m[j] == m[i] and j < i))
        if rank < cap:
            ranked[rank] = i
    return [ranked[r] for r in sorted(ranked)]


def test_ufp_against_rank_brute_force():
    rng = np.random.default_rng(5)
    levels = np.array([0.1, 0.5, 0.5, 0.9, 1.0, 1.5, 3.0], np.float32)
    for _ in range(2000):
        K = int(rng.integers(1, 20))
        m = rng.choice(levels, size=K)
        tau = float(rng.choice([0.0, 0.5, 1.0, 2.0, np.inf]))
        budget = int(rng.integers(0, 40))
        depth = int(rng.integers(1, 6))
        assert oracle.ufp_select(m, tau, budget, depth) == brute_ufp(list(m), tau, budget, depth)


def test_ufp_worked_example_and_edges():
    m = np.array([0.5, 2.0, 0.1, 0.5, 0.9], np.float32)
    # candidates {0, 2, 3, 4}; ascending (m, i): 2, 0, 3, 4; budget 8 / depth 4 -> 2 kept
    assert oracle.ufp_select(m, 1.0, 8, 4) == [2, 0]
    assert oracle.ufp_select(m, 1.0, 100, 1) == [2, 0, 3, 4]
    assert oracle.ufp_select(m, 0.5, 100, 1) == [2]            # strict: m == tau is not a UFP
    assert oracle.ufp_select(m, -np.inf, 100, 1) == []
    assert oracle.ufp_select(m, 1.0, 3, 4) == []               # a whole branch does not fit
    assert oracle.ufp_select(m, np.inf, 100, 1) == [2, 0, 3, 4, 1]


def test_margins_invariant_under_permutation_of_positions():
    # Eq. 2 reads a row as a multiset of (position, value): permuting the
    # positions of a tie-free row leaves the top-1/top-2 values, the margin and
    # the log-sum-exp unchanged and moves the reported indices with it.
    rng = np.random.default_rng(21)
    for vocab in (2, 3, 17, 256, 5000):
        for _ in range(6):
            row = rng.permutation(np.linspace(-6.0, 9.0, vocab)).astype(np.float32)
            perm = rng.permutation(vocab)
            moved = row[perm]                       # moved[j] = row[perm[j]]
            inv = np.empty(vocab, np.int64)
            inv[perm] = np.arange(vocab)
            a = oracle.margins(row[None, :], "f32")
            b = oracle.margins(moved[None, :], "f32")
            assert b["top1_val"][0] == a["top1_val"][0] and b["top2_val"][0] == a["top2_val"][0]
            assert b["margin"][0] == a["margin"][0]
            assert b["lse"][0] == pytest.approx(a["lse"][0], abs=1e-12)
            assert b["top1_idx"][0] == inv[a["top1_idx"][0]]
            assert b["top2_idx"][0] == inv[a["top2_idx"][0]]


def subset_brute_ufp(m, tau, budget, depth):
    """Over every subset of the candidate positions (margin < tau) that fits
    the budget in whole branches, the best is the largest one whose entries,
    listed in ascending (margin, position) order, are lexicographically
    smallest; returned in that order."""
    cand = [i for i in range(len(m)) if m[i] < tau]
    best = None
    for k in range(len(cand) + 1):
        if k * depth > budget:
            break
        for sub in itertools.combinations(cand, k):
            key = sorted((float(m[i]), i) for i in sub)
            if best is None or len(key) > len(best) or (len(key) == len(best) and key < best):
                best = key
    return [i for _, i in best]


def test_ufp_against_subset_brute_force():
    rng = np.random.default_rng(8)
    levels = np.array([0.1, 0.5, 0.5, 0.9, 1.0, 1.5, 3.0], np.float32)
    for _ in range(400):
        K = int(rng.integers(1, 9))
        m = rng.choice(levels, size=K)
        tau = float(rng.choice([0.0, 0.5, 1.0, 2.0, np.inf]))
        budget = int(rng.integers(0, 24))
        depth = int(rng.integers(1, 5))
        assert oracle.ufp_select(m, tau, budget, depth) == subset_brute_ufp(m, tau, budget, depth)
