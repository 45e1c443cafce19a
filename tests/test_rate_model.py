"""The acceptance-compute sweep's arithmetic (no GPU).

Sec. 3.1 models the generation rate as (E[a] + 1) / (C_d + C_v(Pi)); Table 1
reports speedup as a ratio of times per output token (Sec. 4.1) and the
accepted-length gain over the parallel draft. The bench's helpers are pinned
here against Table 1's own numbers and against a hand-worked sweep.
"""

import json
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402

GOLDEN = os.path.join(ROOT, "tests", "golden", "table1_end_to_end.json")


def _table():
    with open(GOLDEN) as f:
        t = json.load(f)
    rows = {name: dict(zip(t["columns"], vals)) for name, vals in t["rows"].items()}
    return t, rows


def test_speedup_reproduces_table1_columns():
    # Every printed speedup is TPOT(target AR) / TPOT(method), to the printed
    # three decimals (HumanEval: 30.430 / 8.718 = 3.490).
    _, rows = _table()
    for name, r in rows.items():
        assert round(bench.speedup(r["tpot_target_ar"], r["tpot_parallel"]), 3) == \
            pytest.approx(r["speedup_parallel"], abs=1e-9), name
        assert round(bench.speedup(r["tpot_target_ar"], r["tpot_method"]), 3) == \
            pytest.approx(r["speedup_method"], abs=1e-9), name
    assert round(bench.speedup(30.430, 8.718), 3) == 3.490


def test_accept_gain_and_quoted_ranges():
    t, rows = _table()
    q = t["quoted"]
    code = t["code_suites"]
    gains = {n: 100 * bench.accept_gain(rows[n]["accepted_parallel"], rows[n]["accepted_method"])
             for n in code}
    assert round(gains["HumanEval"], 1) == q["humaneval_accept_gain_pct"]       # 7.641 / 7.165
    assert round(gains["LCB-lite"], 1) == q["lcb_accept_gain_pct"]              # 6.735 / 6.268
    assert [round(min(gains.values()), 1), round(max(gains.values()), 1)] == q["accept_gain_range_pct"]
    sp = [bench.speedup(rows[n]["tpot_target_ar"], rows[n]["tpot_method"]) for n in code]
    assert [round(min(sp), 2), round(max(sp), 2)] == q["speedup_range"]
    over = [rows[n]["tpot_method"] / rows[n]["tpot_parallel"] for n in code]
    assert [round(min(over), 2), round(max(over), 2)] == q["tpot_overhead_range"]
    he = rows["HumanEval"]
    assert round(bench.speedup(he["tpot_naive_sd"], he["tpot_method"]), 2) == q["humaneval_over_naive_sd"]
    # A gain is the reverse of a loss: the reference row gains nothing.
    assert bench.accept_gain(5.0, 5.0) == 0.0


def test_rate_and_time_per_token_are_one_model():
    # One step costs C_d + C_v and emits E[a] + 1 tokens per sequence.
    assert bench.tpot_model(30.0, 70.0, 4.0) == pytest.approx(20.0)
    assert bench.rate_model(4.0, 1, 30.0, 70.0) == pytest.approx(50000.0)    # 5 / 100 us
    assert bench.rate_model(4.0, 8, 30.0, 70.0) == pytest.approx(400000.0)   # batch of 8
    # The rate ratio of two settings is the speedup of their times per token:
    # with Table 1's HumanEval accepted lengths and a step cost chosen so the
    # model reproduces each measured TPOT, the ratio is the printed TPOT ratio.
    _, rows = _table()
    he = rows["HumanEval"]
    step_par = he["tpot_parallel"] * (he["accepted_parallel"] + 1)
    step_cure = he["tpot_method"] * (he["accepted_method"] + 1)
    assert bench.tpot_model(0.0, step_par, he["accepted_parallel"]) == pytest.approx(he["tpot_parallel"])
    r_par = bench.rate_model(he["accepted_parallel"], 1, 0.0, step_par)
    r_cure = bench.rate_model(he["accepted_method"], 1, 0.0, step_cure)
    assert r_cure / r_par == pytest.approx(bench.speedup(he["tpot_parallel"], he["tpot_method"]))
    assert round(r_par / r_cure, 2) == 1.40          # the quoted TPOT overhead on HumanEval


def test_verify_cost_counts_every_layer():
    # 32 layers of 10 us attention, 5 us margins, 1 us accept, 100 us weights.
    assert bench.verify_cost(32, 10.0, 5.0, 1.0, 100.0) == pytest.approx(426.0)


def test_rate_table_hand_worked():
    # Three budgets, batch 2, one layer, weight stream 40 us.
    rows = [
        {"budget": 0, "tree_nodes": 16, "mean_accepted": 3.0, "attn_us": 50.0,
         "margins_us": 8.0, "accept_us": 2.0},
        {"budget": 8, "tree_nodes": 24, "mean_accepted": 4.0, "attn_us": 80.0,
         "margins_us": 8.0, "accept_us": 2.0},
        {"budget": 16, "tree_nodes": 32, "mean_accepted": 4.5, "attn_us": 120.0,
         "margins_us": 8.0, "accept_us": 2.0},
    ]
    # C_v = attn + 8 + 2 + 40: 100, 130, 170 us.
    table, best = bench.rate_table(rows, 40.0, 1, 2, ratios=(0.25, 2.0))
    assert [r["c_v_us"] for r in table] == [100.0, 130.0, 170.0]
    # C_d = 10 us: rates 4*2/110us = 72727.3, 5*2/140us = 71428.6, 5.5*2/180us = 61111.1.
    assert [r["tokens_per_s_cd0.25"] for r in table] == [72727.3, 71428.6, 61111.1]
    assert best["cd_0.25_x_weights"] == {"budget": 0, "tokens_per_s": 72727.3,
                                         "gain_vs_budget0": 1.0}
    # C_d = 80 us: rates 8/180us = 44444.4, 10/210us = 47619.0, 11/250us = 44000.0;
    # budget 8 wins by (180/4) / (210/5) = 45 / 42 = 1.0714.
    assert [r["tokens_per_s_cd2"] for r in table] == [44444.4, 47619.0, 44000.0]
    assert best["cd_2_x_weights"] == {"budget": 8, "tokens_per_s": 47619.0,
                                      "gain_vs_budget0": 1.0714}


def test_rate_table_ties_go_to_the_smaller_budget():
    # Equal rates: the smaller tree is the cheaper choice.
    rows = [{"budget": b, "tree_nodes": 16 + b, "mean_accepted": 4.0, "attn_us": 10.0,
             "margins_us": 0.0, "accept_us": 0.0} for b in (0, 8)]
    _, best = bench.rate_table(rows, 10.0, 1, 1, ratios=(1.0,))
    assert best["cd_1_x_weights"]["budget"] == 0


def test_chain_acceptance_matches_geometric_closed_form():
    # The sweep's E[a] at budget 0: a pure 16-node chain whose nodes agree with
    # the synthetic target i.i.d. with probability p. The accepted length is the
    # number of leading agreements (Eq. 1), so E[a] = sum_{k=1..16} p^k, 3.887
    # at p = 0.8. The acceptance here is the oracle's; the GPU estimate the
    # sweep reports is checked against the same closed form in the GPU tests.
    import math
    import numpy as np
    import oracle
    from synth import make_workload
    n, p = 3000, 0.8
    w = make_workload("chain", dtype="f32", batch=n, hq=1, hkv=1, d=4, vocab=64,
                      ctx_lens=[1] * n, chain_len=16, n_ufp=0, branch_depth=4, seed=901,
                      p_agree=p)
    acc = np.array([oracle.accept(w.parent[b], w.token[b], w.tgt_planted[b], int(w.root_tgt[b]),
                                  int(w.n_nodes[b]), w.chain_len)["acc_len"] for b in range(n)])
    closed = sum(p ** k for k in range(1, 17))
    assert closed == pytest.approx(p * (1 - p ** 16) / (1 - p))
    se = acc.std() / math.sqrt(n)
    assert abs(acc.mean() - closed) < 4 * se
