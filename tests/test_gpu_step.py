"""GPU: the whole verify-and-repair step (tree attention, margins with the UFP
gate, accept) on named workloads, both as three calls and as the benchmark's
two (cure_tree_attn, cure_margins_accept), checked against the oracle chained
the same way; and the step captured as a HIP graph, replayed several times
with eager work in between, each replay checked against the eager result.
"""

import numpy as np
import pytest
import torch

import oracle
import paper_2608_00531_amd as pc
from synth import preset
from parity_util import (say, upload, gpu_margins, gpu_attn, check_margins, check_attn,
                         check_accept, oracle_attn)

pytestmark = pytest.mark.gpu


def run_step(w, dev, fused=False):
    o, lse, st = gpu_attn(w, dev)
    if fused:
        m = pc.cure_margins_accept(dev["logits"], dev["parent"], dev["token"], dev["root_tgt"],
                                   dev["n_nodes"], w.chain_len, tau=w.tau,
                                   repair_budget=w.repair_budget, branch_depth=w.branch_depth)
        acc = m
    else:
        m = gpu_margins(w, dev)
        acc = pc.cure_accept(dev["parent"], dev["token"], m["top1_idx"], dev["root_tgt"],
                             dev["n_nodes"], w.chain_len)
    return m, (o, lse, st), acc


@pytest.mark.parametrize("fused", [False, True])
@pytest.mark.parametrize("name", ["tiny_fp32", "llama3_8b_ctx2k_b1",
                                  "llama3_8b_ctx8k_b8_budget32", "llama3_8b_ragged_b16",
                                  "llama3_8b_ctx8k_b8_budget64"])
def test_step_chain_matches_oracle_chain(name, fused):
    say("step", name, "fused" if fused else "three calls")
    w = preset(name)
    dev = upload(w)
    m, (o, lse, st), acc = run_step(w, dev, fused)
    torch.cuda.synchronize()
    assert st.tolist() == [pc.CURE_OK] * w.batch
    check_margins(w, m)
    tgt = np.stack([oracle.margins(w.logits[b], w.dtype)["top1_idx"] for b in range(w.batch)])
    assert np.array_equal(tgt, w.tgt_planted)
    check_accept(w, acc, tgt)
    sample = [(b, n) for b in range(w.batch) for n in (0, int(w.n_nodes[b]) - 1)]
    ref_o, ref_l = oracle_attn(w, sample=sample)
    check_attn(w, o, lse, ref_o, ref_l, sample=sample)


@pytest.mark.parametrize("fused", [False, True])
def test_graph_replays_match_eager(fused):
    say("step graph replay", "fused" if fused else "three calls")
    w = preset("llama3_8b_ctx2k_b1")
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        dev = upload(w)
        eager = run_step(w, dev, fused)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            cap = run_step(w, dev, fused)
        for rep in range(4):
            # Eager work and a synchronisation between replays.
            junk = torch.randn(1 << 20, device="cuda").sum()
            torch.cuda.synchronize()
            for t in (cap[0]["top1_idx"], cap[2]["acc_len"], cap[1][0]):
                t.fill_(-7) if t.dtype != torch.bfloat16 else t.zero_()
            g.replay()
            torch.cuda.synchronize()
            for key in ("top1_idx", "top2_idx", "margin", "lse", "ufp_pos", "ufp_cnt"):
                assert torch.equal(cap[0][key], eager[0][key]), (rep, key)
            assert torch.equal(cap[1][0], eager[1][0]) and torch.equal(cap[1][1], eager[1][1])
            for key in ("acc_len", "path", "best", "bonus", "resync"):
                assert torch.equal(cap[2][key], eager[2][key]), (rep, key)
            del junk


def test_graph_replays_ragged_batch_with_repair():
    # The ragged 16-sequence batch (two context splits, the merge launch, the
    # UFP gate on unsplit rows) and the repair-tree builder fed the captured
    # margins, all in one graph: every replay, after eager work, reproduces
    # the eager results bit for bit.
    say("step graph replay, ragged batch + repair")
    w = preset("llama3_8b_ragged_b16")
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        dev = upload(w)
        chain_tok = dev["token"][:, : w.chain_len].contiguous()

        def step():
            m, att, acc = run_step(w, dev, fused=True)
            rep = pc.cure_repair_tree(dev["logits"], m["margin"], m["ufp_pos"], m["ufp_cnt"],
                                      chain_tok, w.repair_budget, w.branch_depth, w.tau)
            return m, att, acc, rep

        eager = step()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            cap = step()
        for rep_i in range(3):
            junk = torch.randn(1 << 20, device="cuda").sum()
            torch.cuda.synchronize()
            cap[0]["top1_idx"].fill_(-7)
            cap[1][0].zero_()
            cap[2]["acc_len"].fill_(-7)
            cap[3]["parent"].fill_(-7)
            g.replay()
            torch.cuda.synchronize()
            for key in ("top1_idx", "top2_idx", "margin", "lse", "ufp_pos", "ufp_cnt"):
                assert torch.equal(cap[0][key], eager[0][key]), (rep_i, key)
            assert torch.equal(cap[1][0], eager[1][0]) and torch.equal(cap[1][1], eager[1][1])
            for key in ("acc_len", "path", "best", "bonus", "resync"):
                assert torch.equal(cap[2][key], eager[2][key]), (rep_i, key)
            for key in ("parent", "token", "n_nodes", "branch_cnt"):
                assert torch.equal(cap[3][key], eager[3][key]), (rep_i, key)
            del junk
