"""GPU: the allocation-free margin pass (cure_margins_noalloc) against
cure_margins on the same logits, on two calls in a row (the second smaller, so
it runs over scratch the first one left behind), plus the oracle's indices and
UFP lists on the same bytes."""

import numpy as np
import pytest
import torch

import paper_2608_00531_amd as pc
from synth import make_workload
from parity_util import say, to_dev, check_margins

pytestmark = pytest.mark.gpu


def _same(a, b):
    for k in a:
        assert torch.equal(a[k], b[k]) if a[k].dtype != torch.float32 else \
            torch.equal(torch.nan_to_num(a[k], nan=7.0), torch.nan_to_num(b[k], nan=7.0)), k


def _case(name, **kw):
    w = make_workload(name, **kw)
    return w, to_dev(w.logits, w.dtype)


def test_noalloc_matches_workspace_entry_point_twice():
    # First call: 2 x 32 rows of a 128256-entry vocabulary, rows split in 8
    # chunks (scratch in use); second call: 1 x 8 rows of 50000 entries in 7
    # chunks, reading scratch the first call wrote beyond its own records.
    cases = [
        dict(dtype="bf16", batch=2, hq=4, hkv=1, d=64, vocab=128256, ctx_lens=[8, 8],
             chain_len=16, n_ufp=4, branch_depth=4, seed=31),
        dict(dtype="bf16", batch=1, hq=4, hkv=1, d=64, vocab=50000, ctx_lens=[8],
             chain_len=4, n_ufp=1, branch_depth=4, seed=32),
    ]
    assert pc.lib().cure_margins_noalloc_scratch_bytes() == 256 * 1024
    for i, kw in enumerate(cases):
        say("noalloc margins call", i, kw["batch"], kw["vocab"])
        w, logits = _case("na%d" % i, **kw)
        args = dict(chain_len=w.chain_len, tau=w.tau, repair_budget=w.repair_budget,
                    branch_depth=w.branch_depth)
        got = pc.cure_margins_noalloc(logits, **args)
        torch.cuda.synchronize()
        ref = pc.cure_margins(logits, **args)
        torch.cuda.synchronize()
        _same(got, ref)
        check_margins(w, got)


def test_noalloc_unsplit_rows_and_no_gate():
    # Rows that are not split (no scratch needed), fp32, without the gate, then
    # a split call again.
    for i, kw in enumerate([
            dict(dtype="f32", batch=8, hq=4, hkv=1, d=64, vocab=3000, ctx_lens=[4] * 8,
                 chain_len=8, n_ufp=2, branch_depth=2, seed=33),
            dict(dtype="bf16", batch=1, hq=4, hkv=1, d=64, vocab=262147, ctx_lens=[4],
                 chain_len=3, n_ufp=1, branch_depth=1, seed=34)]):
        say("noalloc margins no-gate call", i)
        w, logits = _case("nb%d" % i, **kw)
        got = pc.cure_margins_noalloc(logits, gate=False)
        ref = pc.cure_margins(logits, gate=False)
        torch.cuda.synchronize()
        _same(got, ref)
        check_margins(w, got)
