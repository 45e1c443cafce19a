"""GPU parity: cure_tree_attn against the float64 oracle on the same input bytes.

Covers the fp32 vector-ALU path, the bf16 MFMA path and the bf16 vector-ALU
path; forced split counts (split-count invariance through the LSE merge);
ragged batches; context lengths around tile boundaries; single-node, empty
context and 256-node trees; row blocking beyond one workgroup; head dim 64;
malformed trees; and the full-size long-context workload on sampled nodes.
"""

import ctypes

import numpy as np
import pytest
import torch

import paper_2608_00531_amd as pc
from synth import preset, make_workload, bf16_round
from parity_util import say, upload, gpu_attn, oracle_attn, check_attn, Timer, LSE_TOL

pytestmark = pytest.mark.gpu


def test_tiny_fp32_valu():
    say("attn tiny_fp32")
    w = preset("tiny_fp32")
    dev = upload(w)
    o, lse, st = gpu_attn(w, dev)
    torch.cuda.synchronize()
    assert st.tolist() == [pc.CURE_OK]
    ref_o, ref_l = oracle_attn(w)
    check_attn(w, o, lse, ref_o, ref_l)


@pytest.mark.parametrize("out", ["bf16", "f32"])
@pytest.mark.parametrize("flags", [0, pc.CURE_ATTN_FORCE_VALU])
def test_llama_ctx2k_b1(out, flags):
    say("attn llama3_8b_ctx2k_b1 out", out, "flags", flags)
    w = preset("llama3_8b_ctx2k_b1")
    dev = upload(w)
    o, lse, st = gpu_attn(w, dev, out_dtype=torch.bfloat16 if out == "bf16" else torch.float32,
                          flags=flags)
    torch.cuda.synchronize()
    assert st.tolist() == [pc.CURE_OK]
    ref_o, ref_l = oracle_attn(w)
    check_attn(w, o, lse, ref_o, ref_l)


@pytest.mark.parametrize("kv_split", [1, 2, 7, 33])
def test_split_count_invariance(kv_split):
    say("attn split", kv_split)
    w = make_workload("s", batch=2, ctx_lens=[1000, 2113], chain_len=8, n_ufp=2,
                      branch_depth=3, seed=61)
    dev = upload(w)
    o, lse, st = gpu_attn(w, dev, out_dtype=torch.float32, kv_split=kv_split)
    ref_o, ref_l = oracle_attn(w)
    check_attn(w, o, lse, ref_o, ref_l)
    # Against the single-split result: splitting changes only where the bf16
    # rounding of the probabilities (and of their row sums, which are taken on
    # the rounded values the MFMA consumes) happens, so the two agree to the
    # bf16 bars the oracle comparison uses.
    o1, l1, _ = gpu_attn(w, dev, out_dtype=torch.float32, kv_split=1)
    torch.cuda.synchronize()
    assert float((o - o1).abs().max()) < 2e-3
    assert float((lse - l1).abs().max()) < LSE_TOL["bf16"]


@pytest.mark.parametrize("ctx", [0, 1, 63, 64, 65, 127, 128, 700])
def test_context_lengths_around_tiles(ctx):
    say("attn ctx", ctx)
    w = make_workload("c", batch=1, hq=8, hkv=2, d=128, ctx_lens=[ctx], chain_len=6, n_ufp=2,
                      branch_depth=2, seed=70 + ctx)
    dev = upload(w)
    for flags in (0, pc.CURE_ATTN_FORCE_VALU):
        o, lse, st = gpu_attn(w, dev, flags=flags)
        torch.cuda.synchronize()
        ref_o, ref_l = oracle_attn(w)
        check_attn(w, o, lse, ref_o, ref_l)


def test_ragged_nodes_and_contexts():
    say("attn ragged")
    w = make_workload("r", batch=6, ctx_lens=[300, 0, 1500, 64, 999, 50], chain_len=16,
                      n_ufp=4, branch_depth=4, seed=81)
    w.n_nodes[:] = [32, 1, 20, 32, 17, 0]            # prefixes of each tree are trees too
    # Rebuild the cache layout for the shorter trees (rows past n_nodes are dropped).
    rows = w.ctx_len + w.n_nodes
    off = np.concatenate([[0], np.cumsum(rows)[:-1]]).astype(np.int64)
    k = np.concatenate([w.k[w.kv_off[b]: w.kv_off[b] + rows[b]] for b in range(w.batch)])
    v = np.concatenate([w.v[w.kv_off[b]: w.kv_off[b] + rows[b]] for b in range(w.batch)])
    w.kv_off, w.k, w.v, w.kv_rows = off, k, v, int(rows.sum())
    dev = upload(w)
    for flags in (0, pc.CURE_ATTN_FORCE_VALU):
        o, lse, st = gpu_attn(w, dev, flags=flags)
        torch.cuda.synchronize()
        assert st.tolist() == [pc.CURE_OK] * w.batch     # an empty tree is a valid tree
        ref_o, ref_l = oracle_attn(w)
        check_attn(w, o, lse, ref_o, ref_l)


def _trim_trees(w, n_nodes):
    # Keep each tree's first n_nodes[b] nodes (prefixes of a topological order
    # are trees too) and rebuild the packed cache rows for the shorter trees.
    w.n_nodes[:] = n_nodes
    rows = w.ctx_len + w.n_nodes
    off = np.concatenate([[0], np.cumsum(rows)[:-1]]).astype(np.int64)
    k = np.concatenate([w.k[w.kv_off[b]: w.kv_off[b] + rows[b]] for b in range(w.batch)])
    v = np.concatenate([w.v[w.kv_off[b]: w.kv_off[b] + rows[b]] for b in range(w.batch)])
    w.kv_off, w.k, w.v, w.kv_rows = off, k, v, int(rows.sum())


def test_row_blocks_over_ragged_trees():
    # 80-node trees at group 4 (320 rows: one block of seven 48-row waves)
    # trimmed per sequence: 160 rows (waves past the tree have nothing to do),
    # 68 rows, an empty tree and an empty context.
    say("attn row blocks ragged")
    w = make_workload("rb", batch=5, ctx_lens=[500, 1200, 30, 0, 2000], chain_len=16,
                      n_ufp=16, branch_depth=4, seed=83)
    _trim_trees(w, [80, 40, 0, 17, 80])
    dev = upload(w)
    for kv_split in (0, 3):
        o, lse, st = gpu_attn(w, dev, kv_split=kv_split)
        torch.cuda.synchronize()
        assert st.tolist() == [pc.CURE_OK] * w.batch
        ref_o, ref_l = oracle_attn(w)
        check_attn(w, o, lse, ref_o, ref_l)


def _seg_batch(seed=87):
    # Twenty sequences of very different lengths, with an empty context,
    # contexts shorter than a tile, empty trees in the middle and at the end
    # and a one-node tree: a launch whose splits are limited by the workgroups
    # the GPU holds at once, so most sequences get splits of different counts
    # and the last split of each is short.
    rng = np.random.default_rng(5)
    ctx = [int(x) for x in rng.integers(0, 4000, 20)]
    ctx[3], ctx[7], ctx[11] = 0, 5, 63
    nn = [8] * 20
    nn[5], nn[19], nn[12] = 0, 0, 1
    w = make_workload("seg", batch=20, ctx_lens=ctx, chain_len=8, n_ufp=0, branch_depth=1,
                      seed=seed)
    _trim_trees(w, nn)
    return w


def test_split_limited_ragged_batch():
    say("attn split-limited ragged batch")
    w = _seg_batch()
    dev = upload(w)
    ref_o, ref_l = oracle_attn(w)
    for kv_split in (0, 5):                     # planned splits, then 5 forced
        o, lse, st = gpu_attn(w, dev, kv_split=kv_split)
        torch.cuda.synchronize()
        assert st.tolist() == [pc.CURE_OK] * w.batch
        check_attn(w, o, lse, ref_o, ref_l)


def test_split_limited_batch_reports_a_malformed_tree():
    say("attn split-limited ragged batch, malformed tree")
    w = _seg_batch(seed=88)
    w.parent[8, 3] = 5                           # a parent after its child
    dev = upload(w)
    o, lse, st = gpu_attn(w, dev)
    torch.cuda.synchronize()
    want = [pc.CURE_OK] * w.batch
    want[8] = pc.CURE_ERR_BAD_TREE
    assert st.tolist() == want
    keep = [(b, n) for b in range(w.batch) if b != 8 for n in range(int(w.n_nodes[b]))]
    ref_o, ref_l = oracle_attn(w, sample=keep)
    check_attn(w, o, lse, ref_o, ref_l, sample=keep)


def test_no_tree_nodes_anywhere_reports_every_tree_valid():
    # A launch in which no sequence has tree nodes computes nothing, yet every
    # sequence's (empty) tree is valid and its status must say so.
    say("attn no tree nodes")
    w = make_workload("empty", batch=3, ctx_lens=[100, 0, 70], chain_len=4, n_ufp=0,
                      branch_depth=1, seed=95)
    _trim_trees(w, [0, 0, 0])
    dev = upload(w)
    L = pc.lib()
    ptr = lambda t: ctypes.c_void_p(t.data_ptr()) if t is not None else None
    hc = np.ascontiguousarray(w.ctx_len, np.int32)
    hn = np.ascontiguousarray(w.n_nodes, np.int32)
    o = torch.empty(w.batch, w.n_max, w.hq, w.d, dtype=torch.bfloat16, device="cuda")
    for flags, n_max in ((0, w.n_max), (pc.CURE_ATTN_FORCE_VALU, w.n_max), (0, 0)):
        status = torch.full((w.batch,), -7, dtype=torch.int32, device="cuda")
        st = L.cure_tree_attn(ptr(dev["q"]), ptr(dev["k"]), ptr(dev["v"]), ptr(o), None,
                              pc.CURE_BF16, pc.CURE_BF16, w.batch, w.hq, w.hkv, w.d, w.scale,
                              ptr(dev["kv_off"]), ptr(dev["ctx_len"]), ptr(dev["n_nodes"]),
                              ptr(dev["parent"]), n_max, hc.ctypes.data_as(ctypes.c_void_p),
                              hn.ctypes.data_as(ctypes.c_void_p), 0, flags, ptr(status), None, 0,
                              ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
        torch.cuda.synchronize()
        assert st == pc.CURE_OK
        assert status.tolist() == [pc.CURE_OK] * w.batch, (flags, n_max)


def test_largest_tree_with_gqa():
    # 256 nodes (the maximum) at group 4: 1024 rows per kv-head, four 256-row blocks.
    say("attn 256 nodes x group 4")
    w = make_workload("g", batch=1, hq=16, hkv=4, ctx_lens=[333], chain_len=16, n_ufp=15,
                      branch_depth=16, seed=84, vocab=64)
    assert int(w.n_nodes[0]) == 256
    dev = upload(w)
    o, lse, st = gpu_attn(w, dev)
    torch.cuda.synchronize()
    assert st.tolist() == [pc.CURE_OK]
    ref_o, ref_l = oracle_attn(w)
    check_attn(w, o, lse, ref_o, ref_l)


@pytest.mark.parametrize("hq,hkv,d,n_ufp,depth", [(32, 8, 128, 16, 4), (8, 8, 128, 16, 15),
                                                  (4, 1, 128, 8, 4), (4, 1, 64, 8, 4),
                                                  (32, 8, 128, 2, 4), (64, 8, 128, 8, 4),
                                                  (32, 4, 128, 15, 5), (32, 8, 64, 4, 4)])
def test_row_blocking_and_wide_trees(hq, hkv, d, n_ufp, depth):
    # Rows per kv-head = nodes x group:
    # (32,8,128,16,4): 80 x 4 = 320 -> one block of the 48-row-per-wave kernel;
    # (8,8,128,16,15): 256 nodes (the maximum), G1 -> 16-row kernel, 16 waves;
    # (4,1,128,8,4): 48 x 4 = 192 -> 16-row kernel, 12 of 16 waves;
    # (4,1,64,8,4): 192 rows at head dim 64 -> 32-row kernel;
    # (32,8,128,2,4): 24 x 4 = 96 -> 16-row kernel, 6 of 8 waves;
    # (64,8,128,8,4): 48 x 8 = 384 -> two 192-row blocks;
    # (32,4,128,15,5): 91 x 8 = 728 -> three 256-row blocks, the last with 216
    #   rows (its 14th wave half full); hkv 4, so the blocks sit on different XCDs;
    # (32,8,64,4,4): 32 x 4 = 128 rows at head dim 64 -> 16-row kernel.
    say("attn rows", hq, hkv, d, n_ufp, depth)
    w = make_workload("w", batch=1, hq=hq, hkv=hkv, d=d, ctx_lens=[777], chain_len=16,
                      n_ufp=n_ufp, branch_depth=depth, seed=90)
    dev = upload(w)
    for flags in (0, pc.CURE_ATTN_FORCE_VALU):
        o, lse, st = gpu_attn(w, dev, flags=flags)
        torch.cuda.synchronize()
        ref_o, ref_l = oracle_attn(w)
        check_attn(w, o, lse, ref_o, ref_l)


@pytest.mark.parametrize("hq,hkv,n_ufp,depth,ctx,kv_split", [
    (16, 4, 12, 5, [300, 64], 0), (16, 4, 4, 17, [1000, 0], 0), (16, 4, 12, 5, [129, 2500], 3),
    (16, 4, 7, 7, [63, 700], 0), (16, 4, 13, 4, [640, 97], 0), (16, 4, 14, 4, [65, 1300], 0),
    (16, 4, 16, 4, [900, 200], 2), (32, 4, 6, 3, [500, 64], 0), (8, 4, 2, 67, [260, 31], 0),
    (16, 4, 12, 6, [2000, 65], 5), (16, 4, 16, 5, [333, 1111], 0), (16, 4, 12, 7, [129, 64], 0)])
def test_three_row_group_kernel(hq, hkv, n_ufp, depth, ctx, kv_split):
    # 257 - 384 rows per kv-head take the kernel whose waves own two or three
    # 16-row groups (waves with three come first). Group 4: 76 nodes (304
    # rows, 19 row groups: three waves of three), 84 (336: five), 76 with
    # forced splits, 65 (260 rows, just past 256: one), 68 (272: one), 72
    # (288: two), 80 (320: four, every SIMD even) with forced splits, 88 (352:
    # six) with forced splits, 96 (384, the block's capacity: all eight);
    # group 8 at 34 nodes (272 rows) and group 2 at 150 nodes (300 rows); and
    # 100 nodes (400 rows: the 16-row kernel in two blocks) as a neighbour.
    # The second tree is trimmed by 7 nodes so a wave's row groups end
    # mid-node and some waves own no rows.
    say("attn 48-row waves", hq, hkv, n_ufp, depth, ctx, kv_split)
    w = make_workload("r3", batch=2, hq=hq, hkv=hkv, ctx_lens=ctx, chain_len=16, n_ufp=n_ufp,
                      branch_depth=depth, seed=300 + n_ufp * 7 + depth)
    n_tree = int(w.n_nodes[0])
    _trim_trees(w, [n_tree, n_tree - 7])
    dev = upload(w)
    ref_o, ref_l = oracle_attn(w)
    for flags in (0, pc.CURE_ATTN_FORCE_VALU):
        o, lse, st = gpu_attn(w, dev, flags=flags, kv_split=kv_split)
        torch.cuda.synchronize()
        assert st.tolist() == [pc.CURE_OK] * w.batch
        check_attn(w, o, lse, ref_o, ref_l)


@pytest.mark.parametrize("kv_split", [0, 3, 60])
def test_head_dim_64_bf16(kv_split):
    # 60 requested splits give 42 (64-token splits) on the long sequence: more
    # than one batch of merge loads at D = 64.
    say("attn d64 kv_split", kv_split)
    w = make_workload("d", batch=2, hq=16, hkv=4, d=64, ctx_lens=[400, 2600], chain_len=12,
                      n_ufp=3, branch_depth=2, seed=99)
    dev = upload(w)
    ref_o, ref_l = oracle_attn(w)
    for flags in (0, pc.CURE_ATTN_FORCE_VALU):
        o, lse, st = gpu_attn(w, dev, flags=flags, kv_split=kv_split)
        torch.cuda.synchronize()
        check_attn(w, o, lse, ref_o, ref_l)


def test_malformed_tree_status():
    say("attn malformed tree")
    w = make_workload("m", batch=2, hq=8, hkv=2, ctx_lens=[100, 100], chain_len=6, n_ufp=1,
                      branch_depth=2, seed=3)
    w.parent[0, 4] = 6                                # parent index after the node
    dev = upload(w)
    for flags in (0, pc.CURE_ATTN_FORCE_VALU):
        o, lse, st = gpu_attn(w, dev, flags=flags)
        torch.cuda.synchronize()
        assert st.tolist() == [pc.CURE_ERR_BAD_TREE, pc.CURE_OK]
        ok = make_workload("m", batch=2, hq=8, hkv=2, ctx_lens=[100, 100], chain_len=6,
                           n_ufp=1, branch_depth=2, seed=3)
        ref_o, ref_l = oracle_attn(ok, sample=[(1, n) for n in range(int(ok.n_nodes[1]))])
        check_attn(ok, o, lse, ref_o, ref_l, sample=[(1, n) for n in range(int(ok.n_nodes[1]))])


def test_ragged_batch16_full_size():
    say("attn llama3_8b_ragged_b16 full")
    with Timer("generate"):
        w = preset("llama3_8b_ragged_b16")
    dev = upload(w)
    o, lse, st = gpu_attn(w, dev)
    torch.cuda.synchronize()
    assert st.tolist() == [pc.CURE_OK] * w.batch
    with Timer("oracle"):
        ref_o, ref_l = oracle_attn(w)
    check_attn(w, o, lse, ref_o, ref_l)


def test_long_context_full_size_sampled():
    say("attn llama3_8b_ctx32k_b4 sampled")
    with Timer("generate"):
        w = preset("llama3_8b_ctx32k_b4")
    dev = upload(w)
    o, lse, st = gpu_attn(w, dev)
    torch.cuda.synchronize()
    assert st.tolist() == [pc.CURE_OK] * w.batch
    rng = np.random.default_rng(0)
    sample = [(b, int(n)) for b in range(w.batch) for n in rng.choice(32, 3, replace=False)]
    sample += [(0, 0), (3, 31), (2, 16)]
    with Timer("oracle"):
        ref_o, ref_l = oracle_attn(w, sample=sample)
    check_attn(w, o, lse, ref_o, ref_l, sample=sample)


@pytest.mark.parametrize("kv_split", [0, 2])
def test_more_workgroups_than_cus_sampled(kv_split):
    # 64 sequences x 8 kv-heads of 32-node trees (128 rows): 512 workgroups of
    # the 8-wave 16-row kernel at the planned single split (1024 at two splits,
    # then merged), more than the CUs, so two of them share a CU.
    say("attn 64 sequences, more workgroups than CUs, kv_split", kv_split)
    rng = np.random.default_rng(12)
    ctx = [int(x) for x in rng.integers(1, 1600, 64)]
    w = make_workload("wide", batch=64, ctx_lens=ctx, chain_len=16, n_ufp=4, branch_depth=4,
                      seed=13)
    dev = upload(w)
    o, lse, st = gpu_attn(w, dev, kv_split=kv_split)
    torch.cuda.synchronize()
    assert st.tolist() == [pc.CURE_OK] * w.batch
    sample = [(b, int(n)) for b in range(w.batch) for n in rng.choice(32, 2, replace=False)]
    sample += [(0, 0), (63, 31)]
    with Timer("oracle"):
        ref_o, ref_l = oracle_attn(w, sample=sample)
    check_attn(w, o, lse, ref_o, ref_l, sample=sample)


def test_largest_sweep_tree_full_size_sampled():
    # Batch 8, context 8192, 80 nodes: 320 rows per kv-head, one block of seven
    # 48-row waves, in the launch configuration the budget sweep times.
    say("attn llama3_8b_ctx8k_b8_budget64 sampled")
    with Timer("generate"):
        w = preset("llama3_8b_ctx8k_b8_budget64")
    dev = upload(w)
    o, lse, st = gpu_attn(w, dev)
    torch.cuda.synchronize()
    assert st.tolist() == [pc.CURE_OK] * w.batch
    rng = np.random.default_rng(1)
    sample = [(b, int(n)) for b in range(w.batch) for n in rng.choice(80, 2, replace=False)]
    # Chain ends, nodes whose rows straddle the waves' row groups (row 256+ is
    # node 64+ with 4 query heads per kv-head) and the last node.
    sample += [(0, 0), (1, 15), (2, 63), (3, 64), (7, 79)]
    with Timer("oracle"):
        ref_o, ref_l = oracle_attn(w, sample=sample)
    check_attn(w, o, lse, ref_o, ref_l, sample=sample)


def test_nonpositive_scale_takes_the_general_path():
    say("attn negative scale")
    w = make_workload("n", batch=2, hq=8, hkv=2, ctx_lens=[300, 71], chain_len=8, n_ufp=2,
                      branch_depth=2, seed=44, scale=-0.05)
    dev = upload(w)
    o, lse, st = gpu_attn(w, dev)
    torch.cuda.synchronize()
    ref_o, ref_l = oracle_attn(w)
    check_attn(w, o, lse, ref_o, ref_l)


def _climbing_keys(w):
    """Keys whose scores climb along each sequence (a gain from 1 to 7) and two
    late context tokens 60 times stronger still: the running softmax
    reference has to move several times inside one split, and against the
    reference before them the spikes' probabilities (scores near 2^150 times
    the earlier maximum for some rows) overflow float32."""
    bf16 = w.dtype == "bf16"
    k = (w.k.astype(np.uint32) << np.uint32(16)).view(np.float32) if bf16 else w.k.copy()
    for b in range(w.batch):
        off, L = int(w.kv_off[b]), int(w.ctx_len[b]) + int(w.n_nodes[b])
        k[off:off + L] *= (1.0 + 6.0 * np.arange(L) / max(L - 1, 1)).astype(np.float32)[:, None, None]
        for frac in (0.55, 0.9):
            tok = int(frac * (int(w.ctx_len[b]) - 1))
            k[off + tok] *= np.float32(60.0)
    w.k = bf16_round(k) if bf16 else k


@pytest.mark.parametrize("case", ["rows128", "rows192", "rows320", "valu_bf16"])
@pytest.mark.parametrize("kv_split", [0, 1])
def test_softmax_reference_moves_and_spikes(case, kv_split):
    """The tiles' probabilities are taken against a running reference that
    moves only when a row's maximum rises by more than 2^8; the kernels check
    for that after the exponentials and redo a tile when it happens. Climbing
    scores and late spikes make it happen often, including probabilities that
    overflow before the redo, on the 16-row kernel (128 and 192 rows), the
    three-row-group kernel (320 rows) and the bf16 vector-ALU path, with the
    planned splits and with one split per sequence. (fp32 inputs of these
    magnitudes are left out: their scores, near 1e4 before scaling, carry
    fp32 rounding of a few 1e-4 themselves, beyond the absolute fp32 bars.)"""
    say("attn climbing scores", case, "kv_split", kv_split)
    n_ufp = {"rows192": 8, "rows320": 16}.get(case, 4)
    w = make_workload("c", batch=2,
                      ctx_lens=[1500, 3000], chain_len=16, n_ufp=n_ufp, branch_depth=4,
                      seed=71)
    _climbing_keys(w)
    dev = upload(w)
    flags = pc.CURE_ATTN_FORCE_VALU if case == "valu_bf16" else 0
    o, lse, st = gpu_attn(w, dev, kv_split=kv_split, flags=flags)
    torch.cuda.synchronize()
    assert st.tolist() == [pc.CURE_OK] * w.batch
    ref_o, ref_l = oracle_attn(w)
    check_attn(w, o, lse, ref_o, ref_l)


@pytest.mark.parametrize("seed", range(24))
def test_random_shapes(seed):
    # Seeded random shapes: batch, GQA ratio, head dim, chain and branch shapes,
    # ragged contexts (zero included), trees trimmed per sequence and forced
    # split counts, so row blocks, splits and tail tiles combine freely.
    rng = np.random.default_rng(1000 + seed)
    batch = int(rng.integers(1, 5))
    hkv = int(rng.choice([1, 2, 4, 8]))
    group = int(rng.choice([1, 2, 4, 8]))
    d = int(rng.choice([64, 128]))
    chain = int(rng.integers(1, 17))
    n_ufp = int(rng.integers(0, chain + 1))
    depth = int(rng.integers(1, 17))
    while chain + n_ufp * depth > 256:
        n_ufp -= 1
    ctx = [int(c) for c in rng.integers(0, 3000, size=batch)]
    kv_split = int(rng.choice([0, 0, 1, 2, 5]))
    say("attn random", seed, batch, hkv, group, d, chain, n_ufp, depth, ctx, kv_split)
    w = make_workload("rand", batch=batch, hq=hkv * group, hkv=hkv, d=d, ctx_lens=ctx,
                      chain_len=chain, n_ufp=n_ufp, branch_depth=depth, seed=2000 + seed,
                      vocab=64)
    n_tree = int(w.n_nodes[0])
    _trim_trees(w, [int(rng.integers(0, n_tree + 1)) if rng.random() < 0.5 else n_tree
                    for _ in range(batch)])
    dev = upload(w)
    o, lse, st = gpu_attn(w, dev, kv_split=kv_split)
    torch.cuda.synchronize()
    assert st.tolist() == [pc.CURE_OK] * w.batch
    ref_o, ref_l = oracle_attn(w)
    check_attn(w, o, lse, ref_o, ref_l)
