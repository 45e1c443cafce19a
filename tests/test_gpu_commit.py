"""GPU parity: cure_commit (Sec. 3.5, Algorithm 1) against the oracle, bit-exact.

The cache after the commit must equal the oracle's commit_kv byte for byte in
every layer (including rows and layer gaps the commit must not touch), and the
emitted tokens, new context length and replay start must equal commit_tokens.
Paths come from the oracle's acceptance walk, so these tests do not depend on
cure_accept.
"""

import json
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2608_00531_amd as pc
from synth import make_workload, preset
from parity_util import say

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _i32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()


def _i64(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int64)).cuda()


def _dev(a):
    """numpy cache (float32, or uint16 bf16 bits) -> cuda tensor of the same bytes."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(a).cuda()


def _host(t):
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def _padded_paths(paths, acc, n_max):
    out = np.full((len(paths), n_max), -1, np.int32)
    for b, p in enumerate(paths):
        a = max(int(acc[b]), 0)
        out[b, :a] = p[:a]
    return out


def _expected_cache(layers, kv_off, ctx_len, paths, acc, layer_rows):
    """Oracle commit of every layer; layers [L, rows_alloc, ...], of which the
    first layer_rows rows of each layer are the cache and the rest a gap."""
    exp = layers.copy()
    for l in range(layers.shape[0]):
        exp[l, :layer_rows] = oracle.commit_kv(layers[l, :layer_rows], kv_off, ctx_len, paths, acc)
    return exp


def _check_tokens(got, token, paths, acc, bonus, chain_len, ctx_len, n_max):
    for b in range(len(acc)):
        ref = oracle.commit_tokens(token[b], paths[b], int(acc[b]), int(bonus[b]), chain_len)
        e = got["emit"][b].tolist()
        k = len(ref["emit"])
        assert e[:k] == ref["emit"], b
        assert all(x == -1 for x in e[k:]), b
        assert len(e) == n_max + 1
        assert int(got["emit_cnt"][b]) == k
        assert int(got["replay_start"][b]) == ref["replay_start"], b
        assert int(got["new_ctx_len"][b]) == int(ctx_len[b]) + ref["new_ctx_add"]


def _run(k, v, w_kv_off, ctx_len, n_nodes, paths_np, acc, token, bonus, chain_len,
         layer_stride=None):
    return pc.cure_commit(k, v, _i64(w_kv_off), _i32(ctx_len), _i32(n_nodes), _i32(paths_np),
                          _i32(acc), _i32(token), _i32(bonus), chain_len,
                          layer_stride=layer_stride)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_worked_commits(dtype):
    say("commit worked", dtype)
    with open(os.path.join(GOLDEN, "commit_worked.json")) as f:
        g = json.load(f)
    n_max = 8
    rows = 22
    # Row r of layer l holds r, -r, 100 l + r, ... so every moved row is
    # recognisable; hkv = 2, d = 4 (32 B rows in f32, 16 B in bf16).
    base = np.array([[[r, -r, 100 * l + r, 7] * 2 for r in range(rows)] for l in range(3)],
                    np.float32).reshape(3, rows, 2, 4)
    if dtype == "bf16":
        base = (base.view(np.uint32) >> 16).astype(np.uint16)   # small integers: exact in bf16
    paths = _padded_paths(g["path"], g["acc_len"], n_max)
    token = np.full((4, n_max), -7, np.int32)
    for b, t in enumerate(g["token"]):
        token[b, :len(t)] = t
    # One chain_len per call and the fixture's sequences have different ones,
    # so each sequence is committed by its own call with the others marked
    # uncommittable (acc_len = -1).
    for b in range(4):
        kb = _dev(base)
        vb = _dev(base[:, :, ::-1].copy())
        acc = np.array(g["acc_len"], np.int32)
        acc_b = np.where(np.arange(4) == b, acc, -1).astype(np.int32)
        got = _run(kb, vb, g["kv_off"], g["ctx_len"], g["n_nodes"], paths, acc_b, token,
                   g["bonus"], g["chain_len"][b])
        case = g["cases"][b]
        lo = g["kv_off"][b]
        hi = lo + g["ctx_len"][b] + g["n_nodes"][b]
        kk = _host(kb)
        for l in range(3):
            col0 = kk[l, lo:hi, 0, 0]
            if dtype == "bf16":
                col0 = (col0.astype(np.uint32) << 16).view(np.float32)
            assert col0.tolist() == case["rows_after"][0], case["why"]
        exp = _expected_cache(base, g["kv_off"], g["ctx_len"], paths, acc_b, rows)
        assert np.array_equal(kk, exp)
        assert np.array_equal(_host(vb), _expected_cache(base[:, :, ::-1].copy(), g["kv_off"],
                                                         g["ctx_len"], paths, acc_b, rows))
        e = got["emit"][b].tolist()
        assert e[:len(case["emit"])] == case["emit"], case["why"]
        assert int(got["replay_start"][b]) == case["replay_start"]
        assert int(got["new_ctx_len"][b]) == g["ctx_len"][b] + case["new_ctx_add"]
        want = pc.CURE_OK if g["acc_len"][b] >= 0 else pc.CURE_ERR_BAD_TREE
        assert int(got["status"][b]) == want


def _accept_all(w, tgt=None):
    tgt = w.tgt_planted if tgt is None else tgt
    return [oracle.accept(w.parent[b], w.token[b], tgt[b], int(w.root_tgt[b]),
                          int(w.n_nodes[b]), w.chain_len) for b in range(w.batch)]


@pytest.mark.parametrize("dtype,hkv,d,layers,gap,seed", [
    ("f32", 2, 48, 7, 5, 1),       # 384-byte rows: 48 columns per layer, a ragged last workgroup
    ("bf16", 8, 128, 3, 0, 2),     # Llama-3-8B row shape, layers back to back
    ("bf16", 1, 8, 5, 3, 11),      # 16-byte rows
    ("f32", 4, 64, 2, 17, 4),      # the chain wins everywhere: nothing moves
])
def test_random_workloads_every_layer(dtype, hkv, d, layers, gap, seed):
    say("commit random", dtype, hkv, d, layers, gap, seed)
    w = make_workload("commit", dtype=dtype, batch=6, hq=hkv, hkv=hkv, d=d, vocab=64,
                      ctx_lens=[5, 0, 33, 1, 64, 2], chain_len=8, n_ufp=3, branch_depth=3,
                      seed=seed, p_agree=0.9)
    acc_res = _accept_all(w)
    acc = np.array([r["acc_len"] for r in acc_res], np.int32)
    bonus = np.array([r["bonus"] for r in acc_res], np.int32)
    paths = _padded_paths([r["path"] for r in acc_res], acc, w.n_max)
    rng = np.random.default_rng(seed)
    rows = w.kv_rows
    shape = (layers, rows + gap, hkv, d)
    if dtype == "f32":
        cache_k = rng.standard_normal(shape, dtype=np.float32)
        cache_v = rng.standard_normal(shape, dtype=np.float32)
    else:
        cache_k = rng.integers(0, 1 << 16, shape, dtype=np.uint16)
        cache_v = rng.integers(0, 1 << 16, shape, dtype=np.uint16)
    k, v = _dev(cache_k), _dev(cache_v)
    got = _run(k, v, w.kv_off, w.ctx_len, w.n_nodes, paths, acc, w.token, bonus, w.chain_len)
    assert got["status"].tolist() == [pc.CURE_OK] * w.batch
    assert np.array_equal(_host(k), _expected_cache(cache_k, w.kv_off, w.ctx_len, paths, acc, rows))
    assert np.array_equal(_host(v), _expected_cache(cache_v, w.kv_off, w.ctx_len, paths, acc, rows))
    _check_tokens(got, w.token, paths, acc, bonus, w.chain_len, w.ctx_len, w.n_max)
    assert any(r["resync"] for r in acc_res) or seed == 4


def test_deep_paths_span_several_row_groups():
    # Trees of up to 256 nodes whose winning paths run 20-150 deep, so the rows
    # move in several groups and the first moved row falls inside a group.
    say("commit deep paths")
    rng = np.random.default_rng(91)
    B, n_max, chain = 12, 256, 24
    parent = np.full((B, n_max), -1, np.int32)
    n_nodes = rng.integers(40, n_max + 1, B).astype(np.int32)
    n_nodes[:2] = [256, 255]
    for b in range(B):
        for n in range(1, int(n_nodes[b])):
            parent[b, n] = n - 1 if n < chain else int(rng.integers(max(-1, n - 3), n))
    token = rng.integers(0, 1000, (B, n_max)).astype(np.int32)
    # Target that agrees with every node: the deepest node wins (lowest index on ties).
    tgt = np.zeros((B, n_max), np.int32)
    root = np.zeros(B, np.int32)
    acc, bonus, paths = [], [], []
    for b in range(B):
        kids = {}
        for n in range(int(n_nodes[b])):
            kids.setdefault(int(parent[b, n]), []).append(n)
        for p_, ks in kids.items():
            for c in ks:          # every child's token equals its parent's prediction
                token[b, c] = 5
            if p_ < 0:
                root[b] = 5
            else:
                tgt[b, p_] = 5
        r = oracle.accept(parent[b], token[b], tgt[b], int(root[b]), int(n_nodes[b]), chain)
        acc.append(r["acc_len"])
        bonus.append(r["bonus"])
        paths.append(r["path"])
        token[b, :int(n_nodes[b])] = rng.integers(0, 1000, int(n_nodes[b]))
    acc = np.array(acc, np.int32)
    assert acc.min() > 16 and (acc > 48).any()
    paths = _padded_paths(paths, acc, n_max)
    ctx = rng.integers(0, 50, B).astype(np.int32)
    kv_off = np.concatenate([[0], np.cumsum(ctx + n_nodes)[:-1]]).astype(np.int64)
    rows = int((ctx + n_nodes).sum())
    cache_k = rng.standard_normal((2, rows, 1, 4), dtype=np.float32)
    cache_v = rng.standard_normal((2, rows, 1, 4), dtype=np.float32)
    k, v = _dev(cache_k), _dev(cache_v)
    got = _run(k, v, kv_off, ctx, n_nodes, paths, acc, token, bonus, chain)
    assert got["status"].tolist() == [pc.CURE_OK] * B
    assert np.array_equal(_host(k), _expected_cache(cache_k, kv_off, ctx, paths, acc, rows))
    assert np.array_equal(_host(v), _expected_cache(cache_v, kv_off, ctx, paths, acc, rows))
    _check_tokens(got, token, paths, acc, bonus, chain, ctx, n_max)


def test_uncommittable_sequences_are_left_untouched():
    say("commit uncommittable")
    n_max = 6
    # Each sequence: ctx 2, 6 nodes (chain 0-3, branch 4-5 off node 1).
    cases = [
        (4, [0, 1, 4, 5], pc.CURE_OK),          # a repair branch wins
        (-1, [], pc.CURE_ERR_BAD_TREE),         # cure_accept's mark of a malformed tree
        (7, [0, 1, 2, 3, 4, 5], pc.CURE_ERR_BAD_TREE),   # acc_len > n_nodes
        (3, [0, 6, 7], pc.CURE_ERR_BAD_TREE),   # entries past n_nodes
        (3, [0, 2, 2], pc.CURE_ERR_BAD_TREE),   # not increasing
        (2, [1, 0], pc.CURE_ERR_BAD_TREE),      # decreasing
        (1, [-1], pc.CURE_ERR_BAD_TREE),        # negative entry
        (0, [], pc.CURE_OK),                    # nothing accepted
        (4, [0, 1, 2, 3], pc.CURE_OK),          # the chain wins: nothing moves
    ]
    B = len(cases)
    acc = np.array([c[0] for c in cases], np.int32)
    paths = np.full((B, n_max), -1, np.int32)
    for b, c in enumerate(cases):
        paths[b, :len(c[1])] = c[1][:n_max]
    ctx = np.full(B, 2, np.int32)
    n_nodes = np.full(B, 6, np.int32)
    kv_off = (np.arange(B) * 8).astype(np.int64)
    token = np.arange(B * n_max, dtype=np.int32).reshape(B, n_max) + 100
    bonus = np.arange(B, dtype=np.int32) + 900
    rng = np.random.default_rng(5)
    cache = rng.standard_normal((B * 8, 2, 8), dtype=np.float32)
    k, v = _dev(cache), _dev(cache[::-1].copy())
    got = _run(k, v, kv_off, ctx, n_nodes, paths, acc, token, bonus, 4)
    kk = _host(k)
    for b, (a, p, want) in enumerate(cases):
        assert int(got["status"][b]) == want, b
        lo, hi = b * 8, b * 8 + 8
        if want == pc.CURE_OK:
            exp = oracle.commit_kv(cache[lo:hi], [0], [2], [paths[b]], [a])
            assert np.array_equal(kk[lo:hi], exp), b
            ref = oracle.commit_tokens(token[b], paths[b], a, bonus[b], 4)
            assert got["emit"][b].tolist()[:a + 1] == ref["emit"]
            assert int(got["replay_start"][b]) == ref["replay_start"]
            assert int(got["new_ctx_len"][b]) == 2 + a
        else:
            assert np.array_equal(kk[lo:hi], cache[lo:hi]), b
            assert got["emit"][b].tolist() == [-1] * (n_max + 1)
            assert int(got["emit_cnt"][b]) == 0 and int(got["replay_start"][b]) == 0
            assert int(got["new_ctx_len"][b]) == 2
    ok = np.array([c[2] == pc.CURE_OK for c in cases])
    exp_v = oracle.commit_kv(cache[::-1].copy(), kv_off, ctx, paths, np.where(ok, acc, -1))
    assert np.array_equal(_host(v), exp_v)


def test_tokens_only_when_no_layers():
    say("commit no layers")
    w = make_workload("commit", dtype="bf16", batch=3, hq=8, hkv=8, d=128, vocab=64,
                      ctx_lens=[4, 4, 4], chain_len=6, n_ufp=2, branch_depth=2, seed=9,
                      p_agree=0.9)
    acc_res = _accept_all(w)
    acc = np.array([r["acc_len"] for r in acc_res], np.int32)
    bonus = np.array([r["bonus"] for r in acc_res], np.int32)
    paths = _padded_paths([r["path"] for r in acc_res], acc, w.n_max)
    empty = torch.empty(0, w.kv_rows, 8, 128, dtype=torch.bfloat16, device="cuda")
    got = _run(empty, empty.clone(), w.kv_off, w.ctx_len, w.n_nodes, paths, acc, w.token, bonus,
               w.chain_len)
    _check_tokens(got, w.token, paths, acc, bonus, w.chain_len, w.ctx_len, w.n_max)


def test_full_size_llama3_8b_32_layers():
    # The benchmark's configuration: the default workload's tree, a 32-layer
    # cache of Llama-3-8B rows (8 KV heads x 128, bf16), a winning path that runs
    # through the last repair branch. Sampled layers are checked against the
    # oracle; every layer is checked against the moved-rows property on the GPU.
    say("commit full size 32 layers")
    w = preset("llama3_8b_ctx2k_b1")
    L = 32
    leaf = int(w.n_nodes[0]) - 1
    chain_path = []
    n = leaf
    while n >= 0:
        chain_path.append(n)
        n = int(w.parent[0][n])
    chain_path.reverse()
    a = len(chain_path)
    acc = np.array([a], np.int32)
    paths = _padded_paths([chain_path], acc, w.n_max)
    bonus = np.array([7], np.int32)
    g = torch.Generator(device="cuda")
    g.manual_seed(11)
    shape = (L, w.kv_rows, w.hkv, w.d)
    k = torch.randn(shape, device="cuda", dtype=torch.float32, generator=g).to(torch.bfloat16)
    v = torch.randn(shape, device="cuda", dtype=torch.float32, generator=g).to(torch.bfloat16)
    k0, v0 = k.clone(), v.clone()
    got = _run(k, v, w.kv_off, w.ctx_len, w.n_nodes, paths, acc, w.token, bonus, w.chain_len)
    torch.cuda.synchronize()
    assert int(got["status"][0]) == pc.CURE_OK
    base = int(w.ctx_len[0])
    idx = torch.tensor([base + p for p in chain_path], device="cuda")
    for t, t0 in ((k, k0), (v, v0)):
        assert torch.equal(t[:, base:base + a], t0[:, idx])
        assert torch.equal(t[:, :base], t0[:, :base])
        assert torch.equal(t[:, base + a:], t0[:, base + a:])
    for l in (0, 17, 31):
        exp = oracle.commit_kv(_host(k0[l]), w.kv_off, w.ctx_len, paths, acc)
        assert np.array_equal(_host(k[l]), exp)
    _check_tokens(got, w.token, paths, acc, bonus, w.chain_len, w.ctx_len, w.n_max)
    assert int(got["replay_start"][0]) < a


@pytest.mark.parametrize("seed", range(16))
def test_random_shapes(seed):
    # Seeded random commits: batch, kv heads, head dim, dtype, layers, a gap
    # between layers, chain and branch shapes, contexts and how often the target
    # agrees with the draft (which sets how deep the winning paths run).
    rng = np.random.default_rng(8000 + seed)
    batch = int(rng.integers(1, 9))
    hkv = int(rng.choice([1, 2, 4, 8]))
    d = int(rng.choice([8, 32, 64, 128]))
    dtype = "bf16" if rng.random() < 0.6 else "f32"
    layers = int(rng.integers(1, 5))
    gap = int(rng.integers(0, 20))
    chain = int(rng.integers(1, 17))
    n_ufp = int(rng.integers(0, chain + 1))
    depth = int(rng.integers(1, 9))
    while chain + n_ufp * depth > 256:
        n_ufp -= 1
    ctx = [int(c) for c in rng.integers(0, 300, size=batch)]
    say("commit random shapes", seed, batch, hkv, d, dtype, layers, gap, chain, n_ufp, depth)
    w = make_workload("c", dtype=dtype, batch=batch, hq=hkv, hkv=hkv, d=d, vocab=16,
                      ctx_lens=ctx, chain_len=chain, n_ufp=n_ufp, branch_depth=depth,
                      seed=8100 + seed, p_agree=float(rng.choice([0.5, 0.8, 0.95, 1.0])))
    acc_res = _accept_all(w)
    acc = np.array([r["acc_len"] for r in acc_res], np.int32)
    bonus = np.array([r["bonus"] for r in acc_res], np.int32)
    paths = _padded_paths([r["path"] for r in acc_res], acc, w.n_max)
    rows = w.kv_rows
    shape = (layers, rows + gap, hkv, d)
    if dtype == "f32":
        ck = rng.standard_normal(shape, dtype=np.float32)
        cv = rng.standard_normal(shape, dtype=np.float32)
    else:
        ck = rng.integers(0, 1 << 16, shape, dtype=np.uint16)
        cv = rng.integers(0, 1 << 16, shape, dtype=np.uint16)
    k, v = _dev(ck), _dev(cv)
    got = _run(k, v, w.kv_off, w.ctx_len, w.n_nodes, paths, acc, w.token, bonus, w.chain_len)
    assert got["status"].tolist() == [pc.CURE_OK] * w.batch
    assert np.array_equal(_host(k), _expected_cache(ck, w.kv_off, w.ctx_len, paths, acc, rows))
    assert np.array_equal(_host(v), _expected_cache(cv, w.kv_off, w.ctx_len, paths, acc, rows))
    _check_tokens(got, w.token, paths, acc, bonus, w.chain_len, w.ctx_len, w.n_max)
