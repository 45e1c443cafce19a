"""GPU parity of cure_tree_attn on general candidate trees (Sec. 3.4).

Paths that share a prefix merge into shared parents, so a candidate tree is any
topologically ordered parent array: nested branches, wide sibling fans and
several nodes attached straight after the context (parent -1). The interface
takes any such array of up to 256 nodes. These cases draw random parent arrays
of four shapes and run them through every attention kernel: the 16-row MFMA
kernel (head dim 128 up to 256 rows and, in row blocks, beyond 336; head dim 64
up to 128 rows), the kernel with three 16-row groups per wave (head dim 128,
257 - 336 rows), the 32-row MFMA kernel (head dim 64 beyond 128 rows) and the
vector-ALU kernel (bf16 forced, and fp32), against the float64 oracle element
by element.
"""

import numpy as np
import pytest
import torch

import paper_2608_00531_amd as pc
from synth import make_workload
from parity_util import say, upload, gpu_attn, oracle_attn, check_attn

pytestmark = pytest.mark.gpu


def random_parents(rng, n, style):
    """A topologically ordered parent array of n nodes (parent[i] in [-1, i-1])."""
    par = np.full(n, -1, np.int32)
    if style == "uniform":
        # Any earlier node or the context, uniformly: bushy, several roots.
        for i in range(1, n):
            par[i] = int(rng.integers(-1, i))
    elif style == "nested":
        # Mostly extend the previous node, else branch off one of the last 12
        # nodes: long paths with branches inside branches.
        for i in range(1, n):
            par[i] = i - 1 if rng.random() < 0.75 else int(rng.integers(max(-1, i - 12), i))
    elif style == "fans":
        # A few hubs, each with a wide fan of siblings (and the context as one).
        hubs = [-1] + sorted(int(h) for h in rng.choice(max(n // 2, 1), size=max(1, n // 24),
                                                       replace=False))
        for i in range(1, n):
            earlier = [h for h in hubs if h < i]
            par[i] = int(rng.choice(earlier)) if rng.random() < 0.85 else i - 1
    elif style == "forest":
        # Several context-attached roots, each growing its own subtree.
        for i in range(1, n):
            r = rng.random()
            par[i] = -1 if r < 0.08 else (i - 1 if r < 0.6 else int(rng.integers(max(0, i - 30), i)))
    else:
        raise ValueError(style)
    assert all(-1 <= par[i] < i for i in range(n))
    return par


def general_tree_workload(seed, batch, hkv, group, d, n_nodes, ctx, style, dtype="bf16"):
    """Seeded Q/K/V for trees of n_nodes nodes per sequence with random parents;
    trees then trimmed to the per-sequence node counts in n_nodes (a prefix of a
    topological order is a tree too), with the cache rebuilt to match."""
    n_max = max(n_nodes)
    w = make_workload("general", dtype=dtype, batch=batch, hq=hkv * group, hkv=hkv, d=d,
                      ctx_lens=ctx, chain_len=n_max, n_ufp=0, branch_depth=1, seed=seed,
                      vocab=64)
    rng = np.random.default_rng(seed + 17)
    for b in range(batch):
        w.parent[b, :] = -1
        w.parent[b, :n_max] = random_parents(rng, n_max, style)
    w.n_nodes[:] = n_nodes
    rows = w.ctx_len + w.n_nodes
    off = np.concatenate([[0], np.cumsum(rows)[:-1]]).astype(np.int64)
    w.k = np.concatenate([w.k[w.kv_off[b]: w.kv_off[b] + rows[b]] for b in range(batch)])
    w.v = np.concatenate([w.v[w.kv_off[b]: w.kv_off[b] + rows[b]] for b in range(batch)])
    w.kv_off, w.kv_rows = off, int(rows.sum())
    return w


STYLES = ("uniform", "nested", "fans", "forest")

# (hkv, group, head dim, nodes per sequence, contexts): rows per kv-head = nodes x group.
CASES = [
    (2, 1, 128, [256, 201], [700, 0]),       # 256 rows: 16-row kernel, 16 waves
    (1, 4, 128, [256, 130], [333, 1500]),    # 1024 rows: four 256-row blocks
    (1, 8, 64, [256, 97], [64, 900]),        # 2048 rows at d 64: 32-row kernel, 8 blocks
    (2, 4, 64, [100, 100], [1, 1200]),       # 400 rows at d 64: 32-row kernel
    (8, 4, 128, [24, 9], [2048, 65]),        # 96 rows, GQA 4 (the Llama shape)
    (8, 4, 128, [48, 48], [1000, 2500]),     # 192 rows
    (8, 4, 128, [80, 61], [1300, 127]),      # 320 rows: 48-row waves
    (2, 4, 128, [84, 70], [500, 3000]),      # 336 rows: the 48-row block's capacity
    (4, 8, 128, [32, 17], [900, 4000]),      # 256 rows at GQA 8
    (2, 1, 64, [200, 3], [500, 63]),         # 200 rows at d 64 and GQA 1
    (1, 8, 64, [16, 12], [128, 129]),        # 128 rows at d 64: 16-row kernel
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_general_trees_every_kernel(case):
    hkv, group, d, nn, ctx = CASES[case]
    for si, style in enumerate(STYLES):
        seed = 4000 + 10 * case + si
        say("attn general tree case", case, "style", style, "seed", seed, "hkv", hkv,
            "group", group, "d", d, "nodes", nn, "ctx", ctx)
        w = general_tree_workload(seed, len(nn), hkv, group, d, nn, ctx, style)
        dev = upload(w)
        ref_o, ref_l = oracle_attn(w)
        for flags, kv_split in ((0, 0), (0, 3), (pc.CURE_ATTN_FORCE_VALU, 0)):
            o, lse, st = gpu_attn(w, dev, flags=flags, kv_split=kv_split)
            torch.cuda.synchronize()
            assert st.tolist() == [pc.CURE_OK] * w.batch
            check_attn(w, o, lse, ref_o, ref_l)


@pytest.mark.parametrize("style", STYLES)
def test_general_trees_fp32(style):
    # The fp32 vector-ALU path at 1e-5 on the same random tree shapes.
    seed = 4500 + STYLES.index(style)
    say("attn general tree fp32 style", style, "seed", seed)
    w = general_tree_workload(seed, 2, 2, 4, 64, [64, 40], [130, 0], style, dtype="f32")
    dev = upload(w)
    ref_o, ref_l = oracle_attn(w)
    o, lse, st = gpu_attn(w, dev, out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert st.tolist() == [pc.CURE_OK] * w.batch
    check_attn(w, o, lse, ref_o, ref_l)
