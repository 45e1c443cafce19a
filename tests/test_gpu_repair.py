"""GPU parity: cure_repair_tree (Eq. (3), Algorithm 1, Sec. 3.4) against the oracle.

Everything the builder outputs is integer (parent, token, node and branch
counts), so every comparison is bit-exact. The Eq. (3) decision is taken in
float32 on both sides.
"""

import numpy as np
import pytest
import torch

import oracle
import paper_2608_00531_amd as pc
from synth import make_draft_block
from parity_util import say, to_dev

pytestmark = pytest.mark.gpu


def oracle_inputs(blk, tau, budget, depth):
    """Margins and UFP lists from the oracle, per sequence."""
    margin = np.zeros((blk.batch, blk.chain_len), np.float32)
    ufp = []
    for b in range(blk.batch):
        m = oracle.margins(blk.logits[b], blk.dtype)["margin_f32"]
        margin[b] = m
        ufp.append(oracle.ufp_select(m, tau, budget, depth))
    return margin, ufp


def oracle_trees(blk, margin, ufp, budget, depth, scale, b_min, b_max, with_suffix):
    out = []
    for b in range(blk.batch):
        rows = sorted(set(ufp[b]))
        ranked = np.zeros((blk.chain_len, b_max + 1), np.int64)
        if rows:
            _, idx = oracle.topk(blk.logits[b][rows], blk.dtype, b_max + 1)
            ranked[rows] = idx
        sfx = blk.suffix[b][:, :b_max, :depth - 1] if with_suffix else None
        out.append(oracle.repair_tree(blk.chain_tok[b], margin[b], ufp[b], ranked, sfx, budget,
                                      depth, scale, b_min, b_max))
    return out


def ufp_tensors(ufp, K):
    pos = np.full((len(ufp), K), -1, np.int32)
    cnt = np.zeros(len(ufp), np.int32)
    for b, lst in enumerate(ufp):
        pos[b, :len(lst)] = lst
        cnt[b] = len(lst)
    return torch.from_numpy(pos).cuda(), torch.from_numpy(cnt).cuda()


def check_trees(got, refs, K):
    n_nodes = got["n_nodes"].cpu().numpy()
    parent = got["parent"].cpu().numpy()
    token = got["token"].cpu().numpy()
    bcnt = got["branch_cnt"].cpu().numpy()
    for b, t in enumerate(refs):
        n = t["n_nodes"]
        assert n_nodes[b] == n, ("n_nodes", b, n_nodes[b], n)
        assert parent[b, :n].tolist() == t["parent"], ("parent", b)
        assert token[b, :n].tolist() == t["token"], ("token", b)
        nb = len(t["branches"])
        assert bcnt[b, :nb].tolist() == t["branches"], ("branch_cnt", b)
        assert np.all(bcnt[b, nb:] == 0), ("branch_cnt padding", b)


def run_case(blk, tau, budget, depth, scale, b_min, b_max, with_suffix=True, logits_dev=None,
             margin=None, ufp=None):
    if margin is None:
        margin, ufp = oracle_inputs(blk, tau, budget, depth)
    refs = oracle_trees(blk, margin, ufp, budget, depth, scale, b_min, b_max, with_suffix)
    x = to_dev(blk.logits, blk.dtype) if logits_dev is None else logits_dev
    pos, cnt = ufp_tensors(ufp, blk.chain_len)
    sfx = None
    if with_suffix and depth > 1:
        sfx = torch.from_numpy(np.ascontiguousarray(blk.suffix[:, :, :b_max, :depth - 1])).cuda()
    got = pc.cure_repair_tree(x, torch.from_numpy(margin).cuda(), pos, cnt,
                              torch.from_numpy(blk.chain_tok).cuda(), budget, depth, scale,
                              b_min=b_min, b_max=b_max, suffix=sfx)
    torch.cuda.synchronize()
    check_trees(got, refs, blk.chain_len)
    return got, refs


@pytest.mark.parametrize("dtype,vocab", [("bf16", 128256), ("bf16", 262147), ("f32", 1024),
                                         ("f32", 50000), ("bf16", 9)])
def test_trees_match_oracle(dtype, vocab):
    say("repair", dtype, vocab)
    blk = make_draft_block(batch=3, chain_len=16, vocab=vocab, dtype=dtype, seed=vocab % 97,
                           n_low=6, runners=min(6, vocab - 1), depth=4)
    run_case(blk, tau=1.0, budget=24, depth=4, scale=1.0, b_min=1, b_max=5)


@pytest.mark.parametrize("budget,depth,b_min,b_max,scale,suffix", [
    (16, 4, 1, 5, 1.0, True),      # budget-capped after the first UFP or two
    (64, 4, 1, 5, 0.7, True),      # every UFP gets its Eq. (3) count
    (40, 1, 0, 7, 2.0, False),     # depth-1 branches, the widest ranking, b_min = 0
    (7, 2, 2, 2, 1.0, True),       # fixed two branches, odd budget
    (3, 4, 1, 5, 1.0, True),       # budget below one branch: the chain alone
    (100, 15, 1, 5, 1.0, False),   # the paper's depth 15 with placeholder suffixes
])
def test_budget_and_shape_parameters(budget, depth, b_min, b_max, scale, suffix):
    say("repair params", budget, depth, b_min, b_max, scale, suffix)
    blk = make_draft_block(batch=4, chain_len=16, vocab=32000, seed=budget + depth, n_low=8,
                           b_max=b_max, depth=depth)
    run_case(blk, tau=1.5, budget=budget, depth=depth, scale=scale, b_min=b_min, b_max=b_max,
             with_suffix=suffix)


def test_end_to_end_from_gpu_margins():
    # The margin pass on the GPU feeds the builder, as in a decoding step;
    # batch 8, block 16, vocab 128256, budget 16 in depth-4 branches.
    say("repair end-to-end b8")
    blk = make_draft_block(batch=8, chain_len=16, vocab=128256, seed=77, n_low=4)
    x = to_dev(blk.logits, blk.dtype)
    m = pc.cure_margins(x, chain_len=16, tau=1.0, repair_budget=16, branch_depth=4)
    got = pc.cure_repair_tree(x, m["margin"], m["ufp_pos"], m["ufp_cnt"],
                              torch.from_numpy(blk.chain_tok).cuda(), 16, 4, 1.0,
                              suffix=torch.from_numpy(blk.suffix).cuda())
    torch.cuda.synchronize()
    margin, ufp = oracle_inputs(blk, 1.0, 16, 4)
    refs = oracle_trees(blk, margin, ufp, 16, 4, 1.0, 1, 5, True)
    check_trees(got, refs, 16)
    # The tree feeds the acceptance walk and the attention kernel as it is.
    assert all(t["n_nodes"] <= pc.CURE_MAX_TREE_NODES for t in refs)


@pytest.mark.parametrize("kind", ["constant", "few_values", "mostly_ninf"])
def test_ties_and_masked_rows(kind):
    # Rows where thousands of entries tie at the top take the exact fallback
    # selection; rows that are mostly -inf leave chunks with few real entries.
    say("repair ties", kind)
    if kind == "mostly_ninf":
        blk = make_draft_block(batch=2, chain_len=8, vocab=40000, dtype="f32", seed=5, n_low=4,
                               p_ninf=0.999)
    else:
        blk = make_draft_block(batch=2, chain_len=8, vocab=40000, dtype="f32", seed=6, n_low=4)
        rng = np.random.default_rng(9)
        if kind == "constant":
            blk.logits[:] = 0.0
        else:
            blk.logits[:] = rng.integers(-3, 2, size=blk.logits.shape).astype(np.float32)
    # Every chain position is a UFP (tau above every margin), so every row is ranked.
    run_case(blk, tau=np.inf, budget=16, depth=2, scale=1.0, b_min=1, b_max=5)


@pytest.mark.parametrize("ld", [20004, 20008])
def test_padded_rows(ld):
    # ld 20004: rows not 16-byte aligned, so entries are read one by one;
    # ld 20008: aligned rows whose last chunk ends in a partial vector.
    say("repair padded rows, ld", ld)
    blk = make_draft_block(batch=2, chain_len=16, vocab=20001, seed=12, n_low=5)
    pad = np.zeros((2, 16, ld), np.uint16)
    pad[:, :, :20001] = blk.logits
    x = to_dev(pad, "bf16")[:, :, :20001]
    assert x.stride(1) == ld
    run_case(blk, tau=1.0, budget=20, depth=4, scale=1.0, b_min=1, b_max=5, logits_dev=x)


def test_eq3_decisions_on_half_way_margins():
    # Margins handed in directly: multiples of 1/16 (exact halves of Eq. (3)
    # at s = 1 and at s = 0.5) plus random values, against the oracle's float32
    # evaluation. The budget never binds, so every branch count is Eq. (3).
    say("repair eq3 sweep")
    K = 64
    blk = make_draft_block(batch=8, chain_len=K, vocab=256, seed=31, n_low=0, depth=1)
    rng = np.random.default_rng(4)
    for scale in (1.0, 0.5, 0.3, 3.7):
        margin = np.concatenate([np.arange(K * 4, dtype=np.float32) / 16,
                                 rng.uniform(0, 1.2 * scale, K * 4).astype(np.float32)])
        margin = margin.reshape(8, K)
        ufp = [list(range(K)) for _ in range(8)]
        run_case(blk, tau=None, budget=K * 7, depth=1, scale=scale, b_min=1, b_max=5,
                 margin=margin, ufp=ufp)


def test_slot_list_edges():
    # ufp_cnt = 0 gives the chain alone; a list cut short by an entry outside the
    # block stops there; a count above the budget's slot limit is clipped.
    say("repair slot edges")
    K = 8
    blk = make_draft_block(batch=3, chain_len=K, vocab=3000, seed=8, n_low=3, depth=2)
    margin, _ = oracle_inputs(blk, 1.0, 8, 2)
    pos = np.array([[-1] * K, [3, 1, -1, 5, -1, -1, -1, -1], [0, 1, 2, 3, 4, 5, 6, 7]], np.int32)
    cnt = np.array([0, 4, 8], np.int32)
    refs = oracle_trees(blk, margin, [[], [3, 1], [0, 1, 2, 3]], 8, 2, 1.0, 1, 5, True)
    got = pc.cure_repair_tree(to_dev(blk.logits, "bf16"), torch.from_numpy(margin).cuda(),
                              torch.from_numpy(pos).cuda(), torch.from_numpy(cnt).cuda(),
                              torch.from_numpy(blk.chain_tok).cuda(), 8, 2, 1.0,
                              suffix=torch.from_numpy(blk.suffix).cuda())
    torch.cuda.synchronize()
    check_trees(got, refs, K)


def test_largest_block_and_vocabulary():
    # chain_len 1024 (the limit) with 1024 depth-1 slots, and a 524288-entry
    # vocabulary (the limit, 64 chunks per row).
    say("repair limits: chain 1024")
    blk = make_draft_block(batch=1, chain_len=1024, vocab=600, dtype="f32", seed=41, n_low=300,
                           depth=1)
    run_case(blk, tau=np.inf, budget=1024, depth=1, scale=1.0, b_min=0, b_max=3)
    say("repair limits: vocab 524288")
    blk = make_draft_block(batch=2, chain_len=4, vocab=524288, seed=42, n_low=2)
    run_case(blk, tau=1.0, budget=8, depth=4, scale=1.0, b_min=1, b_max=5)


@pytest.mark.parametrize("seed", range(16))
def test_random_parameters(seed):
    # Seeded random blocks and parameters: batch, chain length, vocabulary
    # (8 .. 200000), dtype, b_min/b_max, branch depth, budget, margin scale, tau,
    # the number of low-margin rows, -inf-heavy rows, with and without suffixes.
    rng = np.random.default_rng(7000 + seed)
    batch = int(rng.integers(1, 6))
    chain = int(rng.integers(1, 17))
    vocab = int(np.exp(rng.uniform(np.log(8), np.log(200000))))
    dtype = "bf16" if rng.random() < 0.7 else "f32"
    b_max = int(rng.integers(1, 8))
    b_min = int(rng.integers(0, b_max + 1))
    depth = int(rng.integers(1, 9))
    budget = int(rng.integers(0, chain * depth * 2 + 1))
    while chain + budget > 256:
        budget -= 1
    scale = float(rng.choice([1.0, 0.5, 2.0, 0.3]))
    tau = float(rng.choice([np.inf, 1.0, 1.5, 0.2]))
    n_low = int(rng.integers(0, chain + 1))
    runners = min(int(rng.integers(1, 8)), vocab - 1)
    blk = make_draft_block(batch=batch, chain_len=chain, vocab=vocab, dtype=dtype,
                           seed=9000 + seed, n_low=n_low, runners=runners, b_max=b_max,
                           depth=depth, p_ninf=float(rng.choice([0.0, 0.0, 0.3])))
    suffix = bool(rng.random() < 0.7)
    say("repair random", seed, batch, chain, vocab, dtype, b_min, b_max, depth, budget, scale,
        tau, suffix)
    run_case(blk, tau=tau, budget=budget, depth=depth, scale=scale, b_min=b_min, b_max=b_max,
             with_suffix=suffix)
