"""GPU parity: cure_margins_accept against cure_margins followed by
cure_accept (every output bit for bit), and against the oracle."""

import numpy as np
import pytest
import torch

import paper_2608_00531_amd as pc
import oracle
from synth import preset, make_workload
from parity_util import say

pytestmark = pytest.mark.gpu

MARGIN_KEYS = ("top1_val", "top1_idx", "top2_val", "top2_idx", "lse", "margin")
ACCEPT_KEYS = ("acc_len", "path", "best", "bonus", "resync")


def _logits(w):
    a = np.ascontiguousarray(w.logits)
    if w.dtype == "bf16":
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(a).cuda()


def _t(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.int32)).cuda()


def _check(x, parent, token, root_tgt, n_nodes, chain_len, tau, budget, depth, gate):
    d = (_t(parent), _t(token), _t(root_tgt), _t(n_nodes))
    fused = pc.cure_margins_accept(x, *d, chain_len, tau, budget, depth, gate=gate)
    sep = pc.cure_margins(x, chain_len, tau, budget, depth, gate=gate)
    acc = pc.cure_accept(d[0], d[1], sep["top1_idx"], d[2], d[3], chain_len)
    torch.cuda.synchronize()
    for k in MARGIN_KEYS + (("ufp_pos", "ufp_cnt") if gate else ()):
        assert torch.equal(fused[k], sep[k]), k
    for k in ACCEPT_KEYS:
        assert torch.equal(fused[k], acc[k]), k
    return fused


@pytest.mark.parametrize("name", ["llama3_8b_ctx2k_b1", "llama3_8b_ragged_b16",
                                  "llama3_8b_ctx8k_b8_budget64"])
def test_presets_match_separate_calls_and_oracle(name):
    # The default step (rows split over 16 chunks), the ragged batch (rows
    # unsplit, so the finishing launch runs only the gate and the walk) and
    # the 80-node trees.
    say("margins+accept", name)
    w = preset(name)
    x = _logits(w)
    out = _check(x, w.parent, w.token, w.root_tgt, w.n_nodes, w.chain_len, w.tau,
                 w.repair_budget, w.branch_depth, True)
    top1 = out["top1_idx"].cpu().numpy()
    for b in range(w.batch):
        ref = oracle.accept(w.parent[b], w.token[b], top1[b], int(w.root_tgt[b]),
                                   int(w.n_nodes[b]), w.chain_len)
        assert int(out["acc_len"][b]) == ref["acc_len"]
        assert int(out["best"][b]) == ref["best"]
        assert int(out["bonus"][b]) == ref["bonus"]
        assert int(out["resync"][b]) == ref["resync"]
        p = out["path"][b].tolist()
        assert p[: ref["acc_len"]] == ref["path"] and all(v == -1 for v in p[ref["acc_len"]:])


@pytest.mark.parametrize("seed", range(6))
def test_random_trees_small_vocab(seed):
    # Small vocabularies, so the targets often agree with the tokens and deep
    # paths are accepted; trees of 1 - 256 nodes that mostly extend a recent
    # node; with and without the gate; rows split or not (vocab sizes either
    # side of one chunk).
    rng = np.random.default_rng(4200 + seed)
    B = int(rng.integers(1, 9))
    n_max = int(rng.choice([1, 7, 64, 65, 200, 256]))
    vocab = int(rng.choice([3, 5, 9000, 20000]))
    chain = int(rng.integers(0, n_max + 1))
    gate = bool(seed % 2) and chain >= 1
    say("margins+accept random", seed, B, n_max, vocab, chain, gate)
    x = torch.from_numpy(rng.standard_normal((B, n_max, vocab)).astype(np.float32)).cuda()
    if seed % 3 == 0:
        x = x.to(torch.bfloat16)
    parent = np.full((B, n_max), -1, np.int32)
    n_nodes = rng.integers(0, n_max + 1, B).astype(np.int32)
    n_nodes[0] = n_max
    for b in range(B):
        for n in range(1, int(n_nodes[b])):
            parent[b, n] = int(rng.integers(max(-1, n - 4), n))
    tok_alpha = min(vocab, 3)
    token = rng.integers(0, tok_alpha, (B, n_max)).astype(np.int32)
    root = rng.integers(0, tok_alpha, B).astype(np.int32)
    _check(x, parent, token, root, n_nodes, chain, 0.5, 8, 2, gate)


def test_malformed_tree_and_oversized_count():
    # Sequence 0: parent[2] = 5 is not an earlier node; sequence 1: n_nodes
    # above n_max; sequence 2 is well formed.
    say("margins+accept malformed")
    rng = np.random.default_rng(7)
    x = torch.from_numpy(rng.standard_normal((3, 4, 300)).astype(np.float32)).cuda()
    parent = np.array([[-1, 0, 5, 1], [-1, 0, 1, 2], [-1, 0, 1, 2]], np.int32)
    token = np.zeros((3, 4), np.int32)
    out = _check(x, parent, token, np.zeros(3, np.int32), np.array([4, 5, 4], np.int32), 2,
                 0.5, 4, 2, True)
    assert out["acc_len"][:2].tolist() == [-1, -1] and out["resync"][:2].tolist() == [-1, -1]
    assert out["path"][0].tolist() == [-1] * 4


def test_empty_trees_and_argument_errors():
    say("margins+accept edge cases")
    L = pc.lib()
    # rows = 0: no margin rows, and the walk on empty trees.
    i = dict(dtype=torch.int32, device="cuda")
    outs = [torch.full((2,), 7, **i) for _ in range(4)]
    root = torch.tensor([3, 4], **i)
    nn = torch.zeros(2, **i)
    dummy = torch.zeros(1, **i)
    P = lambda t: t.data_ptr()
    st = L.cure_margins_accept(P(dummy), pc.CURE_F32, 2, 0, 10, 10, P(dummy), P(dummy),
                               P(dummy), P(dummy), P(dummy), P(dummy), 0, 1.0, 0, 1, None, None,
                               P(dummy), P(dummy), P(root), P(nn), P(outs[0]), None,
                               P(outs[1]), P(outs[2]), P(outs[3]), None, 0, None)
    torch.cuda.synchronize()
    assert st == pc.CURE_OK
    assert outs[0].tolist() == [0, 0] and outs[1].tolist() == [-1, -1]
    assert outs[2].tolist() == [3, 4] and outs[3].tolist() == [0, 0]
    # More than 256 rows cannot be tree nodes.
    st = L.cure_margins_accept(P(dummy), pc.CURE_F32, 1, 257, 10, 10, P(dummy), P(dummy),
                               P(dummy), P(dummy), P(dummy), P(dummy), 0, 1.0, 0, 1, None, None,
                               P(dummy), P(dummy), P(root), P(nn), P(outs[0]), P(dummy),
                               P(outs[1]), P(outs[2]), P(outs[3]), P(dummy), 1 << 20, None)
    assert st == pc.CURE_ERR_UNSUPPORTED


@pytest.mark.parametrize("vocab,dtype", [(3001, torch.float32), (40000, torch.bfloat16)])
def test_padded_rows_and_ties(vocab, dtype):
    # Rows padded by 3 entries (ld = vocab + 3: the margin pass's scalar path),
    # rows split (40000) or not (3001), and every row's maximum repeated so the
    # argmax the walk uses is decided by the lowest-index rule.
    say("margins+accept padded", vocab, dtype)
    rng = np.random.default_rng(vocab)
    B, n_max = 3, 40
    big = torch.from_numpy(rng.standard_normal((B, n_max, vocab + 3)).astype(np.float32))
    cols = rng.integers(0, vocab, (B, n_max, 2))
    for b in range(B):
        for n in range(n_max):
            big[b, n, cols[b, n]] = 9.0
    x = big.to(dtype).cuda()[:, :, :vocab]
    assert x.stride(1) == vocab + 3
    parent = np.full((B, n_max), -1, np.int32)
    for b in range(B):
        for n in range(1, n_max):
            parent[b, n] = n - 1 if n < 20 else int(rng.integers(10, n))
    # Tokens equal to the argmax the target will produce, so the chain is accepted.
    am = np.minimum(cols[:, :, 0], cols[:, :, 1]).astype(np.int32)
    token = np.zeros((B, n_max), np.int32)
    root = am[:, 0].copy()
    for b in range(B):
        token[b, 0] = root[b]
        for n in range(1, n_max):
            token[b, n] = am[b, parent[b, n]]
    out = _check(x, parent, token, root, np.full(B, n_max, np.int32), 16, 0.5, 8, 2, True)
    assert out["top1_idx"].cpu().numpy().tolist() == am.tolist()
    assert int(out["acc_len"].min()) >= 20
