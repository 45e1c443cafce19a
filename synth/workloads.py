"""Workload presets and the seeded generator.

Shapes follow a Llama-3-8B-class target (32 query heads, 8 key/value heads,
head dim 128, vocabulary 128256) and the paper's block-parallel setting (draft
block K = 16, Sec. 4.1), with repair branches of fixed depth at seeded
Uncertainty Focal Points. The paper's own workloads (code-generation suites on
Qwen3-8B, Sec. 4.1) are not reproduced: these seeded tensors stand in for them.

Recipe (one sequence b, all draws from per-tensor sub-streams of the seed):

* ctx_len[b] cached tokens, then the tree: a chain of K nodes (parent i-1) plus
  one branch of ``branch_depth`` nodes per UFP position u (its root's parent is
  chain node u-1, or -1 for u = 0). Branch nodes are numbered after the chain,
  branches in ascending u. UFP positions are drawn without replacement from
  [0, K).
* Tokens: uniform over the vocabulary; a branch root's token differs from the
  chain token it replaces.
* Target argmax: each node draws an i.i.d. Bernoulli(p_agree) bit. For every
  parent slot (the context root and every node) the target's argmax is the
  token of its lowest-index child whose bit is set, or, when none is, a token
  different from all of its children's tokens (uniform for leaves).
* Logits row of node n: i.i.d. N(0, logit_std) quantised to the storage type,
  then the entry at the planted argmax is raised to the first representable
  value at or above (largest other entry + gap). Gaps: U(0.02, 0.4) on chain
  rows that are UFP positions, U(0.7, 4) on the other chain rows, U(0.02, 4) on
  repair rows. UFP rows therefore hold the smallest chain margins, and every
  margin is at least 0.02 and below 4 + one unit in the last place.
* Q, K, V: i.i.d. N(0, 1) quantised to the storage type.
* bf16 is stored as raw uint16 bit patterns, rounded to nearest even.
"""

from dataclasses import dataclass, field
import math

import numpy as np


def bf16_round(x):
    """float32 -> bf16 bits, round to nearest, ties to even (finite inputs)."""
    u = np.array(x, dtype=np.float32, copy=True).view(np.uint32)
    lsb = u >> np.uint32(16)
    lsb &= np.uint32(1)
    u += np.uint32(0x7FFF)     # finite values cannot carry out of 32 bits
    u += lsb
    u >>= np.uint32(16)
    return u.astype(np.uint16)


def _bf16_value(bits):
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32)


def bf16_ceil(x):
    """float32 -> the smallest bf16 value >= x, as bits (finite inputs)."""
    x = np.asarray(x, dtype=np.float32)
    r = bf16_round(x)
    v = _bf16_value(r)
    lower = v < x
    if np.any(lower):
        # One step up in magnitude for positives, down for negatives.
        r = r.astype(np.int32)
        pos = _bf16_value(r.astype(np.uint16)) >= 0
        r = np.where(lower & pos, r + 1, np.where(lower & ~pos, r - 1, r))
        r = r.astype(np.uint16)
        # -0.0 stepping down would wrap; values here are never exactly -0.0 - eps.
    return r


@dataclass
class Workload:
    name: str
    dtype: str                 # 'f32' or 'bf16' for logits, q, k, v
    batch: int
    hq: int
    hkv: int
    d: int
    vocab: int
    chain_len: int
    n_max: int
    scale: float
    tau: float
    repair_budget: int
    branch_depth: int
    ctx_len: np.ndarray        # int32 [batch]
    n_nodes: np.ndarray        # int32 [batch]
    kv_off: np.ndarray         # int64 [batch]
    kv_rows: int
    q: np.ndarray              # [batch, n_max, hq, d]
    k: np.ndarray              # [kv_rows, hkv, d]
    v: np.ndarray              # [kv_rows, hkv, d]
    parent: np.ndarray         # int32 [batch, n_max], -1 padding past n_nodes
    token: np.ndarray          # int32 [batch, n_max]
    depth: np.ndarray          # int32 [batch, n_max], by construction
    root_tgt: np.ndarray       # int32 [batch]
    tgt_planted: np.ndarray    # int32 [batch, n_max], argmax planted in the logits
    logits: np.ndarray         # [batch, n_max, vocab]
    ufp_planted: list = field(default_factory=list)   # per sequence, ascending position
    seed: int = 0

    @property
    def rows(self):
        return self.batch * self.n_max

    def elem_bytes(self):
        return 4 if self.dtype == "f32" else 2


def _rng(seed, stream):
    return np.random.default_rng(np.random.SeedSequence([int(seed), int(stream)]))


def _quantise(x, dtype):
    if dtype == "f32":
        return np.ascontiguousarray(x, dtype=np.float32)
    return bf16_round(x)


def _values(a, dtype):
    return a if dtype == "f32" else _bf16_value(a)


def _build_tree(chain_len, ufp, branch_depth):
    parent, depth = [], []
    for i in range(chain_len):
        parent.append(i - 1)
        depth.append(i)
    for u in sorted(ufp):
        for t in range(branch_depth):
            if t == 0:
                parent.append(u - 1)
                depth.append(u)
            else:
                parent.append(len(parent) - 1)
                depth.append(u + t)
    return parent, depth


def make_workload(name="custom", dtype="bf16", batch=1, hq=32, hkv=8, d=128, vocab=128256,
                  ctx_lens=(2048,), chain_len=16, n_ufp=4, branch_depth=4, seed=1,
                  logit_std=3.0, p_agree=0.8, tau=1.0, scale=None, ufp_positions=None,
                  n_max=None):
    """Generate one seeded workload. ctx_lens has one entry per sequence."""
    ctx_lens = [int(c) for c in ctx_lens]
    assert len(ctx_lens) == batch
    assert 0 <= n_ufp <= chain_len and branch_depth >= 1
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    r_tree = _rng(seed, 1)
    r_tok = _rng(seed, 2)
    r_agree = _rng(seed, 3)
    r_logit = _rng(seed, 4)
    r_gap = _rng(seed, 5)
    r_q = _rng(seed, 6)
    r_k = _rng(seed, 7)
    r_v = _rng(seed, 8)

    n_tree = chain_len + n_ufp * branch_depth
    n_max = n_tree if n_max is None else int(n_max)
    assert n_max >= n_tree
    parent = np.full((batch, n_max), -1, np.int32)
    depth = np.zeros((batch, n_max), np.int32)
    token = np.zeros((batch, n_max), np.int32)
    tgt = np.zeros((batch, n_max), np.int32)
    root_tgt = np.zeros(batch, np.int32)
    n_nodes = np.full(batch, n_tree, np.int32)
    ufps = []
    for b in range(batch):
        if ufp_positions is not None:
            ufp = sorted(int(u) for u in ufp_positions[b])
        else:
            ufp = sorted(int(u) for u in r_tree.choice(chain_len, size=n_ufp, replace=False))
        ufps.append(ufp)
        par, dep = _build_tree(chain_len, ufp, branch_depth)
        parent[b, :n_tree] = par
        depth[b, :n_tree] = dep
        # Tokens: uniform; a branch root differs from the chain token it replaces.
        tok = r_tok.integers(0, vocab, size=n_tree).astype(np.int64)
        for bi, u in enumerate(ufp):
            root = chain_len + bi * branch_depth
            while tok[root] == tok[u]:
                tok[root] = r_tok.integers(0, vocab)
        token[b, :n_tree] = tok
        # Planted target argmax, per parent slot (-1 = the context root).
        bits = r_agree.random(n_tree) < p_agree
        children = {p: [] for p in range(-1, n_tree)}
        for n in range(n_tree):
            children[par[n]].append(n)
        for p in range(-1, n_tree):
            kids = children[p]
            choice = None
            for c in kids:
                if bits[c]:
                    choice = int(tok[c])
                    break
            if choice is None:
                taken = {int(tok[c]) for c in kids}
                choice = int(r_agree.integers(0, vocab))
                while choice in taken:
                    choice = int(r_agree.integers(0, vocab))
            if p < 0:
                root_tgt[b] = choice
            else:
                tgt[b, p] = choice
        # Padding slots past the tree get a random argmax.
        for n in range(n_tree, n_max):
            tgt[b, n] = int(r_agree.integers(0, vocab))

    # Logits with planted argmax and gap.
    logits = np.empty((batch, n_max, vocab), np.float32 if dtype == "f32" else np.uint16)
    for b in range(batch):
        vals = r_logit.standard_normal((n_max, vocab), dtype=np.float32)
        vals *= np.float32(logit_std)
        qv = _quantise(vals, dtype)
        del vals
        fv = _values(qv, dtype)
        ufp = set(ufps[b])
        lo = np.empty(n_max, np.float64)
        hi = np.empty(n_max, np.float64)
        for n in range(n_max):
            if n < chain_len:
                lo[n], hi[n] = (0.02, 0.4) if n in ufp else (0.7, 4.0)
            else:
                lo[n], hi[n] = 0.02, 4.0
        gap = r_gap.uniform(lo, hi).astype(np.float32)
        spike = tgt[b].astype(np.int64)
        ar = np.arange(n_max)
        fv[ar, spike] = -np.inf            # fv is a copy for bf16, qv itself for f32
        other = fv.max(axis=1)
        target = (other + gap).astype(np.float32)
        if dtype == "f32":
            short = target - other < gap
            while np.any(short):
                target[short] = np.nextafter(target[short], np.float32(np.inf))
                short = target - other < gap
            qv[ar, spike] = target
        else:
            qv[ar, spike] = bf16_ceil(target)
        logits[b] = qv

    kv_rows_per = [ctx_lens[b] + int(n_nodes[b]) for b in range(batch)]
    kv_off = np.zeros(batch, np.int64)
    for b in range(1, batch):
        kv_off[b] = kv_off[b - 1] + kv_rows_per[b - 1]
    kv_rows = int(sum(kv_rows_per))

    def draw(rng, shape):
        return _quantise(rng.standard_normal(shape, dtype=np.float32), dtype)

    q = draw(r_q, (batch, n_max, hq, d))
    k = draw(r_k, (kv_rows, hkv, d))
    v = draw(r_v, (kv_rows, hkv, d))

    return Workload(
        name=name, dtype=dtype, batch=batch, hq=hq, hkv=hkv, d=d, vocab=vocab,
        chain_len=chain_len, n_max=n_max, scale=float(scale), tau=float(tau),
        repair_budget=n_ufp * branch_depth, branch_depth=branch_depth,
        ctx_len=np.asarray(ctx_lens, np.int32), n_nodes=n_nodes, kv_off=kv_off,
        kv_rows=kv_rows, q=q, k=k, v=v, parent=parent, token=token, depth=depth,
        root_tgt=root_tgt, tgt_planted=tgt, logits=logits, ufp_planted=ufps, seed=seed,
    )


def _ctx_uniform(seed, batch, lo, hi):
    return [int(x) for x in _rng(seed, 0).integers(lo, hi + 1, size=batch)]


# Named workloads. Each is a function of no arguments returning a Workload.
PRESETS = {
    # Single layer, fp32, 128 cached tokens, 4 heads of dim 64, vocab 1024:
    # chain 8 + 2 branches of depth 2 (12 nodes).
    "tiny_fp32": lambda: make_workload(
        "tiny_fp32", dtype="f32", batch=1, hq=4, hkv=4, d=64, vocab=1024, ctx_lens=[128],
        chain_len=8, n_ufp=2, branch_depth=2, seed=0, logit_std=2.0, scale=1.0 / 8.0),
    # Llama-3-8B attention shape, batch 1, context 2048, chain 16 + 4x4 (32 nodes).
    "llama3_8b_ctx2k_b1": lambda: make_workload(
        "llama3_8b_ctx2k_b1", batch=1, ctx_lens=[2048], chain_len=16, n_ufp=4,
        branch_depth=4, seed=1),
    # Batch 16, ragged context U[1024, 4096], chain 16 + 8x4 (48 nodes).
    "llama3_8b_ragged_b16": lambda: make_workload(
        "llama3_8b_ragged_b16", batch=16, ctx_lens=_ctx_uniform(2, 16, 1024, 4096),
        chain_len=16, n_ufp=8, branch_depth=4, seed=2),
    # Batch 4, context 32768, chain 16 + 4x4 (32 nodes).
    "llama3_8b_ctx32k_b4": lambda: make_workload(
        "llama3_8b_ctx32k_b4", batch=4, ctx_lens=[32768] * 4, chain_len=16, n_ufp=4,
        branch_depth=4, seed=3),
}
for _budget in (0, 8, 16, 32, 64):
    # Batch 8, context 8192, chain 16 + repair budget in depth-4 branches.
    PRESETS["llama3_8b_ctx8k_b8_budget%d" % _budget] = (
        lambda bud=_budget: make_workload(
            "llama3_8b_ctx8k_b8_budget%d" % bud, batch=8, ctx_lens=[8192] * 8,
            chain_len=16, n_ufp=bud // 4, branch_depth=4, seed=500 + bud))


def preset(name):
    return PRESETS[name]()


def algorithmic_bytes(w):
    """Bytes each hot-path call must move at least once (inputs read + outputs written).

    attention: K and V of context and tree rows, Q, O (same type as Q), LSE (fp32).
    margins:   the logits, plus 24 B of per-row results (6 x 4 B).
    accept:    parent, token, target argmax (3 x 4 B per node), 5 x 4 B of
               results per sequence plus the path (4 B per node).
    """
    eb = w.elem_bytes()
    kv = sum(int(w.ctx_len[b]) + int(w.n_nodes[b]) for b in range(w.batch)) * w.hkv * w.d * 2 * eb
    qo = 2 * w.batch * w.n_max * w.hq * w.d * eb + w.batch * w.n_max * w.hq * 4
    logits = w.batch * w.n_max * w.vocab * eb + w.batch * w.n_max * 24
    acc = w.batch * w.n_max * 16 + w.batch * 20
    return {"attention": kv + qo, "attention_kv": kv, "margins": logits, "accept": acc}
