"""Seeded draft blocks for the repair-tree builder.

Recipe (one sequence, all draws from per-tensor sub-streams of the seed):

* Logits rows for the K block positions: i.i.d. N(0, logit_std) quantised to
  the storage type. Each row gets a planted head of ``runners + 1`` distinct
  tokens (drawn without replacement): the lead sits at the first representable
  value at or above (largest other entry + 4), the first runner ``gap`` below
  it and each further runner U(0, spacing) below its predecessor (all rounded
  up to a representable value), except that with probability p_tie a further
  runner repeats its predecessor's value exactly. Gaps are U(0.02, 0.4) on
  ``n_low`` seeded low-margin positions and U(0.7, 4) elsewhere. A fraction
  p_ninf of all entries is set to -inf.
* Draft tokens (branch 0): the planted lead with probability p_greedy, else
  with equal odds a planted runner or a uniform token.
* Suffix tokens for every (position, alternative rank, offset): uniform.

Nothing here ranks, compares or selects entries; the structure is planted.
"""

from dataclasses import dataclass

import numpy as np

from .workloads import _rng, _quantise, _values, bf16_ceil


@dataclass
class DraftBlock:
    dtype: str
    batch: int
    chain_len: int
    vocab: int
    b_max: int
    depth: int
    logits: np.ndarray      # [batch, chain_len, vocab] (float32 or bf16 bits)
    chain_tok: np.ndarray   # int32 [batch, chain_len]
    suffix: np.ndarray      # int32 [batch, chain_len, b_max, depth - 1]
    low: list               # per sequence, the planted low-margin positions


def _representable_at_least(x, dtype):
    x = np.asarray(x, np.float32)
    if dtype == "bf16":
        return bf16_ceil(x)
    return x


def make_draft_block(batch=1, chain_len=16, vocab=128256, dtype="bf16", seed=1, n_low=4,
                     runners=6, spacing=0.5, p_tie=0.2, p_greedy=0.75, p_ninf=0.0,
                     logit_std=3.0, b_max=5, depth=4):
    assert 0 <= n_low <= chain_len and runners + 1 <= vocab
    r_base = _rng(seed, 11)
    r_head = _rng(seed, 12)
    r_tok = _rng(seed, 13)
    r_suf = _rng(seed, 14)
    r_inf = _rng(seed, 15)
    logits = np.empty((batch, chain_len, vocab), np.float32 if dtype == "f32" else np.uint16)
    chain_tok = np.zeros((batch, chain_len), np.int32)
    lows = []
    for b in range(batch):
        vals = r_base.standard_normal((chain_len, vocab), dtype=np.float32)
        vals *= np.float32(logit_std)
        if p_ninf > 0:
            vals[r_inf.random((chain_len, vocab)) < p_ninf] = -np.inf
        qv = _quantise(np.where(np.isfinite(vals), vals, 0), dtype)
        if dtype == "bf16":
            qv[~np.isfinite(vals)] = 0xFF80          # -inf
        else:
            qv[~np.isfinite(vals)] = -np.inf
        low = sorted(int(u) for u in r_head.choice(chain_len, size=n_low, replace=False))
        lows.append(low)
        for i in range(chain_len):
            head = r_head.choice(vocab, size=runners + 1, replace=False)
            fv = _values(qv[i], dtype).copy()
            fv[head] = -np.inf
            rest_max = np.float32(fv.max()) if np.isfinite(fv.max()) else np.float32(0)
            gap = r_head.uniform(0.02, 0.4) if i in low else r_head.uniform(0.7, 4.0)
            lead = _representable_at_least(rest_max + np.float32(4), dtype)
            qv[i, head[0]] = lead
            prev = _values(np.asarray([lead]), dtype)[0]
            for j in range(1, runners + 1):
                if j == 1:
                    v = np.float32(prev - np.float32(gap))
                elif r_head.random() < p_tie:
                    v = prev
                else:
                    v = np.float32(prev - np.float32(r_head.uniform(0, spacing)))
                q = _representable_at_least(v, dtype)
                qv[i, head[j]] = q
                prev = _values(np.asarray([q]), dtype)[0]
            pick = r_tok.random()
            if pick < p_greedy:
                chain_tok[b, i] = head[0]
            elif pick < p_greedy + (1 - p_greedy) / 2:
                chain_tok[b, i] = head[1 + r_tok.integers(0, runners)]
            else:
                chain_tok[b, i] = r_tok.integers(0, vocab)
        logits[b] = qv
    suffix = r_suf.integers(0, vocab, size=(batch, chain_len, b_max, max(depth - 1, 0)),
                            dtype=np.int64).astype(np.int32)
    return DraftBlock(dtype=dtype, batch=batch, chain_len=chain_len, vocab=vocab, b_max=b_max,
                      depth=depth, logits=logits, chain_tok=chain_tok, suffix=suffix, low=lows)
