"""Oracle: budget-aware repair-tree construction.

Test infrastructure only (see the package docstring).

Paper passages followed:

* Sec. 3.3, Eq. (3): a UFP's normalised uncertainty u = clip(1 - m / s, 0, 1)
  maps to its local branch budget b = clip(round(b_min + u (b_max - b_min)),
  b_min, b_max); the paper uses b_min = 1, b_max = 5 and leaves the margin
  scale s open.
* Algorithm 1: UFPs are visited in ascending margin order while the tree stays
  within the verification budget; each receives the top-b alternative tokens of
  the draft distribution at its position.
* Sec. 3.4: a repair path keeps the prefix, substitutes the fragile token and
  continues with the suffix drafted under the substitution. Paths sharing a
  prefix share parent nodes, so the result is a parent array in topological
  order, the default path (branch 0) first.

Readings where the paper is silent:

* round() is round-half-to-even, and Eq. (3) is evaluated in float32 on the
  float32 margin, each operation rounded once (no fused multiply-add): the
  precision the GPU takes the same integer decision in. A NaN margin (a row
  whose two best entries are both -inf) counts as fully certain (u = 0).
* b_min may be 0, in which case a UFP can receive no branch.
* Alternatives are the highest-ranked tokens of the draft distribution (value
  descending, index ascending) other than the block's own token at that
  position; under greedy drafting these are ranks 2 .. b + 1.
* The suffix tokens drafted under a substitution come from the caller: the
  drafter is not part of this path. suffix[u][r] holds the depth - 1 tokens
  that follow alternative r at block position u; without them the suffix
  nodes carry the placeholder token -1 (which no target argmax matches).
* Budget: whole branches only. A UFP receives min(b, remaining // depth)
  branches and the walk stops once no whole branch fits.
* Branch nodes follow the chain, UFP by UFP in the given (ascending-margin)
  order and, within a UFP, by alternative rank; a branch's root hangs off the
  chain node before its position (or the context, at position 0).
"""

import numpy as np

from .margins import as_float32


def topk(logits, dtype, k):
    """The first k entries of each row's stable descending order.

    Returns (values float32 [rows, k], indices int32 [rows, k]); ties in value go
    to the lower index.
    """
    x = as_float32(logits, dtype)
    if x.ndim != 2 or not 1 <= k <= x.shape[1]:
        raise ValueError("logits must be [rows, vocab] with 1 <= k <= vocab")
    order = np.argsort(-x.astype(np.float64), axis=1, kind="stable")[:, :k]
    return np.take_along_axis(x, order, axis=1).astype(np.float32), order.astype(np.int32)


def branch_budget(margin_f32, scale, b_min=1, b_max=5):
    """Eq. (3) for one margin, in float32 arithmetic with half-to-even rounding."""
    f = np.float32
    m = f(margin_f32)
    if np.isnan(m):
        return b_min
    u = f(1) - m / f(scale)
    u = min(max(u, f(0)), f(1))
    t = f(b_min) + u * f(b_max - b_min)
    b = int(np.rint(t))
    return min(max(b, b_min), b_max)


def alternatives(topk_idx_row, own_token, count):
    """The first `count` entries of a ranked token list other than own_token."""
    out = [int(t) for t in topk_idx_row if int(t) != int(own_token)]
    if len(out) < count:
        raise ValueError("ranked list too short for the requested alternatives")
    return out[:count]


def repair_tree(chain_tok, margin_f32, ufp_pos, topk_idx, suffix, repair_budget, depth,
                scale, b_min=1, b_max=5):
    """Build one sequence's candidate tree (Algorithm 1 with Eq. (3)).

    chain_tok   [K] the block-parallel draft (branch 0)
    margin_f32  [K] the chain positions' margins (float32)
    ufp_pos     UFP positions in ascending-margin order
    topk_idx    [K][>= b_max + 1] ranked draft tokens per position
    suffix      [K][b_max][depth - 1] caller-drafted suffix tokens, or None
    Returns a dict: parent, token, src (per node: -1 on the chain, else
    u * b_max + r for alternative r at position u), n_nodes, branches (the
    per-UFP branch counts, in ufp_pos order).
    """
    K = len(chain_tok)
    if depth < 1 or repair_budget < 0 or not 0 <= b_min <= b_max or not scale > 0:
        raise ValueError("bad tree parameters")
    parent = [i - 1 for i in range(K)]
    token = [int(t) for t in chain_tok]
    src = [-1] * K
    remaining = int(repair_budget)
    branches = []
    for u in ufp_pos:
        u = int(u)
        fit = remaining // depth
        if fit == 0:
            break
        nb = min(branch_budget(margin_f32[u], scale, b_min, b_max), fit)
        alts = alternatives(topk_idx[u], chain_tok[u], nb)
        for r, alt in enumerate(alts):
            root = len(parent)
            parent.append(u - 1)
            token.append(alt)
            src.append(u * b_max + r)
            for j in range(depth - 1):
                parent.append(root + j)
                token.append(-1 if suffix is None else int(suffix[u][r][j]))
                src.append(u * b_max + r)
        remaining -= nb * depth
        branches.append(nb)
    return {"parent": parent, "token": token, "src": src, "n_nodes": len(parent),
            "branches": branches}
