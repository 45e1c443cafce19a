"""Oracle: committing the accepted path of a verify step.

Test infrastructure only (see the package docstring).

Paper passages followed:

* Sec. 3.5 and Algorithm 1: the verifier returns the accepted tokens of the
  winning path; they become context for the next step, so the target's cache
  must hold their keys and values as context.
* Sec. 3.5 (cache resynchronisation) and Algorithm 1: when a repair branch
  wins, the tokens of the selected repair path are replayed into the draft
  model's cache so that its state matches the verified output.

Readings where the paper is silent:

* The cache rows of tree node n sit at ctx_len + n, after the context, in node
  order. Committing moves the row of the path's depth-j node to ctx_len + j
  for j < a (a = accepted length), so the cache reads as the old context
  followed by the accepted tokens, and the new context length is ctx_len + a.
  Cache rows from ctx_len + a on are not part of the new context and keep
  whatever they held.
* The emitted tokens are the accepted path's tokens followed by the bonus
  token (the target's prediction after the last accepted node): a + 1 tokens.
* The replay into the draft cache starts at the first repair node of the
  winning path (its depth is where the verified output leaves the draft
  chain) and runs to the last accepted node; the emitted tokens from that
  depth to a - 1 are the tokens to replay. With no repair node on the path
  the start is a and nothing needs replaying.
* A sequence whose acceptance result is invalid (acc_len < 0) is left as is.
"""

import numpy as np


def commit_kv(kv, kv_off, ctx_len, path, acc_len):
    """The cache after moving each sequence's accepted path rows into place.

    kv       [rows, ...] one layer of K or V (any row shape), token-major
    kv_off   [batch] first cache row of each sequence
    ctx_len  [batch] context length before the step
    path     [batch][>= a] node indices of the winning path, root first
    acc_len  [batch] accepted length a (negative: left as is)
    Returns a new array; the input is not modified.
    """
    old = np.asarray(kv)
    new = old.copy()
    for b in range(len(kv_off)):
        a = int(acc_len[b])
        base = int(kv_off[b]) + int(ctx_len[b])
        for j in range(max(a, 0)):
            new[base + j] = old[base + int(path[b][j])]
    return new


def commit_tokens(token, path, acc_len, bonus, chain_len):
    """Emitted tokens and the draft-cache replay start for one sequence.

    Returns a dict: emit (the a accepted tokens then the bonus), new_ctx_add (a),
    replay_start (depth of the first node numbered chain_len or higher on the
    path, else a).
    """
    a = int(acc_len)
    if a < 0:
        return {"emit": [], "new_ctx_add": 0, "replay_start": 0}
    nodes = [int(path[j]) for j in range(a)]
    emit = [int(token[n]) for n in nodes] + [int(bonus)]
    replay_start = a
    for j, n in enumerate(nodes):
        if n >= chain_len:
            replay_start = j
            break
    return {"emit": emit, "new_ctx_add": a, "replay_start": replay_start}
