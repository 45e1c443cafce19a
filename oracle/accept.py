"""Oracle: greedy acceptance over the candidate tree.

Test infrastructure only (see the package docstring).

Paper passages followed:

* Sec. 3.1, Eq. (1) and Sec. 3.5, Eq. (4): a(pi) is the accepted length of path
  pi and the verifier keeps the path with the longest accepted prefix.
* Sec. 3.5 and Algorithm 1: when the winning path is not branch 0 (the original
  draft chain) the draft cache must be resynchronised.
* Sec. 4.1: decoding is greedy, so a drafted token is accepted exactly when it
  equals the target's argmax at the position before it.

Readings where the paper is silent:

* tgt[n] is the target's argmax after node n (the prediction for n's child);
  root_tgt is its prediction for the first position after the context, and it
  verifies the depth-0 nodes.
* Ties between equally long accepted paths go to the deepest accepted node
  with the lowest index. The chain (branch 0) is numbered first, so it wins
  ties and needs no resynchronisation.
* acc_len counts accepted draft nodes; the bonus token (the target's argmax
  after the last accepted node) is returned on its own, so one step emits
  acc_len + 1 tokens.
* resync is set when the winning path holds a node numbered chain_len or
  higher, i.e. a repair node.
"""

from .tree import ancestors


def accept(parent, token, tgt, root_tgt, n_nodes, chain_len):
    """Accept walk for one sequence.

    Returns a dict: acc_len, path (node indices root->best), best (-1 if nothing
    is accepted), bonus, resync.
    """
    N = int(n_nodes)
    parent = [int(p) for p in parent[:N]]
    ancestors(parent, N)                      # validates the parent array
    accepted = [False] * N
    depth = [0] * N
    for n in range(N):                        # parents precede children
        p = parent[n]
        if p < 0:
            accepted[n] = int(token[n]) == int(root_tgt)
            depth[n] = 0
        else:
            accepted[n] = accepted[p] and int(token[n]) == int(tgt[p])
            depth[n] = depth[p] + 1
    best = -1
    for n in range(N):
        if accepted[n] and (best < 0 or depth[n] > depth[best]):
            best = n
    if best < 0:
        return {"acc_len": 0, "path": [], "best": -1, "bonus": int(root_tgt), "resync": 0}
    path, j = [], best
    while j >= 0:
        path.append(j)
        j = parent[j]
    path.reverse()
    return {
        "acc_len": depth[best] + 1,
        "path": path,
        "best": best,
        "bonus": int(tgt[best]),
        "resync": int(any(n >= chain_len for n in path)),
    }
