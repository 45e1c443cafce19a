"""CPU oracle for CURE's verify-and-repair hot path.

TEST INFRASTRUCTURE ONLY. Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this package. The product path (the
HIP library and its Python binding) never imports, calls or links anything in
here, and nothing in here imports the product path.

Every function is the plain definition of what the paper's step computes,
written for a reader who checks it against the paper by eye, in float64
unless the paper (or the decision being reproduced) fixes another precision:

* ``margins``       -- predictive confidence margin, Sec. 3.3 Eq. (2): top-1 /
                       top-2 of a row by a full stable sort, plus the
                       log-sum-exp that normalises the row.
* ``ufp_select``    -- Uncertainty Focal Points, Sec. 3.3 and Algorithm 1:
                       positions with margin below tau, ascending margin,
                       capped by the repair budget.
* ``ancestors``     -- the candidate tree as a parent array, Sec. 3.4 (paths
                       sharing a prefix merge into shared parents).
* ``tree_attention``-- single-pass tree-attention verification, Sec. 3.2 and
                       Sec. 3.5: each node attends to the cached context and to
                       its own ancestors.
* ``accept``        -- accepted prefix length per path and the best path,
                       Sec. 3.1 Eq. (1) and Sec. 3.5 Eq. (4).
* ``commit_kv``, ``commit_tokens``
                    -- committing the winner, Sec. 3.5 and Algorithm 1: its
                       cache rows moved after the context in depth order, the
                       emitted tokens, and where the draft-cache replay starts.
* ``topk``, ``branch_budget``, ``repair_tree``
                    -- the repair tree, Eq. (3), Algorithm 1 and Sec. 3.4:
                       ranked alternatives by a full stable sort, the branch
                       budget per UFP, and the budget-capped assembly of the
                       parent/token arrays.

Inputs are the same bytes the GPU path receives: bf16 arrives as raw uint16
bit patterns and is widened here exactly to float32 by this package's own
code. Logit values must be finite or -inf.
"""

from .margins import widen_bf16, as_float32, margins, ufp_select
from .tree import ancestors, tree_attention
from .accept import accept
from .repair import topk, branch_budget, repair_tree
from .commit import commit_kv, commit_tokens

__all__ = [
    "widen_bf16", "as_float32", "margins", "ufp_select",
    "ancestors", "tree_attention", "accept",
    "topk", "branch_budget", "repair_tree", "commit_kv", "commit_tokens",
]
