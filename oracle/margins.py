"""Oracle: predictive confidence margins and UFP selection.

Test infrastructure only (see the package docstring).

Paper passages followed:

* Sec. 3.3, Eq. (2): for block position i the margin is the top-1 minus the
  top-2 unnormalised log-probability of the draft model. Whether the logits or
  the log-softmax values are meant does not change the margin (the row's
  normaliser cancels), so the margin is taken on the logits as given and the
  normaliser (log-sum-exp) is reported on its own.
* Sec. 3.3 and Algorithm 1: a position is an Uncertainty Focal Point when its
  margin is strictly below tau; positions are taken in ascending order of
  margin until the verification budget is used.

Readings where the paper is silent:

* Ties in the top-2 order go to the lowest vocabulary index (a stable sort on
  the negated values). A row whose maximum occurs twice therefore has its
  top-2 at the second such index and margin 0.
* Equal margins in the UFP order go to the lower block position.
* The UFP decision (margin < tau, and the ascending order) is taken on the
  margin rounded to float32, the precision the GPU kernel computes it in; the
  reported margin is the exact float64 difference.
"""

import numpy as np


def widen_bf16(bits):
    """Exact bf16 -> float32: the 16 stored bits become the high half of a float32."""
    b = np.ascontiguousarray(bits).view(np.uint16).astype(np.uint32)
    return (b << np.uint32(16)).view(np.float32)


def as_float32(x, dtype):
    """Values of a logits/QKV buffer as float32. dtype is 'f32' or 'bf16' (raw uint16 bits)."""
    if dtype == "bf16":
        return widen_bf16(x)
    if dtype == "f32":
        return np.asarray(x, dtype=np.float32)
    raise ValueError("dtype must be 'f32' or 'bf16'")


def margins(logits, dtype):
    """Per-row top-1/top-2, log-sum-exp and margin of a [rows, vocab] logits matrix.

    Returns a dict of arrays, one entry per row:
      top1_idx, top2_idx  int32   the first two entries of the stable descending order
      top1_val, top2_val  float32 the logits at those indices (exact copies)
      lse                 float64 log(sum_v exp(x_v)), natural log
      margin              float64 top1_val - top2_val (Eq. 2)
      margin_f32          float32 the same difference rounded to float32
    """
    x = as_float32(logits, dtype)
    if x.ndim != 2 or x.shape[1] < 2:
        raise ValueError("logits must be [rows, vocab] with vocab >= 2")
    rows = x.shape[0]
    out = {
        "top1_idx": np.zeros(rows, np.int32), "top2_idx": np.zeros(rows, np.int32),
        "top1_val": np.zeros(rows, np.float32), "top2_val": np.zeros(rows, np.float32),
        "lse": np.zeros(rows, np.float64), "margin": np.zeros(rows, np.float64),
        "margin_f32": np.zeros(rows, np.float32),
    }
    with np.errstate(invalid="ignore"):     # (-inf) - (-inf) in an all -inf row
        for r in range(rows):
            _row_margin(x, r, out)
    return out


def _row_margin(x, r, out):
    row = x[r].astype(np.float64)
    # Full stable sort, descending by value; equal values keep index order.
    order = np.argsort(-row, kind="stable")
    i1, i2 = int(order[0]), int(order[1])
    out["top1_idx"][r], out["top2_idx"][r] = i1, i2
    out["top1_val"][r], out["top2_val"][r] = x[r, i1], x[r, i2]
    out["margin"][r] = row[i1] - row[i2]
    out["margin_f32"][r] = np.float32(x[r, i1]) - np.float32(x[r, i2])
    # log-sum-exp, shifted by the row maximum.
    mx = row[i1]
    if mx == -np.inf:
        out["lse"][r] = -np.inf
    else:
        out["lse"][r] = mx + np.log(np.sum(np.exp(row - mx)))


def ufp_select(margin_f32, tau, repair_budget, branch_depth):
    """Uncertainty Focal Points of one draft block (Sec. 3.3, Algorithm 1).

    margin_f32: the block's K chain-position margins (float32).
    Candidates are the positions with margin < tau (strict). They are ordered by
    ascending (margin, position) and the first floor(repair_budget / branch_depth)
    are kept, so that whole branches of branch_depth nodes never exceed the
    repair budget. Returns the kept positions, in that order, as a list.
    """
    if branch_depth < 1 or repair_budget < 0:
        raise ValueError("branch_depth must be >= 1 and repair_budget >= 0")
    m = np.asarray(margin_f32, dtype=np.float32)
    tau32 = np.float32(tau)
    candidates = [i for i in range(len(m)) if m[i] < tau32]
    candidates.sort(key=lambda i: (float(m[i]), i))
    return candidates[: repair_budget // branch_depth]
