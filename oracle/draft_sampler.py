"""Drawing the tokens of a draft tree, float64.

TEST INFRASTRUCTURE ONLY: imported by tests/, __graft_entry__.smoke() and the
cpu_baseline leg of bench.py, never by the library.

A draft tree (Def. `de_tree`, Sec. 3.3) gives every node's children tokens
sampled from the draft model's distribution M_s(.|X^j) at their parent j,
either independently (with replacement) or without replacement. Conventions,
the same as the verifier's:

* row j of the draft logits is M_s(.|X^j) after the path root..j, tempered by
  T (softmax(z / T));
* the children of a node are drawn in ascending node index; child c's token is
  the inverse CDF (ascending token order, y = min{y : u*W < C(y)}) of the
  parent's distribution at u[c];
* without replacement, each drawn token is removed and the rest renormalised
  (the draft step of Eq. (e2)) before the next sibling is drawn, so siblings
  never repeat; with replacement every sibling draws from the same row.
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import tv_oracle as O


@dataclass
class DrawResult:
    status: int
    tokens: np.ndarray          # int64 [N+1]; tokens[0] = -1; all -1 on error
    margin: float = float("inf")  # smallest distance of u*W to a CDF boundary, / W


def _valid_parents(parents) -> bool:
    if len(parents) == 0 or int(parents[0]) != -1:
        return False
    return all(0 <= int(parents[i]) < i for i in range(1, len(parents)))


def draw_tree_tokens(parents, draft_logits, temperature, uniforms,
                     mode=O.WITHOUT_REPLACEMENT) -> DrawResult:
    """Tokens of every node of one tree. parents: [N+1] (parents[0] = -1,
    parents[i] < i); draft_logits: [N+1][V] rows (float, or bf16 bits as
    uint16); temperature: the float32 value used; uniforms: [N+1], u[c] draws
    node c's token. Status BAD_PARENT for an invalid tree, NONFINITE for a row
    with children that has NaN/+inf or no finite entry, DEGENERATE when a node
    without replacement has more children than tokens of positive probability;
    the largest of these codes when several rows fail (rows are independent)."""
    n1 = len(parents)
    err = lambda st: DrawResult(st, np.full(n1, -1, np.int64))
    if not _valid_parents(parents):
        return err(O.TREE_BAD_PARENT)
    zs = O.to_f64(draft_logits)
    T = float(np.float32(temperature))
    tokens = np.full(n1, -1, np.int64)
    margin = float("inf")
    status = O.TREE_OK            # rows are independent: the largest code of any row
    for j in range(n1):
        kids = [c for c in range(j + 1, n1) if int(parents[c]) == j]
        if not kids:
            continue
        q = O.tempered_softmax(zs[j], T)
        if q is None:
            status = max(status, O.TREE_NONFINITE)
            continue
        for c in kids:
            y, m = O.inverse_cdf(q, float(uniforms[c]))
            if y < 0:
                status = max(status, O.TREE_DEGENERATE)
                break
            tokens[c] = y
            margin = min(margin, m)
            if mode == O.WITHOUT_REPLACEMENT:
                if not q.sum() - q[y] > 0.0:     # no mass left for another sibling
                    if c != kids[-1]:
                        status = max(status, O.TREE_DEGENERATE)
                    break
                q = O.draft_update_e2(q, y)
    if status != O.TREE_OK:
        return err(status)
    return DrawResult(O.TREE_OK, tokens, margin)
