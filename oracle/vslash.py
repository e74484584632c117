"""Vertical-Slash selection (Appendix C.3) and the cross-modality VERT op.

From the estimate, the vertical lines are the n_v columns with the largest
column score v and the slash lines the n_s diagonals (offset o = q - k) with
the largest diagonal score u, both over the visible extent [0, L_c).
Order: score descending, ties to the smaller index; decided on fp32-rounded
scores. n >= L_c selects everything.

Token predicate: k in Vset  or  (q - k) in Oset (coordinates of the op).
Pinned in tests/test_oracle_core.py against a sort-based brute force and
the reductions n >= L_c -> dense.
"""
import numpy as np


def topk(scores: np.ndarray, n: int, L: int) -> np.ndarray:
    """Indices (ascending) of the n largest of scores[:L] (fp32), ties -> small index."""
    if n >= L:
        return np.arange(L, dtype=np.int64)
    if n <= 0:
        return np.zeros(0, dtype=np.int64)
    x = np.asarray(scores[:L]).astype(np.float32)
    order = np.lexsort((np.arange(L), -x))
    return np.sort(order[:n]).astype(np.int64)

