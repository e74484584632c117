"""Online estimate of the attention map from the last queries (fp64).

Algorithm 1 ("Approximate stride and phase") and Appendix C.3 (Vertical-Slash
head): A_hat = softmax(Q[-last_q:] K^T / sqrt(d) + causal mask), last_q = 64
(Section 4.1). Each row r of the query set R is normalised over every causal
key k <= pos(r) of the whole sequence (all modalities).

Reductions of A_hat used by the patterns, in a key coordinate system kappa
(global positions, or the index inside one modality's position list T_m):
  v[kappa] = sum_r A_hat[r, key(kappa)]            (vertical / column score)
  u[o]     = sum_r A_hat[r, key(kappa_r - o)]       (slash / diagonal score)
where kappa_r is row r's own coordinate. L_c = 1 + the largest coordinate
whose key is visible from some row of R.

Pinned in tests/test_oracle_core.py: LSE against scipy's logsumexp,
each A_hat row sums to 1, v sums to |R|, u against a brute-force double loop.
"""
import math

import numpy as np


def tau(D: int = 128) -> float:
    """Softmax scale sqrt(1/d_h) (Algorithm 5, first line)."""
    return math.sqrt(1.0 / D)


def row_lse(Qr: np.ndarray, K: np.ndarray, rows: np.ndarray, scale: float) -> np.ndarray:
    """LSE_r = ln sum_{k <= pos(r)} exp(scale * q_r . k_k)."""
    s = scale * (K[: int(rows.max()) + 1] @ Qr.T)          # [keys, rows]
    out = np.empty(len(rows))
    for r, p in enumerate(rows):
        col = s[: p + 1, r]
        m = col.max()
        out[r] = m + math.log(np.exp(col - m).sum())
    return out


def visible_extent(rows: np.ndarray, key_pos) -> int:
    pmax = int(rows.max())
    if key_pos is None:
        return pmax + 1
    return int(np.searchsorted(key_pos, pmax, side="right"))


def scores(Qr, K, rows, lse, scale, key_pos=None, row_coord=None):
    """Column scores v and (if row_coord is given) diagonal scores u, over L_c.

    key_pos maps coordinate -> position (None: coordinate = position)."""
    L_c = visible_extent(rows, key_pos)
    kp = np.arange(L_c) if key_pos is None else np.asarray(key_pos[:L_c])
    logits = scale * (K[kp] @ Qr.T)                         # [L_c, rows]
    v = np.zeros(L_c)
    u = None if row_coord is None else np.zeros(L_c)
    for r, p in enumerate(rows):
        a = np.where(kp <= p, np.exp(logits[:, r] - lse[r]), 0.0)
        v += a
        if u is not None:
            kr = int(row_coord[r])
            o = np.arange(0, kr + 1)
            u[o] += a[kr - o]
    return v, u, L_c
