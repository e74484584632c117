"""Grid head: stride/phase search and the row/column permutation.

Search (Algorithm 1, "Online search grid stride and phase"): for every stride
sigma of the stride space phi_g, view the estimate with period sigma and keep
the stride whose view has the largest maximum; the phase is the argmax.
Reading used here (the paper gives no reduction for "view"): fold the column
scores v by sigma and take the mean over periods,
    c_sigma[p] = mean_{t : t*sigma + p < L_c} v[t*sigma + p],
score_sigma = max_p c_sigma[p], p_sigma = smallest argmax. Strides with
2*sigma > L_c (fewer than two periods visible) are dropped. Strides are
scanned in ascending order and a later stride replaces the current best only
if its score exceeds best * (1 + eps_g), eps_g = 0.02 (the paper's strict ">"
is eps_g = 0; the margin keeps multiples of the true period from winning on
rounding noise). Decisions are taken on fp32-rounded scores, with the fp32
product best * 1.02f, so both implementations decide in one precision.
No stride left -> the op falls back to dense.

Permutation (Section 3.1; Appendix C.4, Figure "grid_pattern_permutation"):
tokens are grouped by phase (coordinate mod sigma), each group in coordinate
order, groups packed back to back. Phase p_g is placed last so that the
horizontal lines become the last query blocks and the vertical lines the
rightmost key blocks (Algorithm 1: "only the last and rightmost block"):
the group order is p_g+1, p_g+2, ..., p_g (mod sigma).

Pinned in tests/test_oracle_core.py: planted periods and phases are
recovered, divisors lose, multiples tie toward the smaller stride, the
permutation is a bijection and sigma = 1 is the identity.
"""
import numpy as np

EPS_G = 0.02
MAX_STRIDE = 1024


def candidates(lo: int, hi: int, L_c: int):
    return [s for s in range(max(1, lo), min(hi, MAX_STRIDE) + 1) if 2 * s <= L_c]


def fold64(v: np.ndarray, L_c: int, sigma: int) -> np.ndarray:
    """c_sigma[p] for p in [0, sigma) in fp64 (the mean over periods)."""
    return np.array([v[p:L_c:sigma].mean() for p in range(sigma)])


def fold(v: np.ndarray, L_c: int, sigma: int) -> np.ndarray:
    """c_sigma[p] for p in [0, sigma), fp64 then rounded to fp32."""
    return fold64(v, L_c, sigma).astype(np.float32)


def pick(folds: dict, eps: float = EPS_G):
    """The decision of the search from fp32 folds {sigma: c_sigma}: the
    smallest argmax phase of each stride, strides scanned ascending, a later
    stride replacing the best only if its score exceeds best * (1 + eps)
    (fp32 product). Returns ((sigma, p_g) or None, {sigma: (score, p)})."""
    best = None
    b = np.float32(0.0)
    one_eps = np.float32(1.0 + eps)
    picks = {}
    for s in sorted(folds):
        c = np.asarray(folds[s], dtype=np.float32)
        p = int(np.argmax(c))          # first (smallest) index of the maximum
        sc = c[p]
        picks[s] = (float(sc), p)
        if sc > np.float32(b * one_eps):
            best, b = (s, p), sc
    return best, picks


def search(v: np.ndarray, L_c: int, lo: int, hi: int, eps: float = EPS_G):
    """Returns ((sigma, p_g) or None, {sigma: fp32 fold}, {sigma: (score, p)})."""
    folds = {s: fold(v, L_c, s) for s in candidates(lo, hi, L_c)}
    best, picks = pick(folds, eps)
    return best, folds, picks


def phase_order(sigma: int, p: int):
    """Phases in group order: p+1, p+2, ..., p (mod sigma)."""
    return [(p + 1 + k) % sigma for k in range(sigma)]


def permutation(L: int, sigma: int, p: int):
    """coord_of_slot[x] (slot -> coordinate) and g0[phase] (group start slot)."""
    groups, g0, start = [], np.zeros(sigma, dtype=np.int64), 0
    for ph in phase_order(sigma, p):
        g = np.arange(ph, L, sigma, dtype=np.int64)
        g0[ph] = start
        start += len(g)
        groups.append(g)
    return np.concatenate(groups) if groups else np.zeros(0, np.int64), g0


def predicate(qc, kc, sigma, p, use_h, use_v, use_s):
    """Grid token predicate in coordinates (broadcasting arrays)."""
    out = np.zeros(np.broadcast(qc, kc).shape, dtype=bool)
    if use_s:
        out |= (qc % sigma) == (kc % sigma)
    if use_v:
        out |= (kc % sigma) == p
    if use_h:
        out |= (qc % sigma) == p
    return out
