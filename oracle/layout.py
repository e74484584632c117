"""Modality layout (the modality type index i_m of Algorithms 2 and 3).

T_m is the ascending list of positions of modality m. The estimation query
set of a modality is taken from the final segment of that modality's queries
(Section 3.2, Q-Boundary paragraph): here, the last min(64, n) positions of
the last maximal run of consecutive tokens of modality m. For heads without
modality boundaries the query set is the last 64 positions (Algorithm 1,
last_q = 64; Section 4.1).
"""
import numpy as np

LAST_Q = 64


def modality_array(S, modality):
    if modality is None:
        return np.zeros(S, dtype=np.uint8)
    m = np.asarray(modality, dtype=np.uint8)
    assert m.shape == (S,)
    return m


def positions_of(mod: np.ndarray) -> dict:
    """{m: T_m} for every modality present."""
    return {int(m): np.nonzero(mod == m)[0].astype(np.int64) for m in np.unique(mod)}


def global_rows(S: int) -> np.ndarray:
    return np.arange(max(0, S - LAST_Q), S, dtype=np.int64)


def final_run_rows(T: np.ndarray) -> np.ndarray:
    """Last min(64, n) positions of the last maximal run of consecutive positions."""
    n = len(T)
    start = n - 1
    while start > 0 and T[start - 1] == T[start] - 1:
        start -= 1
    run = T[start:]
    return run[-LAST_Q:].copy()
