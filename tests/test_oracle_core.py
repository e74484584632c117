"""Pins of the oracle's numerics, estimation, Grid search and VS selection.

Each test checks the oracle against something other than itself: torch's
bf16 casts, scipy's logsumexp, brute-force double loops, planted ground truth
and closed-form properties fixed by the paper (Algorithm 1; Appendix C.3).
"""
import math

import numpy as np
import pytest
import torch
from scipy.special import logsumexp

from oracle import estimate, grid, layout, numerics, vslash


# ---------------------------------------------------------------- numerics

def test_bf16_roundtrip_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(10000) * 10, [0.0, -0.0, 1e-40, 65504.0, 3.3e38]])
    ours = numerics.f64_to_bf16_bits(x)
    ref = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    back = numerics.bf16_bits_to_f64(ours)
    ref_back = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).double().numpy()
    assert np.array_equal(back, ref_back)


# ---------------------------------------------------------------- layout

def test_final_run_rows():
    T = np.array([0, 1, 2, 10, 11, 12, 13])
    assert layout.final_run_rows(T).tolist() == [10, 11, 12, 13]
    T = np.arange(5, 205)
    assert layout.final_run_rows(T).tolist() == list(range(141, 205))
    assert layout.global_rows(30).tolist() == list(range(30))


# ---------------------------------------------------------------- estimation

def _rand(S, D=128, seed=0):
    rng = np.random.default_rng(seed)
    return rng.standard_normal((S, D)), rng.standard_normal((S, D))


def test_row_lse_matches_scipy():
    Q, K = _rand(300)
    rows = np.arange(236, 300)
    sc = estimate.tau(128)
    lse = estimate.row_lse(Q[rows], K, rows, sc)
    for r, p in enumerate(rows):
        assert abs(lse[r] - logsumexp(sc * K[: p + 1] @ Q[p])) < 1e-12


def test_scores_global_sum_and_brute_force_diagonals():
    S = 200
    Q, K = _rand(S, seed=1)
    rows = layout.global_rows(S)
    sc = estimate.tau(128)
    lse = estimate.row_lse(Q[rows], K, rows, sc)
    v, u, L_c = estimate.scores(Q[rows], K, rows, lse, sc, None, rows)
    assert L_c == S
    # every estimated row is a probability distribution over its causal keys
    assert abs(v.sum() - len(rows)) < 1e-10
    assert abs(u.sum() - len(rows)) < 1e-10
    A = np.zeros((len(rows), S))
    for r, p in enumerate(rows):
        for k in range(p + 1):
            A[r, k] = math.exp(sc * Q[p] @ K[k] - lse[r])
    assert np.allclose(v, A.sum(0), rtol=0, atol=1e-12)
    ub = np.zeros(S)
    for r, p in enumerate(rows):
        for k in range(p + 1):
            ub[p - k] += A[r, k]
    assert np.allclose(u, ub, rtol=0, atol=1e-12)


def test_scores_local_coordinates():
    """Keys of one modality, rows of the same modality: coordinates are the
    index inside T_m, diagonal offsets are taken in that index."""
    S = 260
    Q, K = _rand(S, seed=2)
    mod = np.zeros(S, np.uint8)
    mod[40:120] = 1
    mod[170:260] = 1
    T = np.nonzero(mod == 1)[0]
    rows = layout.final_run_rows(T)
    loc = np.searchsorted(T, rows)
    sc = estimate.tau(128)
    lse = estimate.row_lse(Q[rows], K, rows, sc)
    v, u, L_c = estimate.scores(Q[rows], K, rows, lse, sc, T, loc)
    assert L_c == len(T)
    vb = np.zeros(len(T))
    ub = np.zeros(len(T))
    for r, p in enumerate(rows):
        for kap, k in enumerate(T):
            if k <= p:
                a = math.exp(sc * Q[p] @ K[k] - lse[r])
                vb[kap] += a
                ub[loc[r] - kap] += a
    assert np.allclose(v, vb, atol=1e-12) and np.allclose(u, ub, atol=1e-12)
    # the rows also attend text keys, so the modality's share is below |R|
    assert v.sum() < len(rows)


# ---------------------------------------------------------------- grid search

def _planted(L, period, phase, rng, noise=1e-3):
    v = rng.random(L) * noise
    v[phase::period] += 1.0
    return v


@pytest.mark.parametrize("period,phase", [(7, 3), (12, 0), (252, 89), (255, 254), (196, 17)])
def test_grid_search_recovers_planted(period, phase):
    rng = np.random.default_rng(period)
    L = period * 20 + 5
    v = _planted(L, period, phase, rng)
    best, folds, picks = grid.search(v, L, max(1, period - 8), period + 8)
    assert best == (period, phase)


def test_grid_search_divisors_lose_and_multiples_tie_to_smallest():
    rng = np.random.default_rng(5)
    v = _planted(12 * 40, 12, 5, rng)
    best, folds, picks = grid.search(v, len(v), 2, 36)
    assert best == (12, 5)
    # multiples score (within noise) the same as the period; divisors half or less
    assert abs(picks[24][0] - picks[12][0]) < 0.01 * picks[12][0]
    assert picks[6][0] < 0.6 * picks[12][0]
    # the paper's literal strict '>' (eps 0) may move to a multiple on noise
    best0, _, _ = grid.search(v, len(v), 12, 12, eps=0.0)
    assert best0 == (12, 5)


def test_grid_search_drops_short_strides_and_falls_back():
    v = np.ones(30)
    best, folds, _ = grid.search(v, 30, 16, 40)
    assert best is None and folds == {}
    best, _, _ = grid.search(v, 30, 1, 1)
    assert best == (1, 0)
    assert grid.candidates(1, 5000, 10 ** 7)[-1] == grid.MAX_STRIDE


def test_grid_permutation_bijection_and_phase_last():
    for L, s, p in [(100, 7, 3), (64, 1, 0), (1000, 252, 251), (37, 5, 0)]:
        cos, g0 = grid.permutation(L, s, p)
        assert sorted(cos.tolist()) == list(range(L))
        # groups are phase-homogeneous and ascending, phase p is the last group
        ph = cos % s
        assert ph[-1] == p and ph[0] == (p + 1) % s
        for x in range(1, L):
            if ph[x] == ph[x - 1]:
                assert cos[x] == cos[x - 1] + s
        assert g0[p] == L - len(range(p, L, s))
    cos, _ = grid.permutation(50, 1, 0)
    assert np.array_equal(cos, np.arange(50))


# ---------------------------------------------------------------- VS top-k

def test_topk_matches_sort_brute_force():
    rng = np.random.default_rng(3)
    for L, n in [(100, 10), (1000, 999), (50, 50), (50, 80), (300, 0)]:
        x = rng.random(L).astype(np.float32)
        x[::7] = x[3]        # plant exact ties
        sel = vslash.topk(x, n, L)
        if n >= L:
            assert sel.tolist() == list(range(L))
            continue
        ref = sorted(range(L), key=lambda i: (-float(x[i]), i))[:n]
        assert sel.tolist() == sorted(ref)
    # only the visible prefix competes
    x = np.arange(10, dtype=np.float32)
    assert vslash.topk(x, 3, 6).tolist() == [3, 4, 5]


def test_qboundary_grid_choice_from_the_modality_final_queries():
    """Q-Boundary Grid: the stride and phase come from the final queries of
    that modality against global key positions. Planted: keys at positions
    = 7 (mod 24) share a direction that only the video queries (positions
    [256, 1536)) carry; text queries carry another, with lines every 10
    positions. Video finds (24, 7) over global positions; the text modality
    (last run [1536, 1600)) finds (10, 3)."""
    from oracle import plan as P
    from synth import config as C
    S, D = 1600, 16
    rng = np.random.default_rng(9)
    mod = np.array([0] * 256 + [1] * 1280 + [0] * 64, dtype=np.uint8)
    K = 0.01 * rng.standard_normal((S, D))
    Q = 0.01 * rng.standard_normal((S, D))
    K[7::24, 0] += 3.0
    K[3::10, 1] += 3.0
    Q[mod == 1, 0] = 3.0
    Q[mod == 0, 1] = 3.0
    cfg = C.qboundary_head({0: C.grid(8, 40), 1: C.grid(16, 40)})
    ops, est, folds = P.choose(cfg, S, mod, lambda r: Q[r], K, scale=1.0)
    assert np.array_equal(est[("q", 1)].rows, np.arange(1472, 1536))
    assert np.array_equal(est[("q", 0)].rows, np.arange(1536, 1600))
    assert (ops[("q", 1)].sigma, ops[("q", 1)].p) == (24, 7)
    assert (ops[("q", 0)].sigma, ops[("q", 0)].p) == (10, 3)
    assert est[("q", 1)].L_c == 1536 and len(ops[("q", 1)].cos) == S
