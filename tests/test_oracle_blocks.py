"""Pins of the oracle's block sets: closed forms == literal lift, reductions.

The literal lift enumerates every (query, key) token pair (causal by original
positions, plus each row's own key block); the closed forms compute the same
set per op without enumeration. They are independent code paths in
oracle/plan.py and must agree exactly.
"""
import itertools

import numpy as np
import pytest

from oracle import plan as P
from synth import config as C

FLAGS = list(itertools.product([False, True], repeat=3))   # (h, v, s)


def _same(hp):
    lifted = P.lift_blocks(hp)
    assert len(lifted) == len(hp.blocks)
    for i, (a, b) in enumerate(zip(hp.blocks, lifted)):
        assert np.array_equal(a, b), (i, a, b)


def _grid_plan(L, s, p, h, v, sflag):
    st = P.grid_state(C.grid(s, s, h, v, sflag), L, s, p)
    return P.assemble(C.HEAD_GLOBAL, L, None, {"g": st})


@pytest.mark.parametrize("L", [333, 128])
def test_grid_closed_form_exhaustive_small_strides(L):
    for s in range(1, 33):
        for p in range(s):
            for h, v, sf in FLAGS:
                _same(_grid_plan(L, s, p, h, v, sf))


def test_grid_closed_form_frame_sized_strides():
    rng = np.random.default_rng(0)
    for L in (2000, 4096, 1111):
        for s in (63, 64, 65, 100, 127, 196, 252, 255, 256, 500):
            for h, v, sf in FLAGS:
                p = int(rng.integers(0, s))
                _same(_grid_plan(L, s, p, h, v, sf))


def test_grid_reductions():
    L = 700
    hp = _grid_plan(L, 1, 0, False, False, True)          # one group, same phase = dense
    nb = hp.nbq
    assert all(np.array_equal(hp.blocks[i], np.arange(i + 1)) for i in range(nb))
    assert np.array_equal(hp.qperm[:L], np.arange(L))
    hp = _grid_plan(L, 9, 4, False, False, False)         # no lines: own blocks only
    assert all(np.array_equal(hp.blocks[i], [i]) for i in range(nb))


def _id_plan(L, st):
    return P.assemble(C.HEAD_GLOBAL, L, None, {"g": st})


def test_ashape_closed_form_and_reductions():
    rng = np.random.default_rng(1)
    for L in (300, 1000, 64 * 9):
        for sink, local in [(128, 256), (7, 64), (0, 100), (128, 0), (1, 1), (500, 50)]:
            _same(_id_plan(L, P.OpState(C.OP_ASHAPE, C.ashape(sink, local), L=L)))
        dense = [np.arange(i + 1) for i in range((L + 63) // 64)]
        for sink, local in [(L, 1), (0, L), (L + 5, L + 5)]:
            hp = _id_plan(L, P.OpState(C.OP_ASHAPE, C.ashape(sink, local), L=L))
            assert all(np.array_equal(a, b) for a, b in zip(hp.blocks, dense))


def test_vslash_closed_form_and_reductions():
    rng = np.random.default_rng(2)
    for L in (300, 1000, 64 * 7 + 1):
        for nv, ns in [(10, 10), (1, 50), (0, 3), (40, 0), (200, 200)]:
            vs = np.sort(rng.choice(L, size=min(nv, L), replace=False))
            ss = np.sort(rng.choice(L, size=min(ns, L), replace=False))
            st = P.OpState(C.OP_VSLASH, C.vslash(nv, ns), vsel=vs, ssel=ss, L=L)
            _same(_id_plan(L, st))
        dense = [np.arange(i + 1) for i in range((L + 63) // 64)]
        for vs, ss in [(np.arange(L), np.zeros(0, np.int64)), (np.zeros(0, np.int64), np.arange(L))]:
            hp = _id_plan(L, P.OpState(C.OP_VSLASH, C.vslash(0, 0), vsel=vs, ssel=ss, L=L))
            assert all(np.array_equal(a, b) for a, b in zip(hp.blocks, dense))


def _random_layout(rng, S, nmod=2, minseg=1, maxseg=300):
    segs, m, n = [], 0, 0
    while n < S:
        ln = int(min(S - n, rng.integers(minseg, maxseg + 1)))
        segs.append(np.full(ln, m, np.uint8))
        n += ln
        m = (m + int(rng.integers(1, nmod))) % nmod
    return np.concatenate(segs)


def _rand_static_op(rng, L):
    k = int(rng.integers(0, 3))
    if k == 0:
        return P.OpState(C.OP_SF_FIXED, C.sf_fixed(int(rng.integers(1, 300)), int(rng.integers(1, 300))), L=L)
    if k == 1:
        return P.OpState(C.OP_SF_STRIDED, C.sf_strided(int(rng.integers(1, 300)), int(rng.integers(1, 300))), L=L)
    return P.OpState(C.OP_TRISHAPE, C.trishape(int(rng.integers(0, 200)), int(rng.integers(0, 300)),
                                               int(rng.integers(0, 200))), L=L)


def _rand_identity_op(rng, L, allow=("dense", "ashape", "vslash", "static")):
    k = allow[int(rng.integers(0, len(allow)))]
    if k == "static":
        return _rand_static_op(rng, L)
    if k == "dense":
        return P.OpState(C.OP_DENSE, C.dense(), L=L)
    if k == "ashape":
        sink, local = int(rng.integers(0, 200)), int(rng.integers(0, 300))
        return P.OpState(C.OP_ASHAPE, C.ashape(sink, local), L=L)
    nv, ns = int(rng.integers(0, 40)), int(rng.integers(0, 40))
    vs = np.sort(rng.choice(L, size=min(nv, L), replace=False))
    ss = np.sort(rng.choice(L, size=min(ns, L), replace=False))
    return P.OpState(C.OP_VSLASH, C.vslash(nv, ns), vsel=vs, ssel=ss, L=L)


def test_qboundary_closed_form_random_layouts():
    rng = np.random.default_rng(3)
    for trial in range(25):
        S = int(rng.integers(100, 1500))
        mod = _random_layout(rng, S, nmod=int(rng.integers(2, 4)), maxseg=int(rng.integers(5, 400)))
        ops = {("q", int(m)): _rand_identity_op(rng, S) for m in np.unique(mod)}
        hp = P.assemble(C.HEAD_QBOUNDARY, S, mod, ops)
        _same(hp)


def test_2d_closed_form_random_layouts():
    rng = np.random.default_rng(4)
    for trial in range(25):
        S = int(rng.integers(100, 1500))
        mod = _random_layout(rng, S, nmod=int(rng.integers(2, 4)), maxseg=int(rng.integers(5, 400)))
        mods = [int(m) for m in np.unique(mod)]
        T = {m: np.nonzero(mod == m)[0] for m in mods}
        ops = {}
        for m in mods:
            L = len(T[m])
            if rng.random() < 0.4 and L >= 2:
                s = int(rng.integers(1, max(2, L // 2) + 1))
                f = FLAGS[int(rng.integers(0, 8))]
                ops[("i", m)] = P.grid_state(C.grid(s, s, *f), L, s, int(rng.integers(0, s)))
            else:
                ops[("i", m)] = _rand_identity_op(rng, L)
        for mq in mods:
            for mk in mods:
                if mq == mk:
                    continue
                r = rng.random()
                L = len(T[mk])
                if r < 0.3:
                    ops[("x", mq, mk)] = P.OpState(C.OP_NONE, C.none(), L=L)
                elif r < 0.6:
                    ops[("x", mq, mk)] = P.OpState(C.OP_DENSE, C.dense(), L=L)
                else:
                    n = int(rng.integers(0, 30))
                    sel = np.sort(rng.choice(L, size=min(n, L), replace=False))
                    ops[("x", mq, mk)] = P.OpState(C.OP_VERT, C.vert(n), vsel=sel, L=L)
        hp = P.assemble(C.HEAD_2D, S, mod, ops)
        _same(hp)


def test_boundary_heads_reduce_to_global_on_one_modality():
    rng = np.random.default_rng(5)
    S = 777
    for trial in range(6):
        st = _rand_identity_op(rng, S)
        g = P.assemble(C.HEAD_GLOBAL, S, None, {"g": st})
        q = P.assemble(C.HEAD_QBOUNDARY, S, None, {("q", 0): st})
        d = P.assemble(C.HEAD_2D, S, None, {("i", 0): st})
        for hp in (q, d):
            assert np.array_equal(hp.qperm, g.qperm)
            assert all(np.array_equal(a, b) for a, b in zip(hp.blocks, g.blocks))
    st = P.grid_state(C.grid(13, 13), S, 13, 5)
    g = P.assemble(C.HEAD_GLOBAL, S, None, {"g": st})
    d = P.assemble(C.HEAD_2D, S, None, {("i", 0): st})
    assert np.array_equal(d.qperm, g.qperm) and np.array_equal(d.kperm, g.kperm)
    assert all(np.array_equal(a, b) for a, b in zip(d.blocks, g.blocks))


def test_2d_all_dense_pairs_is_dense_attention_mask():
    rng = np.random.default_rng(6)
    S = 900
    mod = _random_layout(rng, S, nmod=3, maxseg=200)
    mods = [int(m) for m in np.unique(mod)]
    T = {m: np.nonzero(mod == m)[0] for m in mods}
    ops = {("i", m): P.OpState(C.OP_DENSE, C.dense(), L=len(T[m])) for m in mods}
    ops.update({("x", a, b): P.OpState(C.OP_DENSE, C.dense(), L=len(T[b]))
                for a in mods for b in mods if a != b})
    hp = P.assemble(C.HEAD_2D, S, mod, ops)
    for q in rng.choice(S, 50, replace=False):
        assert np.array_equal(P.element_mask_row(hp, int(q)), np.arange(q + 1))


def test_permutations_are_bijections():
    rng = np.random.default_rng(7)
    S = 1000
    mod = _random_layout(rng, S, nmod=2, maxseg=150)
    T = {m: np.nonzero(mod == m)[0] for m in (0, 1)}
    ops = {("i", 0): P.OpState(C.OP_DENSE, C.dense(), L=len(T[0])),
           ("i", 1): P.grid_state(C.grid(7, 7), len(T[1]), 7, 2),
           ("x", 0, 1): P.OpState(C.OP_DENSE, C.dense(), L=len(T[1])),
           ("x", 1, 0): P.OpState(C.OP_NONE, C.none(), L=len(T[0]))}
    for kind, o in [(C.HEAD_2D, ops),
                    (C.HEAD_QBOUNDARY, {("q", 0): ops[("i", 0)], ("q", 1): ops[("i", 0)]})]:
        hp = P.assemble(kind, S, mod, o)
        for perm in (hp.qperm, hp.kperm):
            assert len(perm) % 64 == 0
            live = perm[perm >= 0]
            assert sorted(live.tolist()) == list(range(S))
            # unpermute(permute(x)) == x
            x = np.random.default_rng(0).random(S)
            y = np.zeros(len(perm))
            y[perm >= 0] = x[live]
            back = np.zeros(S)
            back[live] = y[perm >= 0]
            assert np.array_equal(back, x)


def test_static_baselines_closed_form_and_reductions():
    """Sparse Transformer fixed / strided and Tri-shape (Section 4.1 baselines):
    closed forms == lift over small and frame-sized parameters, and the
    reductions that make them dense or A-shape."""
    for L in (300, 1000, 64 * 9 + 5):
        for seg, stride in [(64, 64), (100, 7), (1, 1), (256, 256), (33, 200), (L + 3, 50)]:
            _same(_id_plan(L, P.OpState(C.OP_SF_FIXED, C.sf_fixed(seg, stride), L=L)))
        for local, stride in [(64, 64), (100, 7), (1, 1), (256, 256), (10, 130), (5, L + 1)]:
            _same(_id_plan(L, P.OpState(C.OP_SF_STRIDED, C.sf_strided(local, stride), L=L)))
        for sink, local, bottom in [(128, 256, 128), (0, 64, 0), (7, 1, 500), (0, 0, 1), (200, 0, 64)]:
            _same(_id_plan(L, P.OpState(C.OP_TRISHAPE, C.trishape(sink, local, bottom), L=L)))
        dense = [np.arange(i + 1) for i in range((L + 63) // 64)]
        for st in (P.OpState(C.OP_SF_FIXED, C.sf_fixed(L, 1), L=L),          # one segment / every key a head
                   P.OpState(C.OP_SF_STRIDED, C.sf_strided(1, 1), L=L),       # every distance
                   P.OpState(C.OP_TRISHAPE, C.trishape(0, 0, L), L=L)):       # every query is final
            hp = _id_plan(L, st)
            assert all(np.array_equal(a, b) for a, b in zip(hp.blocks, dense)), st.kind
        a = _id_plan(L, P.OpState(C.OP_ASHAPE, C.ashape(128, 256), L=L))
        t = _id_plan(L, P.OpState(C.OP_TRISHAPE, C.trishape(128, 256, 0), L=L))
        assert all(np.array_equal(x, y) for x, y in zip(a.blocks, t.blocks))


def test_static_baselines_known_blocks():
    """Hand-derived block sets at S = 512 (8 blocks of 64)."""
    L = 512
    # fixed, segment = stride = 128: own two-block segment (causal) + block 0 and 2, 4, 6 (heads)
    hp = _id_plan(L, P.OpState(C.OP_SF_FIXED, C.sf_fixed(128, 128), L=L))
    assert [b.tolist() for b in hp.blocks] == [[0], [0, 1], [0, 2], [0, 2, 3], [0, 2, 4], [0, 2, 4, 5],
                                              [0, 2, 4, 6], [0, 2, 4, 6, 7]]
    # strided, local 64, stride 192: block 7 (q in [448, 511]) sees keys q-63..q (blocks 6, 7),
    # q-192 (block 4) and q-384 (block 1)
    hp = _id_plan(L, P.OpState(C.OP_SF_STRIDED, C.sf_strided(64, 192), L=L))
    assert hp.blocks[7].tolist() == [1, 4, 6, 7]
    assert hp.blocks[3].tolist() == [0, 2, 3]
    # Tri-shape sink 64, local 64, bottom 64: the last block sees everything
    hp = _id_plan(L, P.OpState(C.OP_TRISHAPE, C.trishape(64, 64, 64), L=L))
    assert hp.blocks[7].tolist() == list(range(8))
    assert hp.blocks[5].tolist() == [0, 4, 5]


def _rand_qb_grid_ops(rng, S, mod):
    """Per modality: a Grid state on global positions (some resolved to the
    dense fallback) or a random identity-order op."""
    ops = {}
    for m in np.unique(mod).tolist():
        r = rng.random()
        if r < 0.45:
            s = int(rng.integers(1, min(70, S // 2) + 1))
            f = FLAGS[int(rng.integers(0, 8))]
            ops[("q", m)] = P.grid_state(C.grid(s, s, *f), S, s, int(rng.integers(0, s)))
        elif r < 0.55:
            ops[("q", m)] = P.OpState(C.OP_DENSE, C.grid(4, 8), L=S)       # Grid search found no stride
        else:
            ops[("q", m)] = _rand_identity_op(rng, S)
    return ops


def test_qboundary_grid_closed_form_random_layouts():
    """Q-Boundary heads with Grid modalities: closed forms == literal lift,
    key layouts (position order first when some modality is not Grid, then
    one Grid order per Grid modality) and per-block layout confinement."""
    rng = np.random.default_rng(11)
    for trial in range(30):
        S = int(rng.integers(150, 1400))
        mod = _random_layout(rng, S, nmod=int(rng.integers(2, 4)), maxseg=int(rng.integers(5, 400)))
        ops = _rand_qb_grid_ops(rng, S, mod)
        hp = P.assemble(C.HEAD_QBOUNDARY, S, mod, ops)
        _same(hp)
        nb = (S + 63) // 64
        mods = sorted(ops)
        grid_mods = [m for (_, m) in mods if ops[("q", m)].op.kind == C.OP_GRID]
        nlay = len(grid_mods) + (len(grid_mods) < len(mods))
        assert len(hp.kperm) == nlay * nb * 64
        for ell in range(nlay):
            seg = hp.kperm[ell * nb * 64:(ell + 1) * nb * 64]
            assert sorted(seg[seg >= 0].tolist()) == list(range(S))
        for i, bs in enumerate(hp.blocks):
            m = P._group_of_block(hp, i)[0]
            assert ((bs >= hp.kbase[m]) & (bs < hp.kbase[m] + nb)).all()


def test_qboundary_grid_query_order_and_global_reduction():
    """A Grid modality's queries follow the Grid order of all positions
    restricted to that modality; with one modality the head is the global
    Grid head (same permutations, same blocks)."""
    rng = np.random.default_rng(12)
    for trial in range(10):
        S = int(rng.integers(200, 1200))
        mod = _random_layout(rng, S, nmod=3, maxseg=250)
        s = int(rng.integers(2, 50))
        st = P.grid_state(C.grid(s, s), S, s, int(rng.integers(0, s)))
        mg = int(mod[-1])
        ops = {("q", m): (st if m == mg else P.OpState(C.OP_DENSE, C.dense(), L=S)) for m in np.unique(mod).tolist()}
        hp = P.assemble(C.HEAD_QBOUNDARY, S, mod, ops)
        assert np.array_equal(hp.groups[mg][1], st.cos[mod[st.cos] == mg])
    for s, p in ((1, 0), (7, 3), (64, 63), (100, 17)):
        for f in FLAGS:
            st = P.grid_state(C.grid(s, s, *f), 900, s, p)
            g = P.assemble(C.HEAD_GLOBAL, 900, None, {"g": st})
            q = P.assemble(C.HEAD_QBOUNDARY, 900, None, {("q", 0): st})
            assert np.array_equal(q.qperm, g.qperm) and np.array_equal(q.kperm, g.kperm)
            assert all(np.array_equal(a, b) for a, b in zip(q.blocks, g.blocks))


def test_qboundary_grid_known_blocks():
    """Hand-derived: S = 256, modality 0 on [0, 64), modality 1 on [64, 256)
    with Grid sigma = 2, phase 1, vertical lines only. Keys in Grid order:
    phase 0 (even positions) in slots 0..127, phase 1 (odd) in 128..255.
    Modality-1 queries: even positions 64..254 (slots 0..95 of its group),
    then odd 65..255. Query block 0 (even 64..190): own keys at slots 32..95
    -> key blocks 0, 1; vertical (odd keys <= 190, slots 128..222) -> 2, 3.
    Block 1 (even 192..254, odd 65..127): own keys at slots 96..127 and
    160..191 -> key blocks 1, 2; vertical (odd keys <= 254) -> 2, 3."""
    S = 256
    mod = np.array([0] * 64 + [1] * 192, dtype=np.uint8)
    st = P.grid_state(C.grid(2, 2, h=False, v=True, s=False), S, 2, 1)
    ops = {("q", 0): P.OpState(C.OP_ASHAPE, C.ashape(0, 64), L=S), ("q", 1): st}
    hp = P.assemble(C.HEAD_QBOUNDARY, S, mod, ops)
    assert hp.kbase == {0: 0, 1: 4}
    assert hp.blocks[0].tolist() == [0]
    assert hp.blocks[1].tolist() == [4 + 0, 4 + 1, 4 + 2, 4 + 3]
    assert hp.blocks[2].tolist() == [4 + 1, 4 + 2, 4 + 3]
    _same(hp)
