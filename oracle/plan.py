"""Per-head plan: estimation -> choices -> permutations -> selected blocks.

A head plan is (qperm, kperm, BS): qperm[x] / kperm[x] give the original
position held by query / key slot x (-1 for padding), and BS[i] is the
ascending list of key blocks selected for query block i (block size B = 64).

Block semantics ("sparse loading, dense computation", Figure
"dynamic_sparse_pipelines"; Algorithms 5-7 load whole B x B blocks): block
(i, j) is selected iff some query of block i and key of block j satisfy
k <= q (original positions) and the head's token predicate, or j is the key
block holding the diagonal element of one of block i's queries (every row
keeps its own key). Every causal element inside a selected block is computed.

Head kinds (Sections 3.1-3.2):
  * global op (No-Boundary / K-Boundary heads, applied to all rows):
    dense, A-shape, Vertical-Slash (identity order) or Grid (Algorithm 1:
    permuted by phase), or one of the static baselines of Section 4.1
    (Sparse Transformer fixed / strided, Tri-shape; identity order), or
    neighborhood attention over a token grid (Appendix F; tile order,
    bidirectional: the only head without the causal condition);
  * Q-Boundary (Algorithm 2): queries grouped by modality (each group padded
    to a multiple of B); each modality's queries use their own op in global
    positions, estimated from that modality's final queries. A Grid modality
    (stride and phase searched on global positions) orders its queries by
    phase (group order p+1, ..., p, position order inside a phase) and reads
    the keys in the Grid order of all S positions (Algorithm 5's strided key
    loads). Keys therefore come in key layouts: the position order (if some
    modality is not Grid) followed by one Grid order per Grid modality in
    ascending modality id, each padded to a multiple of B and concatenated;
    a query block only selects key blocks of its modality's layout;
  * 2D-Boundary (Algorithm 3): queries and keys grouped by modality; inside a
    group tokens are in Grid order when that modality's op is Grid, else in
    position order; each (query modality, key modality) pair has its own op:
    intra pairs use the modality op in modality-local coordinates, cross pairs
    are none, dense, or VERT(n) (the n best key columns of that modality,
    estimated from the query modality's final queries). One softmax per row
    over all pairs (Algorithm 7 carries m and l across key modalities).

Block sets are built two independent ways: closed forms per op (used at every
size) and the literal lift by enumerating token pairs (lift_blocks, used by
the tests at small S to pin the closed forms).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from synth import config as C

from . import estimate, grid, layout, natten, vslash

B = 64


def blk(x):
    return x // B


def pad_to_block(arr):
    n = len(arr)
    npad = (-n) % B
    return np.concatenate([arr, np.full(npad, -1, dtype=np.int64)]) if npad else arr


@dataclass
class Est:
    rows: np.ndarray
    L_c: int
    lse: np.ndarray
    v: np.ndarray
    u: object


@dataclass
class OpState:
    """A resolved op in one coordinate system (kind may have fallen back to dense)."""
    kind: int
    op: C.Op
    sigma: int = 0
    p: int = 0
    vsel: object = None      # selected vertical coordinates
    ssel: object = None      # selected slash offsets
    cos: object = None       # grid: coordinate of slot (local slot space)
    g0: object = None        # grid: group start slot per phase
    L: int = 0               # extent of the coordinate system
    minc: object = None      # smallest coordinate / admitted position per key block (cache)


@dataclass
class HeadPlan:
    kind: int
    S: int
    qperm: np.ndarray
    kperm: np.ndarray
    blocks: list = field(default_factory=list)
    est: dict = field(default_factory=dict)          # key -> Est
    ops: dict = field(default_factory=dict)          # key -> OpState
    folds: dict = field(default_factory=dict)        # key -> {sigma: fp32 fold}
    groups: dict = field(default_factory=dict)       # m -> (slot offset, T_m in group order)
    kbase: dict = field(default_factory=dict)        # Q-Boundary: m -> first key block of its layout
    mod: object = None
    causal: bool = True                              # False only for neighborhood attention

    @property
    def nbq(self):
        return len(self.qperm) // B

    @property
    def nbk(self):
        return len(self.kperm) // B


# --------------------------------------------------------------------------
# estimation + choices

def _estimate(q_rows, K, rows, scale, key_pos, row_coord):
    Qr = q_rows(rows)
    lse = estimate.row_lse(Qr, K, rows, scale)
    v, u, L_c = estimate.scores(Qr, K, rows, lse, scale, key_pos, row_coord)
    return Est(rows, L_c, lse, v, u)


def _resolve(op: C.Op, L: int, e: Est | None, folds_out: dict | None) -> OpState:
    """Take the op's discrete choices from the estimate (fp32 decisions)."""
    if op.kind == C.OP_GRID:
        best, folds, _ = grid.search(e.v, e.L_c, op.stride_lo, op.stride_hi)
        if folds_out is not None:
            folds_out.update(folds)
        if best is None:
            return OpState(C.OP_DENSE, op, L=L)
        s, p = best
        cos, g0 = grid.permutation(L, s, p)
        return OpState(C.OP_GRID, op, sigma=s, p=p, cos=cos, g0=g0, L=L)
    if op.kind == C.OP_VSLASH:
        vs = vslash.topk(e.v, op.n_vertical, e.L_c)
        ss = vslash.topk(e.u, op.n_slash, e.L_c)
        return OpState(C.OP_VSLASH, op, vsel=vs, ssel=ss, L=L)
    if op.kind == C.OP_VERT:
        return OpState(C.OP_VERT, op, vsel=vslash.topk(e.v, op.n_vertical, e.L_c), L=L)
    return OpState(op.kind, op, L=L)


def grid_state(op: C.Op, L: int, sigma: int, p: int) -> OpState:
    cos, g0 = grid.permutation(L, sigma, p)
    return OpState(C.OP_GRID, op, sigma=sigma, p=p, cos=cos, g0=g0, L=L)


def adopt(st: OpState, sigma=None, p=None, vsel=None, ssel=None) -> OpState:
    """The op with the given discrete choices in place of its estimated ones:
    a Grid stride and phase (sigma 0 = no stride, dense fallback), or the
    selected vertical coordinates / slash offsets. Used when another
    implementation's choice differs from this one's only inside a tie."""
    op = st.op
    if op.kind == C.OP_GRID:
        if int(sigma) == 0:
            return OpState(C.OP_DENSE, op, L=st.L)
        return grid_state(op, st.L, int(sigma), int(p))
    if op.kind == C.OP_VSLASH:
        return OpState(C.OP_VSLASH, op, vsel=np.asarray(vsel, dtype=np.int64),
                       ssel=np.asarray(ssel, dtype=np.int64), L=st.L)
    if op.kind == C.OP_VERT:
        return OpState(C.OP_VERT, op, vsel=np.asarray(vsel, dtype=np.int64), L=st.L)
    raise ValueError(f"op kind {op.kind} has no estimated choice")


def choose(cfg: C.HeadCfg, S: int, modality, q_rows, K: np.ndarray, scale=None):
    """Estimation and discrete choices of one head.

    q_rows(positions) -> fp64 [n,128] query rows of this head; K fp64 [S,128]
    (the head's KV head). Returns (ops, est, folds) keyed by
    "g" (global op), ("q", m) (Q-Boundary modality m), ("i", m) (2D intra),
    ("x", mq, mk) (2D cross pair)."""
    scale = estimate.tau(K.shape[1]) if scale is None else scale
    mod = layout.modality_array(S, modality)
    ops, est, folds = {}, {}, {}
    if cfg.kind == C.HEAD_GLOBAL:
        op = cfg.op
        e = None
        if op.kind in (C.OP_GRID, C.OP_VSLASH):
            rows = layout.global_rows(S)
            e = est["g"] = _estimate(q_rows, K, rows, scale, None, rows)
        folds["g"] = {}
        ops["g"] = _resolve(op, S, e, folds["g"])
        return ops, est, folds
    T = layout.positions_of(mod)
    mods = sorted(T)
    if cfg.kind == C.HEAD_QBOUNDARY:
        for m in mods:
            op = cfg.intra_op(m)
            if op.kind not in C.STATIC_OPS + (C.OP_VSLASH, C.OP_GRID):
                raise NotImplementedError("Q-Boundary intra op must be VS, Grid or a static pattern")
            e = None
            if op.kind in (C.OP_GRID, C.OP_VSLASH):
                rows = layout.final_run_rows(T[m])
                e = est[("q", m)] = _estimate(q_rows, K, rows, scale, None, rows)
            folds[("q", m)] = {}
            ops[("q", m)] = _resolve(op, S, e, folds[("q", m)])
        return ops, est, folds
    if cfg.kind == C.HEAD_2D:
        for m in mods:
            op = cfg.intra_op(m)
            if op.kind not in C.STATIC_OPS + (C.OP_VSLASH, C.OP_GRID):
                raise NotImplementedError("2D intra op must be VS, Grid or a static pattern")
            Tm = T[m]
            e = None
            if op.kind in (C.OP_GRID, C.OP_VSLASH):
                rows = layout.final_run_rows(Tm)
                loc = np.searchsorted(Tm, rows)
                e = est[("i", m)] = _estimate(q_rows, K, rows, scale, Tm, loc)
            folds[("i", m)] = {}
            ops[("i", m)] = _resolve(op, len(Tm), e, folds[("i", m)])
        for mq in mods:
            for mk in mods:
                if mq == mk:
                    continue
                op = cfg.cross_op(mq, mk)
                if op.kind not in (C.OP_NONE, C.OP_DENSE, C.OP_VERT):
                    raise NotImplementedError("2D cross op must be none, dense or VERT")
                e = None
                if op.kind == C.OP_VERT:
                    rows = layout.final_run_rows(T[mq])
                    e = est[("x", mq, mk)] = _estimate(q_rows, K, rows, scale, T[mk], None)
                ops[("x", mq, mk)] = _resolve(op, len(T[mk]), e, None)
        return ops, est, folds
    raise ValueError(f"unknown head kind {cfg.kind}")


def assemble(kind: int, S: int, modality, ops: dict) -> HeadPlan:
    """Permutations and closed-form block sets from resolved ops."""
    mod = layout.modality_array(S, modality)
    hp = HeadPlan(kind, S, None, None, mod=mod, ops=ops)
    if kind == C.HEAD_GLOBAL:
        st = ops["g"]
        if st.kind == C.OP_NATTEN:
            o = st.op
            assert int(np.prod(o.grid)) == S and int(np.prod(o.tile)) == B
            hp.causal = False
            hp.qperm = natten.permutation(o.grid, o.tile)
            hp.kperm = hp.qperm.copy()
            hp.groups[0] = (0, hp.qperm[hp.qperm >= 0])
            hp.blocks = [np.array(natten.tile_blocks(o.grid, o.win, o.tile, i), dtype=np.int64)
                         for i in range(hp.nbq)]
            return hp
        if st.kind == C.OP_GRID:
            perm = pad_to_block(st.cos.copy())
        else:
            perm = pad_to_block(np.arange(S, dtype=np.int64))
        hp.qperm, hp.kperm = perm, perm.copy()
        hp.groups[0] = (0, perm[perm >= 0])
        hp.blocks = [_global_row(hp, st, i) for i in range(hp.nbq)]
        return hp
    T = layout.positions_of(mod)
    parts, off = [], 0
    for m in sorted(T):
        arr = T[m]
        if kind == C.HEAD_2D and ops[("i", m)].kind == C.OP_GRID:
            arr = T[m][ops[("i", m)].cos]
        if kind == C.HEAD_QBOUNDARY and ops[("q", m)].kind == C.OP_GRID:
            st = ops[("q", m)]
            rank = (arr - st.p - 1) % st.sigma          # phase p+1 first, phase p last
            arr = arr[np.lexsort((arr, rank))]
        hp.groups[m] = (off, arr)
        part = pad_to_block(arr.copy())
        parts.append(part)
        off += len(part)
    hp.qperm = np.concatenate(parts)
    if kind == C.HEAD_QBOUNDARY:
        grid_mods = [m for m in sorted(T) if ops[("q", m)].op.kind == C.OP_GRID]
        layouts = ([None] if len(grid_mods) < len(T) else []) + grid_mods
        nb = (S + B - 1) // B
        segs = []
        for m in layouts:
            st = None if m is None else ops[("q", m)]
            order = st.cos if st is not None and st.kind == C.OP_GRID else np.arange(S, dtype=np.int64)
            segs.append(pad_to_block(order.copy()))
        hp.kperm = np.concatenate(segs)
        for m in T:
            hp.kbase[m] = layouts.index(m if m in grid_mods else None) * nb
        hp.blocks = [_qb_row(hp, i) for i in range(hp.nbq)]
    elif kind == C.HEAD_2D:
        hp.kperm = hp.qperm.copy()
        hp.blocks = [_2d_row(hp, i) for i in range(hp.nbq)]
    else:
        raise ValueError(kind)
    return hp


def plan_head(cfg: C.HeadCfg, S: int, modality, q_rows, K: np.ndarray,
              scale=None) -> HeadPlan:
    ops, est, folds = choose(cfg, S, modality, q_rows, K, scale)
    hp = assemble(cfg.kind, S, modality, ops)
    hp.est, hp.folds = est, folds
    return hp


# --------------------------------------------------------------------------
# closed-form block sets

def _runs(coords):
    """Maximal runs of consecutive integers in an ascending array -> [(a, b)]."""
    out = []
    a = prev = int(coords[0])
    for c in coords[1:]:
        c = int(c)
        if c != prev + 1:
            out.append((a, prev))
            a = c
        prev = c
    out.append((a, prev))
    return out


def _identity_op_blocks(st: OpState, runs, kbase: int):
    """Key blocks for dense / A-shape / VS ops whose keys sit in coordinate order
    at key slot kbase*B + coordinate. runs: row coordinates as [(a, b)]."""
    qmax = runs[-1][1]
    out = set()
    if st.kind == C.OP_DENSE or (st.kind == C.OP_TRISHAPE and qmax >= st.L - st.op.bottom):
        out.update(range(0, blk(qmax) + 1))
    elif st.kind in (C.OP_ASHAPE, C.OP_TRISHAPE):
        sink, local = st.op.sink, st.op.local
        if sink > 0:
            out.update(range(0, blk(min(sink - 1, qmax)) + 1))
        if local > 0:
            for a, b in runs:
                out.update(range(blk(max(0, a - local + 1)), blk(b) + 1))
    elif st.kind == C.OP_SF_FIXED:
        seg, stride = st.op.local, st.op.stride_lo
        for a, b in runs:                         # own segment, causal part
            out.update(range(blk(a // seg * seg), blk(b) + 1))
        out.update(blk(np.arange(0, qmax + 1, stride)).tolist())   # segment heads
    elif st.kind == C.OP_SF_STRIDED:
        local, stride = st.op.local, st.op.stride_lo
        for a, b in runs:
            out.update(range(blk(max(0, a - local + 1)), blk(b) + 1))
            m = np.arange(0, b // stride + 1)
            lo, hi = blk(np.maximum(0, a - m * stride)), blk(b - m * stride)
            for x, y in zip(lo.tolist(), hi.tolist()):
                out.update(range(x, y + 1))
    elif st.kind == C.OP_VSLASH:
        out.update(blk(st.vsel[st.vsel <= qmax]).tolist())
        for a, b in runs:
            o = st.ssel[st.ssel <= b]
            lo, hi = blk(np.maximum(0, a - o)), blk(b - o)
            out.update(lo.tolist())
            out.update(hi.tolist())
            for w in np.nonzero(hi - lo > 1)[0]:      # runs longer than one block
                out.update(range(int(lo[w]), int(hi[w]) + 1))
    else:
        raise ValueError(st.kind)
    return {kbase + j for j in out}


def _block_min(st: OpState):
    """Smallest coordinate held by each key block of a grid-ordered group."""
    if st.minc is None:
        L = st.L
        pad = pad_to_block(st.cos.copy())
        big = np.where(pad >= 0, pad, np.iinfo(np.int64).max)
        st.minc = big.reshape(-1, B).min(axis=1)
        assert len(st.minc) == (L + B - 1) // B
    return st.minc


def _grid_blocks(st: OpState, il: int, kbase: int):
    """Grid closed forms in the local slot space [0, L) of one group."""
    L, s, p, cos, g0 = st.L, st.sigma, st.p, st.cos, st.g0
    lo, hi = il * B, min(il * B + B, L) - 1
    out = {il}
    if st.op.use_s:
        out.update(range(blk(int(g0[cos[lo] % s])), il + 1))
    maxc = int(cos[lo:hi + 1].max())
    if st.op.use_v and maxc >= p:
        f = (maxc - p) // s
        out.update(range(blk(int(g0[p])), blk(int(g0[p]) + f) + 1))
    if st.op.use_h and hi >= g0[p]:
        qh = int(cos[hi])
        out.update(np.nonzero(_block_min(st) <= qh)[0].tolist())
    return {kbase + j for j in out}


def _global_row(hp: HeadPlan, st: OpState, i: int):
    S = hp.S
    if st.kind == C.OP_GRID:
        bs = _grid_blocks(st, i, 0)
    else:
        bs = _identity_op_blocks(st, [(i * B, min(i * B + B, S) - 1)], 0)
        bs.add(i)
    return np.array(sorted(bs), dtype=np.int64)


def _group_of_block(hp: HeadPlan, i: int):
    x = i * B
    for m, (off, arr) in hp.groups.items():
        if off <= x < off + len(arr) + ((-len(arr)) % B):
            return m, off, arr
    raise IndexError(i)


def _qb_grid_blocks(st: OpState, rows: np.ndarray, kbase: int):
    """Grid closed forms for query positions `rows` (any set of positions)
    against keys in the Grid order of all S positions: coordinate c sits at
    slot g0[c mod sigma] + c // sigma."""
    s, p, g0 = st.sigma, st.p, st.g0
    ph = rows % s
    out = set(blk(g0[ph] + rows // s).tolist())          # forced: each row's own key
    if st.op.use_s:                                      # same phase, k <= q
        for f in np.unique(ph).tolist():
            qmax = int(rows[ph == f].max())
            out.update(range(blk(int(g0[f])), blk(int(g0[f]) + qmax // s) + 1))
    maxq = int(rows.max())
    if st.op.use_v and maxq >= p:                        # phase-p keys, k <= q
        out.update(range(blk(int(g0[p])), blk(int(g0[p]) + (maxq - p) // s) + 1))
    if st.op.use_h and (ph == p).any():                  # phase-p rows see every k <= q
        qh = int(rows[ph == p].max())
        out.update(np.nonzero(_block_min(st) <= qh)[0].tolist())
    return {kbase + j for j in out}


def _qb_row(hp: HeadPlan, i: int):
    m, off, Tm = _group_of_block(hp, i)
    lo = i * B - off
    rows = Tm[lo:lo + B]
    st = hp.ops[("q", m)]
    kbase = hp.kbase[m]
    if st.kind == C.OP_GRID:
        return np.array(sorted(_qb_grid_blocks(st, rows, kbase)), dtype=np.int64)
    runs = _runs(rows)
    bs = _identity_op_blocks(st, runs, kbase)
    for a, b in runs:                       # forced: each row's own key block
        bs.update(range(kbase + blk(a), kbase + blk(b) + 1))
    return np.array(sorted(bs), dtype=np.int64)


def _cross_block_min(st: OpState, arrk):
    """Per key block of the key group: smallest position of a key the cross op
    admits (every key for dense, the selected columns for VERT). Cached."""
    if st.minc is None:
        big = np.iinfo(np.int64).max
        keys = pad_to_block(arrk.copy())
        if st.kind == C.OP_DENSE:
            cand = np.where(keys >= 0, keys, big)
        elif st.kind == C.OP_VERT:
            selpos = np.sort(arrk)[st.vsel]
            cand = np.where((keys >= 0) & np.isin(keys, selpos), keys, big)
        else:
            raise ValueError(st.kind)
        st.minc = cand.reshape(-1, B).min(axis=1)
    return st.minc


def _2d_row(hp: HeadPlan, i: int):
    mq, offq, arrq = _group_of_block(hp, i)
    il = i - offq // B
    lo = il * B
    rows_pos = arrq[lo:lo + B]
    maxpos = int(rows_pos.max())
    out = {i}
    for mk, (offk, arrk) in hp.groups.items():
        kbase = offk // B
        if mk == mq:
            st = hp.ops[("i", mq)]
            if st.kind == C.OP_GRID:
                out |= _grid_blocks(st, il, kbase)
            else:
                hi = min(lo + B, len(arrq)) - 1
                out |= _identity_op_blocks(st, [(lo, hi)], kbase)
            continue
        st = hp.ops[("x", mq, mk)]
        if st.kind == C.OP_NONE:
            continue
        kmin = _cross_block_min(st, arrk)
        out.update((kbase + np.nonzero(kmin <= maxpos)[0]).tolist())
    return np.array(sorted(out), dtype=np.int64)


# --------------------------------------------------------------------------
# literal lift (small S): enumerate token pairs

def _local_index(hp: HeadPlan):
    """position -> index inside its modality's ascending position list."""
    loc = np.zeros(hp.S, dtype=np.int64)
    for m in np.unique(hp.mod):
        T = np.nonzero(hp.mod == m)[0]
        loc[T] = np.arange(len(T))
    return loc


def _op_pred(st: OpState, qc, kc):
    if st.kind == C.OP_DENSE:
        return np.ones(np.broadcast(qc, kc).shape, dtype=bool)
    if st.kind == C.OP_NONE:
        return np.zeros(np.broadcast(qc, kc).shape, dtype=bool)
    if st.kind == C.OP_ASHAPE:
        return (kc < st.op.sink) | ((qc - kc) < st.op.local)
    if st.kind == C.OP_TRISHAPE:
        return (kc < st.op.sink) | ((qc - kc) < st.op.local) | (qc >= st.L - st.op.bottom)
    if st.kind == C.OP_SF_FIXED:
        return ((qc // st.op.local) == (kc // st.op.local)) | (kc % st.op.stride_lo == 0)
    if st.kind == C.OP_SF_STRIDED:
        return ((qc - kc) < st.op.local) | ((qc - kc) % st.op.stride_lo == 0)
    if st.kind == C.OP_VSLASH:
        return np.isin(kc, st.vsel) | np.isin(qc - kc, st.ssel)
    if st.kind == C.OP_VERT:
        return np.isin(kc, st.vsel) & np.ones_like(qc, dtype=bool)
    if st.kind == C.OP_GRID:
        o = st.op
        return grid.predicate(qc, kc, st.sigma, st.p, o.use_h, o.use_v, o.use_s)
    if st.kind == C.OP_NATTEN:
        return natten.predicate(qc, kc, st.op.grid, st.op.win)
    raise ValueError(st.kind)


def token_predicate(hp: HeadPlan, qpos: np.ndarray, kpos: np.ndarray) -> np.ndarray:
    """pred(q, k) for position arrays (qpos[:, None], kpos[None, :])."""
    qp, kp = qpos[:, None], kpos[None, :]
    if hp.kind == C.HEAD_GLOBAL:
        return _op_pred(hp.ops["g"], qp, kp)
    mod = hp.mod
    out = np.zeros((len(qpos), len(kpos)), dtype=bool)
    if hp.kind == C.HEAD_QBOUNDARY:
        for m in np.unique(mod[qpos]):
            r = mod[qpos] == m
            out[r] = _op_pred(hp.ops[("q", int(m))], qpos[r][:, None], kp)
        return out
    loc = _local_index(hp)
    for mq in np.unique(mod[qpos]):
        r = mod[qpos] == mq
        for mk in np.unique(mod[kpos]):
            c = mod[kpos] == mk
            key = ("i", int(mq)) if mq == mk else ("x", int(mq), int(mk))
            st = hp.ops[key]
            sub = _op_pred(st, loc[qpos[r]][:, None], loc[kpos[c]][None, :])
            out[np.ix_(r, c)] = sub
    return out


def _key_span(hp: HeadPlan, i: int):
    """Key slots [lo, hi) that query block i reads: its modality's key layout
    for a Q-Boundary head, all key slots otherwise."""
    if hp.kind == C.HEAD_QBOUNDARY:
        m = _group_of_block(hp, i)[0]
        nb = (hp.S + B - 1) // B
        return hp.kbase[m] * B, (hp.kbase[m] + nb) * B
    return 0, len(hp.kperm)


def lift_blocks(hp: HeadPlan):
    """BS by enumeration: causal pairs satisfying the predicate, plus each
    row's own key block."""
    spans = {}
    out = []
    for i in range(hp.nbq):
        span = _key_span(hp, i)
        if span not in spans:
            seg = hp.kperm[span[0]:span[1]]
            live = np.nonzero(seg >= 0)[0]
            kslot_of = np.full(hp.S, -1, dtype=np.int64)
            kslot_of[seg[live]] = span[0] + live
            spans[span] = (span[0] + live, seg[live], kslot_of)
        kvalid, kpos, kslot_of = spans[span]
        rows = hp.qperm[i * B:(i + 1) * B]
        rows = rows[rows >= 0]
        m = token_predicate(hp, rows, kpos)
        if hp.causal:
            m &= kpos[None, :] <= rows[:, None]
        hit = kvalid[m.any(axis=0)]
        bs = set(blk(hit).tolist()) | set(blk(kslot_of[rows]).tolist())
        out.append(np.array(sorted(bs), dtype=np.int64))
    return out


def element_mask_row(hp: HeadPlan, q: int) -> np.ndarray:
    """Positions k (ascending) that query position q attends to: every key of
    its selected blocks, causal (k <= q) unless the head is bidirectional."""
    x = int(np.nonzero(hp.qperm == q)[0][0])
    keys = []
    lim = q if hp.causal else hp.S
    for j in hp.blocks[x // B]:
        ks = hp.kperm[j * B:(j + 1) * B]
        keys.append(ks[(ks >= 0) & (ks <= lim)])
    return np.sort(np.concatenate(keys)) if keys else np.zeros(0, np.int64)
