"""Modality-aware sparse pattern search (Appendix A, Algorithm 4; Appendix
C.5), one head, fp64. Test infrastructure: the reference the GPU search is
checked against.

Reading (the paper gives the three steps, the search space and the FLOPs
target; the rest is stated here):
  * cost of a configuration over a set of query blocks = the number of
    selected blocks there (the work the kernel runs: "kernel-aware"); a
    candidate is admissible iff its cost does not exceed the budget, the
    cost of the target pattern A-shape(1024 sink, 4096 local) over the same
    query blocks in the same coordinates;
  * error = sum over the decided rows of the squared difference between
    the candidate's attention output and the reference output (the search
    scores candidates on the attention output, V included);
  * choice = the admissible candidate of smallest error, the earlier one in
    table order on equal error; no admissible candidate -> the target
    pattern itself.
The candidate lists and the target are inputs (synth/search_space.py holds
the paper's; tests at small S pass scaled-down ones).
Steps:
  1. intra (per modality m, modality-local coordinates): 2D-Boundary heads
     whose cross pairs select nothing; candidate c on every modality at once
     (rows of m depend only on m's intra op); reference: every intra op
     dense. Decided rows: T_m.
  2. cross (per ordered pair (a, b)): 2D-Boundary heads with the step-1
     intra ops, candidate x on the pairs (a, (a + k) mod n) for one k at a
     time, every other pair dense; reference: dense causal attention. Cost =
     the pair's blocks; budget = step-1 budget of a minus the cost of a's
     chosen intra op (no keys is always admissible).
  3. inter: the best global op (the intra candidates over all rows, budget
     the global target pattern; No-Boundary and K-Boundary heads are this
     kind), the Q-Boundary head with the step-1 ops in global positions, the
     2D-Boundary head with the step-1 and step-2 ops; the admissible one of
     smallest error over all rows (order global, Q-Boundary, 2D-Boundary on
     ties), else the one of smallest cost.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from synth import config as C

from . import attention, layout, plan

B = plan.B


@dataclass
class Cand:
    name: str
    cost: dict          # key (modality, pair or "all") -> selected blocks
    err: dict           # same keys -> sum of squared output differences


@dataclass
class Report:
    budget1: dict = field(default_factory=dict)      # m -> budget (step 1)
    step1: list = field(default_factory=list)        # [Cand]
    intra: dict = field(default_factory=dict)        # m -> (name, op)
    step2: dict = field(default_factory=dict)        # k -> [Cand]
    cross: dict = field(default_factory=dict)        # (a, b) -> (name, op)
    budget3: int = 0
    step3_global: list = field(default_factory=list)
    global_op: tuple = None                          # (name, op)
    step3: list = field(default_factory=list)        # [Cand] for global, qboundary, 2d
    kind: str = ""
    own: dict = field(default_factory=dict)          # this search's own picks where others were adopted


def _run(cfg, S, mod, Q, K, V):
    hp = plan.plan_head(cfg, S, mod, lambda r: Q[r], K)
    O, _ = attention.permuted_blockwise(hp, Q, K, V)
    return hp, O


def _block_modality(hp, i):
    return plan._group_of_block(hp, i)[0]


def _costs_by_modality(hp):
    out = {}
    for i, bs in enumerate(hp.blocks):
        m = _block_modality(hp, i)
        out[m] = out.get(m, 0) + len(bs)
    return out


def _pair_cost(hp, a, b):
    off, arr = hp.groups[b]
    lo, hi = off // B, off // B + (len(arr) + B - 1) // B
    tot = 0
    for i, bs in enumerate(hp.blocks):
        if _block_modality(hp, i) == a:
            tot += int(((bs >= lo) & (bs < hi)).sum())
    return tot


def _sqerr(O, R, rows):
    d = O[rows] - R[rows]
    return float((d * d).sum())


def _pick(cands, key, budget):
    best = None
    for c in cands:
        if c.cost[key] <= budget and (best is None or c.err[key] < best.err[key]):
            best = c
    return best


def search_head(Q, K, V, S: int, modality, cands, xc, target, adopt=None):
    """Q, K, V: fp64 [S, D] of one head; cands / xc: [(name, op)] intra and
    cross candidates in table order; target: the FLOPs target op. Returns
    (HeadCfg, Report).

    adopt (for comparing another implementation step by step): choices to
    carry into the later steps instead of this search's own picks, as
    {("intra", m): name, ("cross", a, b): name, "global": name, "kind":
    name}; each own pick that differs is kept in Report.own under the same
    key, and every step is still scored here."""
    adopt = adopt or {}

    def take(key, own_name):
        if key in adopt and adopt[key] != own_name:
            rep.own[key] = own_name
            return adopt[key]
        return own_name
    mod = layout.modality_array(S, modality)
    T = layout.positions_of(mod)
    mods = sorted(T)
    n = len(mods)
    rep = Report()
    none_all = {(a, b): C.none() for a in mods for b in mods if a != b}
    dense_all = {(a, b): C.dense() for a in mods for b in mods if a != b}

    # step 1: intra-modality search
    _, ref1 = _run(C.boundary2d_head({m: C.dense() for m in mods}, none_all), S, mod, Q, K, V)
    hp_b, _ = _run(C.boundary2d_head({m: target for m in mods}, none_all), S, mod, Q, K, V)
    rep.budget1 = _costs_by_modality(hp_b)
    for name, op in cands:
        hp, O = _run(C.boundary2d_head({m: op for m in mods}, none_all), S, mod, Q, K, V)
        cost = _costs_by_modality(hp)
        rep.step1.append(Cand(name, cost, {m: _sqerr(O, ref1, T[m]) for m in mods}))
    ops1 = dict(cands, target=target)
    for m in mods:
        c = _pick(rep.step1, m, rep.budget1[m])
        name = take(("intra", m), c.name if c else "target")
        rep.intra[m] = (name, ops1[name])
    intra = {m: rep.intra[m][1] for m in mods}

    # step 2: cross-modality search
    dense_head = C.global_head(C.dense())
    _, ref = _run(dense_head, S, mod, Q, K, V)
    hp_i, _ = _run(C.boundary2d_head(intra, none_all), S, mod, Q, K, V)
    intra_cost = _costs_by_modality(hp_i)
    for k in range(1, n):
        rep.step2[k] = []
        for name, op in xc:
            cross = dict(dense_all)
            for ai, a in enumerate(mods):
                cross[(a, mods[(ai + k) % n])] = op
            hp, O = _run(C.boundary2d_head(intra, cross), S, mod, Q, K, V)
            cost = {a: _pair_cost(hp, a, mods[(ai + k) % n]) for ai, a in enumerate(mods)}
            rep.step2[k].append(Cand(name, cost, {a: _sqerr(O, ref, T[a]) for a in mods}))
        for ai, a in enumerate(mods):
            b = mods[(ai + k) % n]
            c = _pick(rep.step2[k], a, rep.budget1[a] - intra_cost[a])
            name = take(("cross", a, b), c.name if c else "none")
            rep.cross[(a, b)] = (name, dict(xc, none=C.none())[name])
    cross = {ab: v[1] for ab, v in rep.cross.items()}

    # step 3: inter-modality search
    allrows = np.arange(S)
    hp_g, _ = _run(C.global_head(target), S, mod, Q, K, V)
    rep.budget3 = sum(len(b) for b in hp_g.blocks)
    for name, op in cands:
        hp, O = _run(C.global_head(op), S, mod, Q, K, V)
        rep.step3_global.append(Cand(name, {"all": sum(len(b) for b in hp.blocks)},
                                     {"all": _sqerr(O, ref, allrows)}))
    c = _pick(rep.step3_global, "all", rep.budget3)
    name = take("global", c.name if c else "target")
    rep.global_op = (name, ops1[name])
    heads = [("global", C.global_head(rep.global_op[1])), ("qboundary", C.qboundary_head(intra)),
             ("2d", C.boundary2d_head(intra, cross))]
    for name, cfg in heads:
        hp, O = _run(cfg, S, mod, Q, K, V)
        rep.step3.append(Cand(name, {"all": sum(len(b) for b in hp.blocks)}, {"all": _sqerr(O, ref, allrows)}))
    c = _pick(rep.step3, "all", rep.budget3)
    if c is None:
        c = min(rep.step3, key=lambda x: x.cost["all"])
    rep.kind = take("kind", c.name)
    return dict(heads)[rep.kind], rep
