"""Modality-aware sparse pattern search (Appendix A, Algorithm 4) on the GPU
path: every candidate is a plan built and executed by libmmi, scored by the
library's output-difference kernel (mmi_output_sqerr), and costed by the
blocks its plan selects (the work the attention kernel runs). All heads of
the layer are searched together: each plan carries one configuration per
head.

Rules (Appendix A and C.5; the parts the paper leaves open are readings):
  * cost of a configuration over a set of query blocks = the selected
    blocks there; admissible iff it does not exceed the cost of the FLOPs
    target pattern (A-shape with 1k sink and 4k local tokens) over the same
    query blocks in the same coordinates;
  * error = sum over the decided rows of the squared difference between the
    candidate's output and the reference output;
  * choice = admissible candidate of smallest error (earlier in table order
    on equal error); none admissible -> the target pattern.
  1. intra, per modality m (modality-local coordinates): 2D-Boundary heads
     whose cross pairs select nothing, the candidate on every modality at
     once; reference: every intra op dense; rows: modality m.
  2. cross, per ordered pair (a, b): 2D-Boundary heads with the chosen intra
     ops, the candidate on the pairs (a, (a + k) mod n) for one k at a time,
     the other pairs dense; reference: dense causal attention; cost: the
     pair's blocks; budget: a's intra budget minus its chosen intra cost.
  3. inter: the best global op (No-/K-Boundary), the Q-Boundary head with the
     chosen intra ops, the 2D-Boundary head with the chosen intra and cross
     ops; smallest error over all rows among those within the global target
     cost (order global, Q-Boundary, 2D on ties), else the cheapest.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List

import numpy as np
import torch

from synth import config as C

from . import mmi


@dataclass
class Scored:
    name: str
    cost: Dict
    err: Dict


@dataclass
class HeadSearch:
    budget1: Dict = field(default_factory=dict)
    step1: List[Scored] = field(default_factory=list)
    intra: Dict = field(default_factory=dict)          # m -> (name, op)
    step2: Dict = field(default_factory=dict)          # k -> [Scored]
    cross: Dict = field(default_factory=dict)          # (a, b) -> (name, op)
    budget3: int = 0
    step3_global: List[Scored] = field(default_factory=list)
    global_op: tuple = None
    step3: List[Scored] = field(default_factory=list)
    kind: str = ""


class _Runner:
    """Plans one configuration per head, executes it, and reads back costs."""

    def __init__(self, ctx, S, Hq, Hkv, modality, q, k, v, stream):
        self.ctx, self.S, self.Hq, self.q, self.k, self.v, self.stream = ctx, S, Hq, q, k, v, stream
        self.mod = np.zeros(S, np.uint8) if modality is None else np.asarray(modality, np.uint8)
        self.mods = sorted(int(m) for m in np.unique(self.mod))
        self.cls_of = {m: i for i, m in enumerate(self.mods)}
        cls = np.array([self.cls_of.get(m, 255) for m in range(256)], np.uint8)[self.mod]
        self.cls = torch.as_tensor(cls, device=q.device)
        self.prob = mmi.Problem(S, Hq, Hkv, modality)
        self.err_out = torch.empty(Hq * len(self.mods), dtype=torch.float64, device=q.device)
        self.plans = 0

    def run(self, heads):
        """-> (O, costs): costs[h] = {"all": n, m: n, ("pair", a, b): n}, the
        selected blocks of the head, of modality m's query blocks, and of m's
        query blocks against b's key blocks (from the plan's statistics)."""
        plan = mmi.Plan(self.ctx, self.prob, heads, self.q, self.k, self.stream)
        o = torch.empty_like(self.q)
        plan.execute(self.q, self.k, self.v, o, None, self.stream)
        self.plans += 1
        costs = []
        try:
            for h in range(self.Hq):
                st = plan.stats(h)
                bm = st.blocks_by_modality
                c = {"all": int(st.nnz_blocks)}
                for a in self.mods:
                    c[a] = sum(int(bm[a][b]) for b in range(mmi.MAXM))
                    for b in self.mods:
                        c[("pair", a, b)] = int(bm[a][b])
                costs.append(c)
        finally:
            plan.destroy()
        return o, costs

    def sqerr(self, o, ref):
        """err[h] = {m: squared difference over modality m's rows, "all": total}."""
        mmi.mmi_output_sqerr(self.prob, o, ref, self.cls, len(self.mods), self.err_out, self.stream)
        e = self.err_out.cpu().numpy().reshape(self.Hq, len(self.mods))
        out = []
        for h in range(self.Hq):
            d = {m: float(e[h, i]) for i, m in enumerate(self.mods)}
            tot = 0.0
            for m in self.mods:
                tot += d[m]
            d["all"] = tot
            out.append(d)
        return out


def _choose(scored: List[Scored], key, budget):
    best = None
    for s in scored:
        if s.cost[key] <= budget and (best is None or s.err[key] < best.err[key]):
            best = s
    return best


def search(ctx, S, Hq, Hkv, modality, q, k, v, cands, xc, target, stream=None):
    """Algorithm 4 for every head of one layer on a calibration sample.

    q, k, v: device bf16 [S, H, 128]; cands / xc: [(name, op)] intra and
    cross candidates in table order; target: the FLOPs target op.
    Returns ([HeadCfg] per head, [HeadSearch] per head, plans built)."""
    R = _Runner(ctx, S, Hq, Hkv, modality, q, k, v, stream)
    mods, n = R.mods, len(R.mods)
    reps = [HeadSearch() for _ in range(Hq)]
    none_all = {(a, b): C.none() for a in mods for b in mods if a != b}
    dense_all = {(a, b): C.dense() for a in mods for b in mods if a != b}
    cand_op, xc_op = dict(cands), dict(xc)

    # 1. intra-modality
    ref1, _ = R.run([C.boundary2d_head({m: C.dense() for m in mods}, none_all)] * Hq)
    _, bc = R.run([C.boundary2d_head({m: target for m in mods}, none_all)] * Hq)
    for h in range(Hq):
        reps[h].budget1 = {m: bc[h][m] for m in mods}
    for name, op in cands:
        o, cc = R.run([C.boundary2d_head({m: op for m in mods}, none_all)] * Hq)
        ee = R.sqerr(o, ref1)
        for h in range(Hq):
            reps[h].step1.append(Scored(name, {m: cc[h][m] for m in mods}, {m: ee[h][m] for m in mods}))
    for h in range(Hq):
        for m in mods:
            s = _choose(reps[h].step1, m, reps[h].budget1[m])
            reps[h].intra[m] = (s.name, cand_op[s.name]) if s else ("target", target)
    intra = [{m: reps[h].intra[m][1] for m in mods} for h in range(Hq)]
    del ref1

    # 2. cross-modality
    ref, _ = R.run([C.global_head(C.dense())] * Hq)
    _, ic = R.run([C.boundary2d_head(intra[h], none_all) for h in range(Hq)])
    for kk in range(1, n):
        for h in range(Hq):
            reps[h].step2[kk] = []
        for name, op in xc:
            heads = []
            for h in range(Hq):
                cross = dict(dense_all)
                for ai, a in enumerate(mods):
                    cross[(a, mods[(ai + kk) % n])] = op
                heads.append(C.boundary2d_head(intra[h], cross))
            o, cc = R.run(heads)
            ee = R.sqerr(o, ref)
            for h in range(Hq):
                cost = {a: cc[h][("pair", a, mods[(ai + kk) % n])] for ai, a in enumerate(mods)}
                reps[h].step2[kk].append(Scored(name, cost, {a: ee[h][a] for a in mods}))
        for h in range(Hq):
            for ai, a in enumerate(mods):
                b = mods[(ai + kk) % n]
                s = _choose(reps[h].step2[kk], a, reps[h].budget1[a] - ic[h][a])
                reps[h].cross[(a, b)] = (s.name, xc_op[s.name]) if s else ("none", C.none())
    cross = [{ab: v2[1] for ab, v2 in reps[h].cross.items()} for h in range(Hq)]

    # 3. inter-modality
    _, gc = R.run([C.global_head(target)] * Hq)
    for h in range(Hq):
        reps[h].budget3 = gc[h]["all"]
    for name, op in cands:
        o, cc = R.run([C.global_head(op)] * Hq)
        ee = R.sqerr(o, ref)
        for h in range(Hq):
            reps[h].step3_global.append(Scored(name, {"all": cc[h]["all"]}, {"all": ee[h]["all"]}))
    for h in range(Hq):
        s = _choose(reps[h].step3_global, "all", reps[h].budget3)
        reps[h].global_op = (s.name, cand_op[s.name]) if s else ("target", target)
    kinds = {
        "global": [C.global_head(reps[h].global_op[1]) for h in range(Hq)],
        "qboundary": [C.qboundary_head(intra[h]) for h in range(Hq)],
        "2d": [C.boundary2d_head(intra[h], cross[h]) for h in range(Hq)],
    }
    for kind, heads in kinds.items():
        o, cc = R.run(heads)
        ee = R.sqerr(o, ref)
        for h in range(Hq):
            reps[h].step3.append(Scored(kind, {"all": cc[h]["all"]}, {"all": ee[h]["all"]}))
    out = []
    for h in range(Hq):
        s = _choose(reps[h].step3, "all", reps[h].budget3)
        if s is None:
            s = min(reps[h].step3, key=lambda x: x.cost["all"])
        reps[h].kind = s.name
        out.append(kinds[s.name][h])
    return out, reps, R.plans
