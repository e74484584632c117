"""Modality-aware sparse pattern search (Appendix A, Algorithm 4): the C
call mmi_search runs the whole search in libmmi (every candidate a plan of
the library, scored by its output-difference kernel and costed by the blocks
its plan selects; the rules are stated with the call in include/mmi.h).
This module only marshals: candidates in, and the call's report turned into
per-head records with the candidates' names and the chosen configurations
as head configs.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List

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
    abi_cfg: object = None                             # the chosen mmi_head_cfg as the C call wrote it


_KINDS = ("global", "qboundary", "2d")


def search(ctx, S, Hq, Hkv, modality, q, k, v, cands, xc, target, stream=None):
    """Algorithm 4 for every head of one layer on a calibration sample.

    q, k, v: device bf16 [S, H, 128]; cands / xc: [(name, op)] intra and
    cross candidates in table order; target: the FLOPs target op.
    Returns ([HeadCfg] per head, [HeadSearch] per head, plans built)."""
    prob = mmi.Problem(S, Hq, Hkv, modality)
    cfgs, r = mmi.mmi_search(ctx, prob, q, k, v, [op for _, op in cands], [op for _, op in xc], target, stream)
    mods, n = r["mods"], r["n_mod"]
    pick = lambda lst, i, fallback: (lst[i][0], lst[i][1]) if i >= 0 else fallback
    heads, reps = [], []
    for h in range(Hq):
        g = HeadSearch()
        g.budget1 = {m: int(r["budget1"][h, i]) for i, m in enumerate(mods)}
        g.step1 = [Scored(name, {m: int(r["step1_cost"][h, c, i]) for i, m in enumerate(mods)},
                          {m: float(r["step1_err"][h, c, i]) for i, m in enumerate(mods)})
                   for c, (name, _) in enumerate(cands)]
        g.intra = {m: pick(cands, int(r["intra"][h, i]), ("target", target)) for i, m in enumerate(mods)}
        for kk in range(1, n):
            g.step2[kk] = [Scored(name, {m: int(r["step2_cost"][h, kk - 1, x, i]) for i, m in enumerate(mods)},
                                  {m: float(r["step2_err"][h, kk - 1, x, i]) for i, m in enumerate(mods)})
                           for x, (name, _) in enumerate(xc)]
            for i, a in enumerate(mods):
                j = (i + kk) % n
                g.cross[(a, mods[j])] = pick(xc, int(r["cross"][h, i, j]), ("none", C.none()))
        g.budget3 = int(r["budget3"][h])
        g.step3_global = [Scored(name, {"all": int(r["step3g_cost"][h, c])}, {"all": float(r["step3g_err"][h, c])})
                          for c, (name, _) in enumerate(cands)]
        g.global_op = pick(cands, int(r["global_"][h]), ("target", target))
        g.step3 = [Scored(kd, {"all": int(r["step3_cost"][h, i])}, {"all": float(r["step3_err"][h, i])})
                   for i, kd in enumerate(_KINDS)]
        g.kind = _KINDS[int(r["kind"][h])]
        g.abi_cfg = cfgs[h]
        intra = {m: g.intra[m][1] for m in mods}
        if g.kind == "global":
            heads.append(C.global_head(g.global_op[1]))
        elif g.kind == "qboundary":
            heads.append(C.qboundary_head(intra))
        else:
            heads.append(C.boundary2d_head(intra, {ab: v2[1] for ab, v2 in g.cross.items()}))
        reps.append(g)
    return heads, reps, int(r["plans"])
