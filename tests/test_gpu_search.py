"""GPU pattern search (Algorithm 4 through libmmi) against the oracle's, on
the 4096-token text/video sample with the scaled search space of the oracle
pins: every candidate's block cost bit-exact and errors within the bf16
output band at all three steps (the oracle carries the GPU's choices
forward), and the same choices (a different one only where the oracle's
errors of the two are inside that band)."""
import math

import numpy as np
import pytest
import torch

from oracle import search as OS
from synth import config as C

from parity import full_check, say
from test_oracle_search import S, F, sample, small_space

pytestmark = pytest.mark.gpu


def _band(rows):
    # |sqrt(e_gpu) - sqrt(e_oracle)| <= ||O_gpu - O_oracle|| + ||R_gpu - R_oracle||:
    # bf16 output rounding (<= 2^-8 relative, |O| < 1 here) on rows x 128 values
    return 2 * 2.0 ** -8 * math.sqrt(rows * 128)


def _close(eg, eo, rows):
    return abs(math.sqrt(max(eg, 0.0)) - math.sqrt(max(eo, 0.0))) <= _band(rows) + 1e-2 * math.sqrt(eo)


def _same_choice(got, want, scored, key, rows):
    if got == want:
        return True
    e = {s.name: s.err[key] for s in scored}
    return got in e and want in e and _close(e[got], e[want], rows)


def test_search_matches_oracle():
    """All three steps compared, whatever was chosen before: the oracle
    carries the GPU's choices into its later steps (adopt) and keeps its own
    picks beside them; every own pick that differs must be a tie inside the
    bf16 error band. Costs bit-exact, errors in the band, at every step."""
    from paper_2504_16083_amd import mmi
    from paper_2504_16083_amd import search as GS
    mod, (Q, K, V) = sample()
    cands, xc, target = small_space()
    # the oracle's bf16 inputs, on the device
    q, k, v = (torch.from_numpy(x).to(torch.bfloat16).cuda() for x in (Q, K, V))
    ctx = mmi.Ctx(0)
    try:
        heads, reps, nplans = GS.search(ctx, S, 2, 1, mod, q, k, v, cands, xc, target)
    finally:
        ctx.close()
    say(f"[gpu] search: {nplans} plans; kinds {[r.kind for r in reps]}")
    assert nplans == 8 + 2 * len(cands) + len(xc)
    for h in range(2):    # the configuration the C call chose is the one the records name
        assert bytes(mmi._head_cfg(heads[h])) == bytes(reps[h].abi_cfg), h
    rows = {m: int((mod == m).sum()) for m in (0, 1)}
    ties = 0
    for h in range(2):
        g = reps[h]
        adopt = {("intra", m): g.intra[m][0] for m in (0, 1)}
        adopt.update({("cross",) + ab: g.cross[ab][0] for ab in g.cross})
        adopt.update({"global": g.global_op[0], "kind": g.kind})
        cfg, orep = OS.search_head(Q[:, h], K[:, 0], V[:, 0], S, mod, cands, xc, target, adopt=adopt)
        say(f"  head {h}: gpu {g.kind} {[g.intra[m][0] for m in (0, 1)]} {[v2[0] for v2 in g.cross.values()]} "
            f"{g.global_op[0]}; oracle's own differing picks {orep.own}")
        assert g.budget1 == orep.budget1 and g.budget3 == orep.budget3
        for a, b in zip(g.step1, orep.step1):
            assert a.name == b.name and a.cost == b.cost, (a, b)
            for m in (0, 1):
                assert _close(a.err[m], b.err[m], rows[m]), (h, a.name, m, a.err[m], b.err[m])
        for kk in g.step2:
            assert [a.name for a in g.step2[kk]] == [b.name for b in orep.step2[kk]]
            for a, b in zip(g.step2[kk], orep.step2[kk]):
                assert a.cost == b.cost, (a, b)
                for m in (0, 1):
                    assert _close(a.err[m], b.err[m], rows[m])
        for a, b in zip(g.step3_global, orep.step3_global):
            assert a.name == b.name and a.cost == b.cost
            assert _close(a.err["all"], b.err["all"], S)
        for a, b in zip(g.step3, orep.step3):
            assert a.name == b.name and a.cost == b.cost
            assert _close(a.err["all"], b.err["all"], S)
        # a pick of the oracle's own that differs from the GPU's is a tie
        for key, own in orep.own.items():
            ties += 1
            if key[0] == "intra":
                assert _same_choice(g.intra[key[1]][0], own, orep.step1, key[1], rows[key[1]]), key
            elif key[0] == "cross":
                a, b = key[1:]
                kk = (b - a) % 2                 # the step-2 round that decides pair (a, b)
                assert _same_choice(g.cross[(a, b)][0], own, orep.step2[kk], a, rows[a]), key
            elif key == "global":
                assert _same_choice(g.global_op[0], own, orep.step3_global, "all", S), key
            else:
                assert _same_choice(g.kind, own, orep.step3, "all", S), key
    say(f"  ties {ties}")


def test_search_calibration_costs():
    """The search on its calibration sample (24,576 tokens, 28 heads, the
    paper's search space) in the configuration bench.py times: every head
    gets a valid configuration; head 0's step-1 block costs of all 24
    candidates and the budgets equal the oracle's closed-form block counts."""
    from oracle import numerics as ON
    from oracle import plan as OP
    from paper_2504_16083_amd import mmi
    from paper_2504_16083_amd import search as GS
    from synth import generate, workloads
    from synth import search_space as SP
    wl = workloads.search_calibration()
    q, k, v = generate.make_qkv(wl, "cuda")
    cands, xc, target = SP.intra_candidates(wl.frame), SP.cross_candidates(), SP.budget_op()
    ctx = mmi.Ctx(0)
    try:
        heads, reps, nplans = GS.search(ctx, wl.S, wl.Hq, wl.Hkv, wl.modality, q, k, v, cands, xc, target)
    finally:
        ctx.close()
    say(f"[gpu] calibration search: {nplans} plans, kinds {[r.kind for r in reps]}")
    assert len(heads) == wl.Hq and all(r.kind in ("global", "qboundary", "2d") for r in reps)
    Q, K = ON.torch_bf16_to_f64(q[:, 0]), ON.torch_bf16_to_f64(k[:, 0])
    none_all = {(0, 1): C.none(), (1, 0): C.none()}

    def costs(op):
        hp = OP.plan_head(C.boundary2d_head({0: op, 1: op}, none_all), wl.S, wl.modality, lambda r: Q[r], K)
        out = {0: 0, 1: 0}
        for i, bs in enumerate(hp.blocks):
            out[OP._group_of_block(hp, i)[0]] += len(bs)
        return out

    assert reps[0].budget1 == costs(target)
    mism = []
    for (name, op), sc in zip(cands, reps[0].step1):
        assert sc.name == name
        got, want = sc.cost, costs(op)
        if got != want:
            mism.append((name, op, got, want))
            say(f"  {name}: cost {got} vs oracle {want}")
    # a different cost is accepted only as the consequence of a tied choice:
    # the candidate's plan for head 0 passes the layered comparison (which
    # accepts a different Grid stride/phase or VS selection only inside the
    # tie band, then checks the block index under the GPU's choice) with at
    # least one tie
    none_all = {(0, 1): C.none(), (1, 0): C.none()}
    for name, op, got, want in mism:
        cfg = C.boundary2d_head({0: op, 1: op}, none_all)
        rows = np.arange(wl.S - 256, wl.S)
        ctx = mmi.Ctx(0)
        try:
            rep = full_check(ctx, wl.S, wl.Hq, wl.Hkv, wl.modality, [cfg] * wl.Hq, q, k, v, rows=rows,
                             heads_to_check=[0])
        finally:
            ctx.close()
        say(f"  {name}: " + rep.line())
        assert rep.ties, (name, got, want)
        assert sum(rep.nnz.values()) == sum(got.values())


def test_search_reports_a_bad_candidate():
    """A candidate the library rejects stops the search with the plan's own
    status and message (here an op kind out of range), and the context stays
    usable: the same search with valid candidates runs after it."""
    from paper_2504_16083_amd import mmi
    from paper_2504_16083_amd import search as GS
    mod, (Q, K, V) = sample()
    cands, xc, target = small_space()
    q, k, v = (torch.from_numpy(x).to(torch.bfloat16).cuda() for x in (Q, K, V))
    bad = C.Op(kind=99)
    ctx = mmi.Ctx(0)
    try:
        with pytest.raises(mmi.MMIError) as e:
            GS.search(ctx, S, 2, 1, mod, q, k, v, [("bad", bad)] + list(cands), xc, target)
        assert e.value.status == -3 and len(str(e.value)) > 0, str(e.value)
        heads, reps, nplans = GS.search(ctx, S, 2, 1, mod, q, k, v, cands, xc, target)
        assert nplans == 8 + 2 * len(cands) + len(xc) and len(heads) == 2
    finally:
        ctx.close()
    say(f"[gpu] bad candidate reported: {e.value}")
