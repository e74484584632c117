"""Parity helpers: run the HIP path through the C-ABI and compare it with the
oracle on the same seeded inputs (test infrastructure).

Layered comparison (discrete choices first, so bit-exactness of the block
index is not hostage to fp32-vs-fp64 noise):
  1. scores   GPU v/u/fold vs oracle fp64, relative error on significant entries;
  2. choices  Grid (sigma, phase) and VS/VERT selections equal the oracle's
              (a mismatch is accepted only where the oracle's own decision
              margin is below the tie tolerance; such heads are reported and
              their blocks/outputs checked for validity only);
  3. blocks   permutations and CSR bit-exact against the oracle's closed forms;
  4. outputs  O max-abs <= 2e-2 (bf16), LSE |diff| <= 1e-3 * max(1, |LSE|).
"""
from __future__ import annotations

import sys
from dataclasses import dataclass, field

import numpy as np
import torch

from oracle import attention as OA
from oracle import numerics as ON
from oracle import plan as OP
from synth import config as C

O_TOL = 2e-2
LSE_TOL = 1e-3
SCORE_RTOL = 2e-3
TIE_RTOL = 1e-4


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def slot_of(key):
    if key == "g":
        return 0
    if key[0] in ("q", "i"):
        return key[1]
    return 8 + key[1] * 8 + key[2]


@dataclass
class Report:
    ties: list = field(default_factory=list)
    max_o: float = 0.0
    max_lse: float = 0.0
    rows: int = 0
    nnz: dict = field(default_factory=dict)


def run_gpu(ctx, S, Hq, Hkv, modality, heads, q, k, v):
    from paper_2504_16083_amd import mmi
    prob = mmi.Problem(S, Hq, Hkv, modality)
    o = torch.empty_like(q)
    lse = torch.full((Hq, S), float("nan"), device=q.device, dtype=torch.float32)
    plan = mmi.Plan(ctx, prob, heads, q, k)
    plan.execute(q, k, v, o, lse)
    torch.cuda.synchronize()
    return plan, o, lse


def _rel_err(gpu, ref):
    ref = np.asarray(ref, dtype=np.float64)
    gpu = np.asarray(gpu, dtype=np.float64)
    if ref.size == 0:
        return 0.0
    big = np.abs(ref) >= 1e-6 * max(np.abs(ref).max(), 1e-300)
    if not big.any():
        return 0.0
    return float((np.abs(gpu - ref)[big] / np.abs(ref)[big]).max())


def compare_head(plan, h, hp: OP.HeadPlan, rep: Report, exact_choices=True):
    """Steps 1-3 for one head. Returns True if the block index was compared exactly."""
    tied = False
    for key, est in hp.est.items():
        s = slot_of(key)
        gv = plan.export(h, "v", s)
        assert len(gv) == est.L_c, (h, key, len(gv), est.L_c)
        if est.L_c == 0:
            # a cross pair whose key modality has no token before the final
            # query rows: nothing to select, the library runs no estimation
            continue
        ev = _rel_err(gv, est.v)
        assert ev <= SCORE_RTOL, f"head {h} {key}: v rel err {ev}"
        if est.u is not None and hp.ops[key].op.kind == C.OP_VSLASH:
            gu = plan.export(h, "u", s)
            eu = _rel_err(gu, est.u)
            assert eu <= SCORE_RTOL, f"head {h} {key}: u rel err {eu}"
        gl = plan.export(h, "est_lse", s)
        assert np.abs(gl - est.lse).max() <= 1e-3 * max(1.0, np.abs(est.lse).max()), (h, key)
    for key, st in hp.ops.items():
        s = slot_of(key)
        if st.op.kind == C.OP_GRID:
            prm = plan.export(h, "params", s)
            got = (int(prm[0]), int(prm[1]))
            want = (st.sigma, st.p) if st.kind == C.OP_GRID else (0, 0)
            if got != want:
                folds = hp.folds[key]
                if want[0] and got[0] in folds and want[0] in folds:
                    a, b = folds[want[0]].max(), folds[got[0]].max()
                    gap = abs(float(a) - float(b)) / max(float(a), 1e-30)
                    if gap < TIE_RTOL:
                        tied = True
                        rep.ties.append((h, key, want, got))
                        continue
                raise AssertionError(f"head {h} {key}: grid choice gpu {got} oracle {want}")
        if st.kind in (C.OP_VSLASH, C.OP_VERT):
            gsel = plan.export(h, "vsel", s)
            if not np.array_equal(gsel, st.vsel):
                tied |= _tie_ok(hp.est[key].v, gsel, st.vsel, f"head {h} {key} vsel")
                rep.ties.append((h, key, "vsel"))
            if st.kind == C.OP_VSLASH:
                gss = plan.export(h, "ssel", s)
                if not np.array_equal(gss, st.ssel):
                    tied |= _tie_ok(hp.est[key].u, gss, st.ssel, f"head {h} {key} ssel")
                    rep.ties.append((h, key, "ssel"))
    gq = plan.export(h, "qperm")
    gk = plan.export(h, "kperm")
    if not tied:
        assert np.array_equal(gq, hp.qperm), f"head {h}: qperm differs"
        assert np.array_equal(gk, hp.kperm), f"head {h}: kperm differs"
        rp = plan.export(h, "row_ptr")
        col = plan.export(h, "col_idx")
        want_rp = np.concatenate([[0], np.cumsum([len(b) for b in hp.blocks])])
        assert np.array_equal(rp, want_rp), f"head {h}: row_ptr differs"
        assert np.array_equal(col, np.concatenate(hp.blocks)), f"head {h}: col_idx differs"
        rep.nnz[h] = len(col)
    return not tied


def _tie_ok(score, gsel, osel, what):
    """A different selection is valid only if every swapped element is within
    the tie tolerance of the selection threshold (oracle fp64 scores)."""
    x = np.asarray(score, dtype=np.float64)
    assert len(gsel) == len(osel), f"{what}: size {len(gsel)} vs {len(osel)}"
    only_g = np.setdiff1d(gsel, osel)
    only_o = np.setdiff1d(osel, gsel)
    thr = x[osel].min() if len(osel) else 0.0
    scale = max(x.max(), 1e-300)
    bad = [(i, x[i]) for i in np.concatenate([only_g, only_o]) if abs(x[i] - thr) > TIE_RTOL * scale]
    assert not bad, f"{what}: selection differs beyond ties: {bad[:5]}"
    return True


def compare_outputs(h, hp, Q, K, V, kvh, O, LSE, rows, rep: Report):
    Oo, Lo = OA.head_rows(hp, Q[:, h], K[:, kvh], V[:, kvh], rows)
    eo = float(np.abs(O[rows, h] - Oo).max())
    el = float((np.abs(LSE[h, rows] - Lo) / np.maximum(1.0, np.abs(Lo))).max())
    rep.max_o = max(rep.max_o, eo)
    rep.max_lse = max(rep.max_lse, el)
    rep.rows += len(rows)
    assert eo <= O_TOL, f"head {h}: max |O - O_oracle| = {eo}"
    assert el <= LSE_TOL, f"head {h}: LSE rel err {el}"


def full_check(ctx, S, Hq, Hkv, modality, heads, q, k, v, rows=None, heads_to_check=None):
    """GPU run + oracle plans + layered comparison. q/k/v: CUDA bf16 tensors."""
    plan, o, lse = run_gpu(ctx, S, Hq, Hkv, modality, heads, q, k, v)
    Q, K, V = (ON.torch_bf16_to_f64(t) for t in (q, k, v))
    O = ON.torch_bf16_to_f64(o)
    LSE = lse.cpu().double().numpy()
    G = Hq // Hkv
    rep = Report()
    try:
        for h in (heads_to_check if heads_to_check is not None else range(Hq)):
            hp = OP.plan_head(heads[h], S, modality, lambda r, h=h: Q[r, h], K[:, h // G])
            exact = compare_head(plan, h, hp, rep)
            if exact:
                rr = np.arange(S) if rows is None else rows
                compare_outputs(h, hp, Q, K, V, h // G, O, LSE, rr, rep)
    finally:
        plan.destroy()
    return rep


def sample_rows(S, modality, rng, n_uniform=64, last=64, around=8):
    """Stratified query rows: the last rows, rows on both sides of every
    modality boundary, and uniform rows (seeded)."""
    rows = set(range(max(0, S - last), S))
    if modality is not None:
        cut = np.nonzero(np.diff(np.asarray(modality).astype(np.int16)))[0] + 1
        for c in cut[:64]:
            rows.update(range(max(0, c - around), min(S, c + around)))
    rows.update(rng.choice(S, size=min(n_uniform, S), replace=False).tolist())
    return np.array(sorted(rows), dtype=np.int64)


def sampled_check(ctx, wl, q, k, v, heads_to_check, rows_extra=None, seed=0):
    """Full-size parity: every head's scores, choices, permutations and block
    index are compared in full; O/LSE on stratified sampled rows (including
    each Grid head's first horizontal-line rows)."""
    plan, o, lse = run_gpu(ctx, wl.S, wl.Hq, wl.Hkv, wl.modality, wl.heads, q, k, v)
    G = wl.Hq // wl.Hkv
    rng = np.random.default_rng(seed)
    base_rows = sample_rows(wl.S, wl.modality, rng)
    kv_cache = {}

    def kv(g):
        if g not in kv_cache:
            kv_cache.clear()
            kv_cache[g] = (ON.torch_bf16_to_f64(k[:, g]), ON.torch_bf16_to_f64(v[:, g]))
        return kv_cache[g]

    rep = Report()
    try:
        for h in heads_to_check:
            qh = q[:, h]

            def q_rows(r, qh=qh):
                return ON.torch_bf16_to_f64(qh[torch.as_tensor(np.asarray(r), device=qh.device)])

            K, V = kv(h // G)
            hp = OP.plan_head(wl.heads[h], wl.S, wl.modality, q_rows, K)
            if not compare_head(plan, h, hp, rep):
                continue
            rows = base_rows
            if hp.qperm is not None and hp.nbq:
                lastblk = hp.qperm[(hp.nbq - 1) * OP.B:hp.nbq * OP.B]
                rows = np.union1d(rows, lastblk[lastblk >= 0][:8])
            Oo, Lo = OA.head_rows(hp, q_rows, K, V, rows)
            Og = ON.torch_bf16_to_f64(o[torch.as_tensor(rows, device=o.device), h])
            Lg = lse[h, torch.as_tensor(rows, device=lse.device)].cpu().double().numpy()
            eo = float(np.abs(Og - Oo).max())
            el = float((np.abs(Lg - Lo) / np.maximum(1.0, np.abs(Lo))).max())
            rep.max_o = max(rep.max_o, eo)
            rep.max_lse = max(rep.max_lse, el)
            rep.rows += len(rows)
            assert eo <= O_TOL, f"head {h}: max |O - O_oracle| = {eo}"
            assert el <= LSE_TOL, f"head {h}: LSE rel err {el}"
    finally:
        plan.destroy()
    return rep
