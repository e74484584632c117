"""GPU-vs-oracle comparison of one head, on host arrays only (test
infrastructure; numpy and the oracle, no torch and no GPU, so it also runs
in worker processes).

Layered protocol (discrete choices first, so that the bit-exact comparison of
the block index is not hostage to fp32-vs-fp64 noise):
  1. scores   GPU v, u, Grid folds and estimation LSE against the oracle's
              fp64 values: relative error <= SCORE_RTOL on entries at least
              1e-6 of the largest;
  2. choices  the oracle's decision rules re-run on the GPU's own score
              arrays (Grid folds -> stride and phase; v, u -> top-k) give the
              GPU's choices bit for bit;
  3. blocks   the oracle builds permutations and the CSR block index from the
              choices of step 4; they equal the GPU's bit for bit;
  4. choices  the oracle's own choices (from its fp64 scores) equal the GPU's;
              a difference is accepted only inside a tie (every decision that
              separates the two has an oracle margin below TIE_RTOL), is
              counted, and the oracle then adopts the GPU's choice;
  5. outputs  O and LSE on every evaluated row: |dO| <= O_TOL + half a bf16
              ulp of the oracle value (the output rounding), |dLSE| <=
              LSE_TOL * max(1, |LSE|).
No head skips a step: a tied head is compared in full under the adopted
choice.
"""
from __future__ import annotations

import numpy as np

from oracle import attention as OA
from oracle import grid as OG
from oracle import layout as OL
from oracle import numerics as ON
from oracle import plan as OP
from oracle import vslash as OV
from synth import config as C

O_TOL = 2e-2
LSE_TOL = 1e-3
SCORE_RTOL = 1e-3
TIE_RTOL = 1e-4
FLT_MIN = float(np.finfo(np.float32).tiny)
FOLD_PITCH = 1024           # the library's fold export: [stride - lo][1024]
ESTIMATED = (C.OP_GRID, C.OP_VSLASH, C.OP_VERT)


def slot_of(key):
    """Export slot of an op key (include/mmi.h, mmi_plan_export)."""
    if key == "g":
        return 0
    if key[0] in ("q", "i"):
        return key[1]
    return 8 + key[1] * 8 + key[2]


def op_keys(cfg: C.HeadCfg, S: int, modality):
    """[(key, op)] of every op of the head that takes an estimated choice."""
    if cfg.kind == C.HEAD_GLOBAL:
        out = [("g", cfg.op)]
    else:
        mods = sorted(OL.positions_of(OL.modality_array(S, modality)))
        if cfg.kind == C.HEAD_QBOUNDARY:
            out = [(("q", m), cfg.intra_op(m)) for m in mods]
        else:
            out = [(("i", m), cfg.intra_op(m)) for m in mods]
            out += [(("x", a, b), cfg.cross_op(a, b)) for a in mods for b in mods if a != b]
    return [(k, op) for k, op in out if op.kind in ESTIMATED]


def bf16_half_ulp(x):
    """Half the spacing of bfloat16 values at |x| (8 significand bits)."""
    ax = np.maximum(np.abs(np.asarray(x, dtype=np.float64)), FLT_MIN)
    return np.ldexp(1.0, np.floor(np.log2(ax)).astype(np.int64) - 8)


def rel_err(gpu, ref):
    ref = np.asarray(ref, dtype=np.float64)
    gpu = np.asarray(gpu, dtype=np.float64)
    if ref.size == 0:
        return 0.0
    big = np.abs(ref) >= 1e-6 * max(np.abs(ref).max(), 1e-300)
    if not big.any():
        return 0.0
    return float((np.abs(gpu - ref)[big] / np.abs(ref)[big]).max())


# ------------------------------------------------------------------ ties
def grid_outcomes(f64: dict, eps=OG.EPS_G, tol=TIE_RTOL):
    """Every (stride, phase) the Grid search can end on when each of its
    decisions whose margin in the fp64 folds {stride: c} is within tol
    (relative) may go either way: the phase argmax of a stride, and each
    'score > best * (1 + eps)' comparison of the ascending scan.
    (0, 0) stands for no stride."""
    states = {(0.0, (0, 0))}
    for s in sorted(f64):
        c = np.asarray(f64[s], dtype=np.float64)
        mx = float(c.max())
        phases = [int(p) for p in np.nonzero(mx - c <= tol * abs(mx))[0]]
        nxt = set()
        for b, ch in states:
            thr = b * (1.0 + eps)
            d = mx - thr
            near = thr > 0 and abs(d) <= tol * max(abs(thr), abs(mx))
            if d > 0 or near:
                nxt.update((mx, (s, p)) for p in phases)
            if d <= 0 or near:
                nxt.add((b, ch))
        states = nxt
        if len(states) > 64:
            raise AssertionError("Grid search: too many near-tied decisions to enumerate")
    return {ch for _, ch in states}


def selection_tie(score64, gsel, osel, what):
    """A different top-k selection is a tie iff it has the same size and every
    element selected by one side only lies within TIE_RTOL (relative) of the
    oracle's selection threshold, its smallest selected fp64 score (or below
    the smallest normal fp32 value, where both sides decide on zero)."""
    x = np.asarray(score64, dtype=np.float64)
    gsel, osel = np.asarray(gsel), np.asarray(osel)
    assert len(gsel) == len(osel), f"{what}: {len(gsel)} selected, oracle {len(osel)}"
    thr = float(x[osel].min()) if len(osel) else 0.0
    band = max(TIE_RTOL * abs(thr), 2 * FLT_MIN)
    diff = np.concatenate([np.setdiff1d(gsel, osel), np.setdiff1d(osel, gsel)])
    bad = [(int(i), float(x[i])) for i in diff if abs(x[i] - thr) > band]
    assert not bad, f"{what}: selection differs beyond the tie band around {thr}: {bad[:5]}"
    return len(diff) // 2


# ------------------------------------------------------------------ rows
def hline_rows(S, modality, cfg: C.HeadCfg, gpu):
    """Positions on the horizontal line of every Grid op of the head (rows
    whose coordinate is the chosen phase modulo the stride), from the GPU's
    exported stride and phase."""
    mod = OL.modality_array(S, modality)
    out = []
    for key, op in op_keys(cfg, S, modality):
        if op.kind != C.OP_GRID or key[0] == "x":
            continue
        sigma, p = (int(x) for x in gpu["slots"][key]["params"][:2])
        if sigma == 0:
            continue
        if key == "g":
            pos = np.arange(S)
            coord = pos
        else:
            pos = np.nonzero(mod == key[1])[0]
            coord = np.arange(len(pos)) if key[0] == "i" else pos
        out.append(pos[coord % sigma == p])
    return np.concatenate(out) if out else np.zeros(0, np.int64)


def sample_rows(S, modality, cfg, gpu, n_target=4096, seed=0, per_block=16, max_hline_blocks=None):
    """Stratified, seeded sample of query positions for one head: the last 64
    rows; the first row of every permuted query block that holds a Grid
    horizontal-line row (or of max_hline_blocks of them, evenly spaced);
    16 rows on each side of every modality boundary; the rest drawn
    uniformly as whole permuted query blocks (per_block rows of each, so the
    oracle gathers each block's keys once). All rows if S <= n_target."""
    if S <= n_target:
        return np.arange(S, dtype=np.int64)
    rng = np.random.default_rng(seed)
    qperm = np.asarray(gpu["qperm"], dtype=np.int64)
    slot = np.full(S, -1, np.int64)
    live = qperm >= 0
    slot[qperm[live]] = np.nonzero(live)[0]
    rows = set(range(S - 64, S))
    hl = hline_rows(S, modality, cfg, gpu)
    hb = np.unique(slot[hl] // 64)
    if max_hline_blocks is not None and len(hb) > max_hline_blocks:
        hb = hb[np.linspace(0, len(hb) - 1, max_hline_blocks).round().astype(np.int64)]
    for b in hb:
        blk = qperm[b * 64:(b + 1) * 64]
        rows.add(int(blk[blk >= 0][0]))
    if modality is not None:
        cut = np.nonzero(np.diff(np.asarray(modality).astype(np.int16)))[0] + 1
        for c in cut:
            rows.update(range(max(0, c - 16), min(S, c + 16)))
    nb = len(qperm) // 64
    for b in rng.permutation(nb):
        if len(rows) >= n_target:
            break
        blk = qperm[b * 64:(b + 1) * 64]
        blk = blk[blk >= 0]
        take = rng.choice(blk, size=min(per_block, len(blk), n_target - len(rows)), replace=False)
        rows.update(int(x) for x in take)
    return np.array(sorted(rows), dtype=np.int64)


# ------------------------------------------------------------------ one head
def check_head(h, cfg: C.HeadCfg, S, modality, q_rows, K, V, gpu, rows, O_rows, LSE_rows):
    """Steps 1-5 for one head. q_rows(positions) -> fp64 query rows of the
    head; K, V fp64 [S, 128] of its KV head; gpu: the head's exports (qperm,
    kperm, row_ptr, col_idx and, per estimated op key, v / u / fold /
    est_lse / params / vsel / ssel); O_rows, LSE_rows: the GPU's output at
    `rows` (fp64 decoded). Raises AssertionError on any mismatch; returns a
    report dict."""
    rep = dict(head=h, ties=[], score_err=0.0, max_o=0.0, max_o_excess=0.0, max_lse=0.0, rows=len(rows),
               nnz=0, adopted=0)
    ops, est, folds = OP.choose(cfg, S, modality, q_rows, K)
    for key, op in op_keys(cfg, S, modality):
        g = gpu["slots"][key]
        st = ops[key]
        e = est.get(key)
        assert e is not None, f"head {h} {key}: oracle ran no estimation"
        # step 1: scores
        assert len(g["v"]) == e.L_c, f"head {h} {key}: L_c {len(g['v'])} vs {e.L_c}"
        assert int(g["params"][2]) == e.L_c, f"head {h} {key}: params {g['params']} vs L_c {e.L_c}"
        # (a cross pair whose key modality has no token before the final query
        # rows selects nothing: the library then runs no estimation for it)
        assert e.L_c == 0 or int(g["params"][3]) == len(e.rows), \
            f"head {h} {key}: params {g['params']} vs {len(e.rows)} estimation rows"
        if e.L_c > 0:
            errs = [rel_err(g["v"], e.v)]
            if op.kind == C.OP_VSLASH:
                errs.append(rel_err(g["u"], e.u))
            gl = np.asarray(g["est_lse"], dtype=np.float64)
            lse_err = float(np.abs(gl - e.lse).max() / max(1.0, np.abs(e.lse).max()))
            assert lse_err <= LSE_TOL, f"head {h} {key}: estimation LSE error {lse_err}"
        else:
            errs = []
        cands = OG.candidates(op.stride_lo, op.stride_hi, e.L_c) if op.kind == C.OP_GRID else []
        lo = max(1, op.stride_lo)
        gfold = {s: np.asarray(g["fold"][(s - lo) * FOLD_PITCH:(s - lo) * FOLD_PITCH + s]) for s in cands}
        f64 = {s: OG.fold64(e.v, e.L_c, s) for s in cands}
        errs += [rel_err(gfold[s], f64[s]) for s in cands]
        if errs:
            err = max(errs)
            rep["score_err"] = max(rep["score_err"], err)
            assert err <= SCORE_RTOL, f"head {h} {key}: score relative error {err}"
        if op.kind == C.OP_GRID:
            got = (int(g["params"][0]), int(g["params"][1]))
            # step 2: the decision rule on the GPU's folds
            best, _ = OG.pick(gfold)
            assert (best or (0, 0)) == got, f"head {h} {key}: GPU folds give {best}, GPU chose {got}"
            # step 4: against the oracle's own choice
            want = (st.sigma, st.p) if st.kind == C.OP_GRID else (0, 0)
            if got != want:
                outs = grid_outcomes(f64)
                assert got in outs, f"head {h} {key}: Grid choice GPU {got}, oracle {want} (tie outcomes {outs})"
                rep["ties"].append((key, "grid", want, got))
                ops[key] = OP.adopt(st, sigma=got[0], p=got[1])
        else:
            gv = np.asarray(g["vsel"], dtype=np.int64)
            assert np.array_equal(OV.topk(g["v"], op.n_vertical, e.L_c), gv), \
                f"head {h} {key}: top-k of the GPU's v differs from its selection"
            new_v, new_s = st.vsel, st.ssel
            if not np.array_equal(gv, st.vsel):
                n = selection_tie(e.v, gv, st.vsel, f"head {h} {key} vertical")
                rep["ties"].append((key, "vsel", n))
                new_v = gv
            if op.kind == C.OP_VSLASH:
                gs = np.asarray(g["ssel"], dtype=np.int64)
                assert np.array_equal(OV.topk(g["u"], op.n_slash, e.L_c), gs), \
                    f"head {h} {key}: top-k of the GPU's u differs from its selection"
                if not np.array_equal(gs, st.ssel):
                    n = selection_tie(e.u, gs, st.ssel, f"head {h} {key} slash")
                    rep["ties"].append((key, "ssel", n))
                    new_s = gs
            if new_v is not st.vsel or new_s is not st.ssel:
                ops[key] = OP.adopt(st, vsel=new_v, ssel=new_s)
    rep["adopted"] = len(rep["ties"])
    # step 3: permutations and block index from the (adopted) choices
    hp = OP.assemble(cfg.kind, S, modality, ops)
    assert np.array_equal(gpu["qperm"], hp.qperm), f"head {h}: qperm differs"
    assert np.array_equal(gpu["kperm"], hp.kperm), f"head {h}: kperm differs"
    want_rp = np.concatenate([[0], np.cumsum([len(b) for b in hp.blocks])])
    assert np.array_equal(gpu["row_ptr"], want_rp), f"head {h}: row_ptr differs"
    assert np.array_equal(gpu["col_idx"], np.concatenate(hp.blocks)), f"head {h}: col_idx differs"
    rep["nnz"] = int(want_rp[-1])
    # step 5: outputs
    if len(rows):
        Oo, Lo = OA.head_rows(hp, q_rows, K, V, rows)
        d = np.abs(np.asarray(O_rows, dtype=np.float64) - Oo)
        excess = d - bf16_half_ulp(Oo)
        el = float((np.abs(np.asarray(LSE_rows, dtype=np.float64) - Lo) / np.maximum(1.0, np.abs(Lo))).max())
        rep["max_o"] = float(d.max())
        rep["max_o_excess"] = float(excess.max())
        rep["max_lse"] = el
        assert rep["max_o_excess"] <= O_TOL, \
            f"head {h}: |O - O_oracle| exceeds {O_TOL} + half a bf16 ulp by {rep['max_o_excess'] - O_TOL}"
        assert el <= LSE_TOL, f"head {h}: LSE relative error {el}"
    return rep


# ------------------------------------------------------------------ worker side
_KV = {}


def _kv_fp64(path_k, path_v, g):
    """K, V of KV head g decoded to fp64 from the shared [Hkv, S, 128] bf16
    bit files (the last one decoded is kept)."""
    key = (path_k, g)
    if key not in _KV:
        _KV.clear()
        kb = np.load(path_k, mmap_mode="r")
        vb = np.load(path_v, mmap_mode="r")
        _KV[key] = (ON.bf16_bits_to_f64(np.asarray(kb[g])), ON.bf16_bits_to_f64(np.asarray(vb[g])))
    return _KV[key]


def rows_lookup(pos, bits):
    """q_rows callable over a gathered set of query rows (bf16 bits)."""
    pos = np.asarray(pos, dtype=np.int64)
    vals = ON.bf16_bits_to_f64(bits)

    def q_rows(r):
        r = np.asarray(r, dtype=np.int64)
        i = np.searchsorted(pos, r)
        assert (i < len(pos)).all() and (pos[np.minimum(i, len(pos) - 1)] == r).all(), "query row not gathered"
        return vals[i]
    return q_rows


def run_task(task):
    """One head in a worker process: task = dict(h, g, cfg, S, modality, gpu,
    q_pos, q_bits, rows, o_bits, lse, path_k, path_v)."""
    K, V = _kv_fp64(task["path_k"], task["path_v"], task["g"])
    q_rows = rows_lookup(task["q_pos"], task["q_bits"])
    O = ON.bf16_bits_to_f64(task["o_bits"])
    return check_head(task["h"], task["cfg"], task["S"], task["modality"], q_rows, K, V, task["gpu"],
                      task["rows"], O, task["lse"])
