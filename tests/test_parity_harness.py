"""CPU tests of the GPU-vs-oracle comparison itself (parity_core, and the
worker fan-out of parity.py): exports built from the oracle's own plan pass;
planted differences in scores, choices, permutations, block indices and
outputs fail; a choice that differs only inside a tie passes, is counted,
and is then checked in full under the adopted choice; the stratified row
sample has the strata it promises."""
import numpy as np
import pytest

import parity_core as PC
from oracle import attention as OA
from oracle import numerics as ON
from oracle import plan as OP
from synth import config as C
from synth import generate, workloads


def mock_exports(hp, cfg, S, modality):
    """The library's export layout, filled from an oracle plan (fp32 scores,
    folds at [stride - lo][1024], params {sigma, phase, L_c, rows})."""
    gpu = dict(qperm=hp.qperm.astype(np.int32), kperm=hp.kperm.astype(np.int32),
               row_ptr=np.concatenate([[0], np.cumsum([len(b) for b in hp.blocks])]).astype(np.int32),
               col_idx=np.concatenate(hp.blocks).astype(np.int32), slots={})
    for key, op in PC.op_keys(cfg, S, modality):
        e, st = hp.est[key], hp.ops[key]
        sig = st.sigma if st.kind == C.OP_GRID else 0
        d = dict(params=np.array([sig, st.p if sig else 0, e.L_c, len(e.rows)], np.int32),
                 v=e.v.astype(np.float32), est_lse=e.lse.astype(np.float32))
        if op.kind == C.OP_GRID:
            lo = max(1, op.stride_lo)
            f = np.zeros((max(0, min(op.stride_hi, e.L_c // 2) - lo + 1), PC.FOLD_PITCH), np.float32)
            for s, c in hp.folds[key].items():
                f[s - lo, :s] = c
            d["fold"] = f.reshape(-1)
        else:
            d["vsel"] = st.vsel.astype(np.int32)
        if op.kind == C.OP_VSLASH:
            d["u"] = e.u.astype(np.float32)
            d["ssel"] = st.ssel.astype(np.int32)
        gpu["slots"][key] = d
    return gpu


def _case(seed=0):
    wl = workloads.config0()
    q, k, v = generate.make_qkv(wl, "cpu")
    Q, K, V = (ON.torch_bf16_to_f64(t) for t in (q, k, v))
    return wl, Q, K[:, 0], V[:, 0]


def _run(wl, Q, K, V, cfg, h=0, gpu=None, rows=None, perturb_o=0.0):
    S = wl.S
    hp = OP.plan_head(cfg, S, wl.modality, lambda r: Q[r, h], K)
    gpu = mock_exports(hp, cfg, S, wl.modality) if gpu is None else gpu
    rows = np.arange(S - 300, S) if rows is None else rows
    O, L = OA.head_rows(hp, Q[:, h], K, V, rows)
    Ob = ON.bf16_bits_to_f64(ON.f64_to_bf16_bits(O)) + perturb_o
    return PC.check_head(h, cfg, S, wl.modality, lambda r: Q[r, h], K, V, gpu, rows, Ob, L), hp, gpu


@pytest.fixture(scope="module")
def case():
    return _case()


def test_oracle_exports_pass(case):
    wl, Q, K, V = case
    rep, _, _ = _run(wl, Q, K, V, wl.heads[0])
    assert rep["ties"] == [] and rep["nnz"] == 206
    # the slot embedding on V makes outputs large: the half-ulp term is used
    assert rep["max_o"] > 0


@pytest.mark.parametrize("what", ["col_idx", "qperm", "phase", "fold", "v", "output"])
def test_planted_differences_fail(case, what):
    wl, Q, K, V = case
    cfg = wl.heads[0]
    _, hp, gpu = _run(wl, Q, K, V, cfg)
    g = gpu["slots"]["g"]
    if what == "col_idx":
        gpu["col_idx"] = gpu["col_idx"].copy()
        gpu["col_idx"][5] += 1
    elif what == "qperm":
        gpu["qperm"] = gpu["qperm"].copy()
        gpu["qperm"][[3, 4]] = gpu["qperm"][[4, 3]]
    elif what == "phase":           # a phase far from the maximum, the folds unchanged
        g["params"] = g["params"].copy()
        g["params"][1] = (g["params"][1] + 7) % g["params"][0]
    elif what == "fold":            # one fold entry off by 1%
        g["fold"] = g["fold"].copy()
        g["fold"][int(np.argmax(g["fold"]))] *= 1.01
    elif what == "v":
        g["v"] = g["v"].copy()
        g["v"][int(np.argmax(g["v"]))] *= 1.01
    with pytest.raises(AssertionError):
        _run(wl, Q, K, V, cfg, gpu=gpu, perturb_o=0.03 if what == "output" else 0.0)


def test_grid_tie_outcomes():
    """Decisions inside the tie band may go either way; others may not."""
    f = {10: np.array([1.0, 3.0, 3.0 * (1 - 5e-5)]), 11: np.array([2.0, 3.0 * 1.02 * (1 + 5e-5), 0.0])}
    outs = PC.grid_outcomes(f)
    assert outs == {(10, 1), (10, 2), (11, 1)}
    f2 = {10: np.array([1.0, 3.0, 2.0]), 11: np.array([2.0, 3.0 * 1.05, 0.0])}
    assert PC.grid_outcomes(f2) == {(11, 1)}


def test_selection_tie_band():
    x = np.array([5.0, 4.0, 3.0, 3.0 * (1 + 5e-5), 1.0])
    assert PC.selection_tie(x, [0, 1, 2], [0, 1, 3], "t") == 1
    with pytest.raises(AssertionError):
        PC.selection_tie(x, [0, 1, 4], [0, 1, 3], "t")
    with pytest.raises(AssertionError):
        PC.selection_tie(x, [0, 1], [0, 1, 3], "t")


def test_vslash_tie_is_adopted_and_checked_in_full(case, monkeypatch):
    """A VS head whose exported selection swaps two slash offsets of equal
    oracle score: counted as a tie, then the block index and outputs are
    compared under the GPU's selection (the oracle's own CSR then fails)."""
    from oracle import vslash as OV
    wl, Q, K, V = case
    S = wl.S
    cfg = C.global_head(C.vslash(30, 20))
    order = {}
    real_choose = OP.choose

    def choose_with_tie(*a_, **kw):
        # the oracle's estimate with the 20th and 21st slash scores made equal
        ops_, est_, folds_ = real_choose(*a_, **kw)
        u = est_["g"].u
        if not order:
            o = np.lexsort((np.arange(len(u)), -u.astype(np.float32)))
            order.update(a=int(o[19]), b=int(o[20]))
        u[order["b"]] = u[order["a"]]
        ops_["g"] = OP.adopt(ops_["g"], vsel=ops_["g"].vsel, ssel=OV.topk(u, 20, est_["g"].L_c))
        return ops_, est_, folds_

    monkeypatch.setattr(OP, "choose", choose_with_tie)
    hp = OP.plan_head(cfg, S, wl.modality, lambda r: Q[r, 0], K)
    st, e = hp.ops["g"], hp.est["g"]
    a, b = order["a"], order["b"]
    picked, other = (a, b) if a in st.ssel else (b, a)
    gsel = np.sort(np.concatenate([st.ssel[st.ssel != picked], [other]]))
    ops = dict(hp.ops)
    ops["g"] = OP.adopt(st, vsel=st.vsel, ssel=gsel)
    hp_g = OP.assemble(cfg.kind, S, wl.modality, ops)
    hp_g.est, hp_g.folds = hp.est, hp.folds
    gpu = mock_exports(hp_g, cfg, S, wl.modality)
    gu = gpu["slots"]["g"]["u"]
    gu[other] = gu[picked] * np.float32(1 + 1e-6)          # the GPU's own top-k takes `other`
    assert np.array_equal(OV.topk(gu, 20, e.L_c), gsel)
    rows = np.arange(S - 200, S)
    O, L = OA.head_rows(hp_g, Q[:, 0], K, V, rows)
    rep = PC.check_head(0, cfg, S, wl.modality, lambda r: Q[r, 0], K, V, gpu, rows, O, L)
    assert rep["ties"] and rep["ties"][0][1] == "ssel"
    own = mock_exports(hp, cfg, S, wl.modality)
    if not np.array_equal(own["col_idx"], gpu["col_idx"]):
        bad = dict(gpu, row_ptr=own["row_ptr"], col_idx=own["col_idx"])
        with pytest.raises(AssertionError):
            PC.check_head(0, cfg, S, wl.modality, lambda r: Q[r, 0], K, V, bad, rows, O, L)


def test_sample_rows_strata():
    """Last 64 rows, a first row per horizontal-line block, both sides of
    every boundary, and the total; rows are positions, sorted, unique."""
    S = 20000
    mod = np.ones(S, np.uint8)
    mod[5000:5600] = 0
    cfg = C.global_head(C.grid(100, 100))
    hp = OP.assemble(cfg.kind, S, mod, {"g": OP.grid_state(cfg.op, S, 100, 37)})
    gpu = dict(qperm=hp.qperm, slots={"g": dict(params=np.array([100, 37, S, 64]))})
    rows = PC.sample_rows(S, mod, cfg, gpu, n_target=4096, seed=3)
    assert len(rows) == 4096 and np.all(np.diff(rows) > 0)
    assert set(range(S - 64, S)) <= set(rows.tolist())
    assert set(range(4984, 5016)) | set(range(5584, 5616)) <= set(rows.tolist())
    hl = np.arange(37, S, 100)
    first = {int(hp.qperm[b * 64]) for b in range(len(hp.qperm) // 64)
             if np.isin(hp.qperm[b * 64:(b + 1) * 64], hl).any()}
    assert first <= set(rows.tolist())
    assert len(PC.sample_rows(3000, None, cfg, gpu)) == 3000


def test_worker_pool_matches_in_process(tmp_path):
    """The spawn worker fan-out gives the same reports as the in-process
    check (K/V through bf16 bit files, query rows through the task)."""
    import parity
    wl = workloads.config0()
    q, k, v = generate.make_qkv(wl, "cpu")
    S = wl.S
    Q, K, V = (ON.torch_bf16_to_f64(t) for t in (q, k, v))
    path_k, path_v = str(tmp_path / "k.npy"), str(tmp_path / "v.npy")
    np.save(path_k, parity._bits(k.transpose(0, 1)))
    np.save(path_v, parity._bits(v.transpose(0, 1)))
    tasks = []
    for h in range(2):
        cfg = wl.heads[h]
        hp = OP.plan_head(cfg, S, wl.modality, lambda r, h=h: Q[r, h], K[:, 0])
        gpu = mock_exports(hp, cfg, S, wl.modality)
        rows = PC.sample_rows(S, wl.modality, cfg, gpu, n_target=512, seed=h)
        O, L = OA.head_rows(hp, Q[:, h], K[:, 0], V[:, 0], rows)
        qpos = np.union1d(rows, np.arange(S - 64, S))
        tasks.append(dict(h=h, g=0, cfg=cfg, S=S, modality=wl.modality, gpu=gpu, q_pos=qpos,
                          q_bits=parity._bits(q[qpos, h]), rows=rows, o_bits=ON.f64_to_bf16_bits(O), lse=L,
                          path_k=path_k, path_v=path_v))
    rep = parity.run_tasks(tasks, workers=2)
    assert sorted(rep.heads) == [0, 1] and not rep.ties and rep.rows == 1024
    assert rep.nnz == {0: 206, 1: 206}
