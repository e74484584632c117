"""Pins of the oracle's modality-aware pattern search (Algorithm 4), on a
4096-token text/video sample with planted structure and a search space
scaled to that length (the paper's space and 1k + 4k target assume about
25K tokens)."""
import numpy as np
import pytest

from oracle import attention as A
from oracle import numerics as ON
from oracle import plan as P
from oracle import search as OS
from synth import config as C
from synth import generate
from synth.generate import Structure, Workload

S, F = 4096, 64


def small_space():
    cands = []
    for mode in ("frame", "window"):
        for h, v, s in [(1, 0, 0), (0, 1, 0), (0, 0, 1), (1, 1, 0), (0, 1, 1), (1, 1, 1)]:
            op = C.grid_frame(F, h, v, s) if mode == "frame" else C.grid_window(F, 4, h, v, s)
            cands.append((f"grid_{mode}_{h}{v}{s}", op))
    cands += [(f"ashape_{a}_{b}", C.ashape(a, b)) for a, b in [(16, 128), (16, 256), (16, 512)]]
    cands += [(f"vslash_{a}_{b}", C.vslash(a, b)) for a, b in [(64, 64), (64, 128), (128, 128), (256, 32)]]
    xc = [("none", C.none())] + [(f"vert_{n}", C.vert(n)) for n in (32, 64, 128)] + [("dense", C.dense())]
    return cands, xc, C.ashape(64, 256)


def sample(seed=123):
    mod = np.array([0] * 256 + [1] * (F * 24) + [0] * 256 + [1] * (S - 512 - F * 24), dtype=np.uint8)
    st = Structure(sigma=[F], amp=2.0, text_amp=1.0)
    st.line_slot = [5]
    wl = Workload("search_sample", S, 2, 1, mod, [C.global_head(C.dense())] * 2, st, seed, frame=F)
    q, k, v = generate.make_qkv(wl, "cpu")
    return mod, [ON.torch_bf16_to_f64(t) for t in (q, k, v)]


@pytest.fixture(scope="module")
def searched():
    mod, (Q, K, V) = sample()
    cands, xc, target = small_space()
    cfg, rep = OS.search_head(Q[:, 0], K[:, 0], V[:, 0], S, mod, cands, xc, target)
    return mod, (Q, K, V), cfg, rep


def _ashape_count(L, sink, local):
    """Blocks of A-shape(sink, local) per query block over L tokens in
    position order: {key blocks below the sink} U {blocks of the window}."""
    tot = 0
    for i in range((L + 63) // 64):
        a, b = 64 * i, min(L, 64 * i + 64) - 1
        s = set(range(0, min(sink - 1, b) // 64 + 1)) if sink else set()
        s |= set(range(max(0, a - local + 1) // 64, b // 64 + 1))
        tot += len(s)
    return tot


def test_budget_is_the_target_pattern_in_modality_coordinates(searched):
    mod, _, _, rep = searched
    for m in (0, 1):
        assert rep.budget1[m] == _ashape_count(int((mod == m).sum()), 64, 256)
    assert rep.budget3 == _ashape_count(S, 64, 256)


def test_choices_are_admissible_minima(searched):
    mod, _, cfg, rep = searched
    for m, (name, op) in rep.intra.items():
        c = next(c for c in rep.step1 if c.name == name)
        assert c.cost[m] <= rep.budget1[m]
        assert all(d.err[m] >= c.err[m] for d in rep.step1 if d.cost[m] <= rep.budget1[m])
    fin = next(c for c in rep.step3 if c.name == rep.kind)
    assert fin.cost["all"] <= rep.budget3
    assert all(d.err["all"] >= fin.err["all"] for d in rep.step3 if d.cost["all"] <= rep.budget3)


def test_errors_match_direct_attention(searched):
    """The recorded error of the chosen head equals the squared difference of
    the direct masked-softmax rows and plain causal attention."""
    mod, (Q, K, V), cfg, rep = searched
    hp = P.plan_head(cfg, S, mod, lambda r: Q[r, 0], K[:, 0])
    rows = np.arange(S)
    O, _ = A.head_rows(hp, Q[:, 0], K[:, 0], V[:, 0], rows)
    R, _ = A.dense_causal_rows(Q[:, 0], K[:, 0], V[:, 0], rows)
    want = float(((O - R) ** 2).sum())
    got = next(c for c in rep.step3 if c.name == rep.kind).err["all"]
    assert abs(got - want) <= 1e-9 * max(1.0, want)


def test_planted_structure_is_found(searched):
    """Video tokens attend to same-slot tokens of every frame (planted period
    64): the video modality gets a Grid op with slash lines; text (local
    structure) gets a local pattern; the head is modality-aware."""
    _, _, cfg, rep = searched
    vid = rep.intra[1][1]
    assert vid.kind == C.OP_GRID and vid.use_s
    assert rep.intra[0][1].kind in (C.OP_ASHAPE, C.OP_VSLASH)
    assert rep.kind in ("qboundary", "2d")


def test_one_modality_reduces_to_the_global_search():
    _, (Q, K, V) = sample(7)
    cands, xc, target = small_space()
    n = 2048
    cfg, rep = OS.search_head(Q[:n, 1], K[:n, 0], V[:n, 0], n, None, cands, xc, target)
    assert rep.global_op[0] == rep.intra[0][0]
    g = {c.name: c for c in rep.step3_global}
    for c in rep.step1:
        assert c.cost[0] == g[c.name].cost["all"]
        assert abs(c.err[0] - g[c.name].err["all"]) <= 1e-9 * max(1.0, c.err[0])


def test_adopted_choices_are_carried_into_later_steps(searched):
    """Adopting the search's own picks changes nothing; adopting another
    intra choice records the own pick, scores step 1 the same, and builds
    the step-2 candidates on the adopted intra ops (so their costs and
    errors are those of a search whose step 1 chose it)."""
    mod, (Q, K, V), cfg, rep = searched
    cands, xc, target = small_space()
    own = {("intra", m): rep.intra[m][0] for m in (0, 1)}
    own.update({("cross",) + ab: rep.cross[ab][0] for ab in rep.cross})
    own.update({"global": rep.global_op[0], "kind": rep.kind})
    cfg2, rep2 = OS.search_head(Q[:, 0], K[:, 0], V[:, 0], S, mod, cands, xc, target, adopt=own)
    assert rep2.own == {} and rep2.kind == rep.kind and rep2.intra == rep.intra and rep2.cross == rep.cross
    other = next(n for n, _ in cands if n != rep.intra[1][0] and n.startswith("ashape"))
    cfg3, rep3 = OS.search_head(Q[:, 0], K[:, 0], V[:, 0], S, mod, cands, xc, target,
                                adopt={("intra", 1): other})
    assert rep3.own == {("intra", 1): rep.intra[1][0]} and rep3.intra[1][0] == other
    assert [(c.name, c.cost, c.err) for c in rep3.step1] == [(c.name, c.cost, c.err) for c in rep.step1]
    # step 2 ran with the adopted video op: its candidates' costs equal a
    # direct plan of that configuration
    intra = {0: rep.intra[0][1], 1: dict(cands)[other]}
    cross = {(0, 1): C.dense(), (1, 0): C.dense()}
    name, op = xc[1]
    cross[(0, 1)] = op
    hp = P.plan_head(C.boundary2d_head(intra, cross), S, mod, lambda r: Q[r, 0], K[:, 0])
    off, arr = hp.groups[1]
    lo, hi = off // 64, off // 64 + (len(arr) + 63) // 64
    want = sum(int(((bs >= lo) & (bs < hi)).sum()) for i, bs in enumerate(hp.blocks)
               if P._group_of_block(hp, i)[0] == 0)
    got = next(c for c in rep3.step2[1] if c.name == name).cost[0]
    assert got == want
