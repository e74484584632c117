"""HIP path vs oracle through the C-ABI (needs an MI355X)."""
import numpy as np
import pytest
import torch

from synth import config as C
from synth import generate, workloads

from parity import full_check, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ctx():
    from paper_2504_16083_amd import mmi
    c = mmi.Ctx(0)
    yield c
    c.close()


def _rand_qkv(S, Hq, Hkv, seed, scale_k=1.0):
    g = torch.Generator().manual_seed(seed)
    q = torch.randn(S, Hq, 128, generator=g)
    k = torch.randn(S, Hkv, 128, generator=g) * scale_k
    v = torch.randn(S, Hkv, 128, generator=g)
    return [t.to(torch.bfloat16).cuda() for t in (q, k, v)]


@pytest.mark.parametrize("S", [64, 200, 1000, 4096 + 37])
def test_dense_small(ctx, S):
    say(f"[gpu] dense S={S}")
    q, k, v = _rand_qkv(S, 2, 1, seed=S)
    heads = [C.global_head(C.dense())] * 2
    rep = full_check(ctx, S, 2, 1, None, heads, q, k, v)
    say(f"  max|dO|={rep.max_o:.3g} lse={rep.max_lse:.3g}")


def test_config0_grid(ctx):
    say("[gpu] config0 grid 4096")
    wl = workloads.config0()
    q, k, v = generate.make_qkv(wl, "cpu")
    q, k, v = q.cuda(), k.cuda(), v.cuda()
    rep = full_check(ctx, wl.S, wl.Hq, wl.Hkv, wl.modality, wl.heads, q, k, v)
    assert not rep.ties
    assert all(n == 206 for n in rep.nnz.values()), rep.nnz
    say(f"  nnz={rep.nnz} max|dO|={rep.max_o:.3g}")


@pytest.mark.parametrize("kind", ["ashape", "vslash", "grid_window", "grid_lines"])
def test_global_ops_small(ctx, kind):
    say(f"[gpu] global op {kind}")
    S = 2500
    q, k, v = _rand_qkv(S, 2, 1, seed=7, scale_k=2.0)
    op = {"ashape": C.ashape(64, 300), "vslash": C.vslash(40, 30),
          "grid_window": C.grid(50, 70), "grid_lines": C.grid(30, 31, True, True, False)}[kind]
    rep = full_check(ctx, S, 2, 1, None, [C.global_head(op)] * 2, q, k, v)
    say(f"  nnz={rep.nnz} ties={rep.ties} max|dO|={rep.max_o:.3g}")


def _mm_layout(S, seed):
    rng = np.random.default_rng(seed)
    mod = np.zeros(S, np.uint8)
    pos, m = 0, 0
    while pos < S:
        n = int(rng.integers(50, 700))
        mod[pos:pos + n] = m
        pos += n
        m ^= 1
    return mod


def test_boundary_heads_small(ctx):
    say("[gpu] boundary heads")
    S = 3000
    mod = _mm_layout(S, 3)
    q, k, v = _rand_qkv(S, 4, 2, seed=11, scale_k=2.0)
    heads = [
        C.qboundary_head({0: C.ashape(32, 200), 1: C.vslash(30, 20)}),
        C.boundary2d_head({0: C.ashape(32, 200), 1: C.grid(20, 40)}, {(0, 1): C.vert(40), (1, 0): C.dense()}),
        C.boundary2d_head({0: C.vslash(20, 20), 1: C.dense()}, {(0, 1): C.dense(), (1, 0): C.none()}),
        C.qboundary_head({0: C.dense(), 1: C.ashape(0, 128)}),
    ]
    rep = full_check(ctx, S, 4, 2, mod, heads, q, k, v)
    say(f"  nnz={rep.nnz} ties={rep.ties} max|dO|={rep.max_o:.3g}")


def test_static_baselines(ctx):
    """Section 4.1 baselines as block sets on the same kernel: Sparse
    Transformer fixed / strided and Tri-shape as global heads (frame-sized
    parameters) and as Q-Boundary / 2D-Boundary modality ops."""
    say("[gpu] static baselines")
    S = 3000
    mod = _mm_layout(S, 5)
    q, k, v = _rand_qkv(S, 6, 2, seed=13, scale_k=2.0)
    heads = [
        C.global_head(C.sf_fixed(196, 196)),
        C.global_head(C.sf_strided(196, 196)),
        C.global_head(C.trishape(128, 512, 128)),
        C.qboundary_head({0: C.trishape(32, 200, 100), 1: C.sf_strided(64, 150)}),
        C.boundary2d_head({0: C.sf_fixed(100, 37), 1: C.grid(20, 40)}, {(0, 1): C.vert(40), (1, 0): C.dense()}),
        C.boundary2d_head({0: C.trishape(0, 64, 300), 1: C.sf_strided(30, 90)}, {(0, 1): C.dense(), (1, 0): C.none()}),
    ]
    rep = full_check(ctx, S, 6, 2, mod, heads, q, k, v)
    say(f"  nnz={rep.nnz} ties={rep.ties} max|dO|={rep.max_o:.3g}")


def test_qboundary_grid(ctx):
    """Grid as a Q-Boundary modality op: stride and phase from the modality's
    final queries on global positions, phase-ordered queries, keys through
    one Grid layout per Grid modality (with and without the position-order
    layout), on a text/video layout with 196-token frames."""
    from synth.generate import Structure, Workload
    say("[gpu] Q-Boundary Grid")
    S, F = 16384, 196
    rng = np.random.default_rng(17)
    segs, n, m = [], 0, 0
    while n < S:
        ln = int(rng.integers(300, 900)) if m == 0 else F * int(rng.integers(8, 30))
        ln = min(ln, S - n)
        segs.append(np.full(ln, m, np.uint8))
        n += ln
        m ^= 1
    mod = np.concatenate(segs)
    st = Structure(sigma=[F, F], amp=2.0, text_amp=1.0)
    st.line_slot = [int(rng.integers(0, F)) for _ in range(2)]
    heads = [
        C.qboundary_head({0: C.ashape(128, 1024), 1: C.grid_frame(F)}),
        C.qboundary_head({0: C.vslash(100, 64), 1: C.grid_window(F)}),
        C.qboundary_head({0: C.grid(8, 64), 1: C.grid_frame(F)}),
        C.qboundary_head({0: C.dense(), 1: C.grid(F - 4, F + 4, True, False, False)}),
    ]
    wl = Workload("qb_grid_16k", S, 4, 2, mod, heads, st, 20250416 + 17, frame=F)
    q, k, v = generate.make_qkv(wl, "cuda")
    rows = np.unique(np.concatenate([np.arange(S - 64, S), np.random.default_rng(2).choice(S, 512, replace=False)]))
    rep = full_check(ctx, S, 4, 2, mod, heads, q, k, v, rows=rows)
    say(f"  nnz={rep.nnz} ties={rep.ties} max|dO|={rep.max_o:.3g} lse={rep.max_lse:.3g}")
    assert len(rep.ties) <= 1


def test_natten(ctx):
    """Neighborhood attention (bidirectional) through the tile permutation:
    3D and 2D grids of 2880 tokens, tiles cut by the grid border (padding
    masked), a near-full window and a 1x1x1 window."""
    say("[gpu] neighborhood attention")
    S = 2880
    q, k, v = _rand_qkv(S, 5, 1, seed=19)
    heads = [
        C.global_head(C.natten((6, 20, 24), (3, 7, 9), (2, 4, 8))),
        C.global_head(C.natten((1, 48, 60), (1, 11, 11), (1, 8, 8))),
        C.global_head(C.natten((6, 20, 24), (5, 19, 23), (1, 8, 8))),
        C.global_head(C.natten((5, 24, 24), (3, 5, 7), (4, 4, 4))),
        C.global_head(C.natten((3, 30, 32), (1, 1, 1), (1, 4, 16))),
    ]
    rep = full_check(ctx, S, 5, 1, None, heads, q, k, v)
    say(f"  nnz={rep.nnz} max|dO|={rep.max_o:.3g} lse={rep.max_lse:.3g}")


@pytest.mark.parametrize("S", [1, 2, 63, 64, 65, 127])
def test_tiny_sequences(ctx, S):
    """Sequences of one token to two blocks, every global op kind (a Grid
    search with too few tokens falls back to dense; 1-token windows)."""
    say(f"[gpu] tiny S={S}")
    q, k, v = _rand_qkv(S, 8, 2, seed=100 + S)
    heads = [C.global_head(C.dense()), C.global_head(C.ashape(1, 4)), C.global_head(C.vslash(3, 2)),
             C.global_head(C.grid(1, 8)), C.global_head(C.trishape(1, 3, 2)), C.global_head(C.sf_fixed(5, 3)),
             C.global_head(C.sf_strided(2, 7)),
             C.global_head(C.natten((1, 1, S), (1, 1, 1 if S < 3 else 3), (1, 1, 64)))]
    rep = full_check(ctx, S, 8, 2, None, heads, q, k, v)
    say(f"  nnz={rep.nnz} max|dO|={rep.max_o:.3g}")


def test_eight_modalities(ctx):
    """Eight modalities in short interleaved segments (1-89 tokens, most
    groups below one block): Q-Boundary heads with a different op per
    modality (two Grid modalities: three key layouts) and 2D-Boundary heads
    with none / dense / VERT cross pairs."""
    say("[gpu] eight modalities")
    S = 700
    rng = np.random.default_rng(8)
    mod = np.zeros(S, np.uint8)
    pos, m = 0, 0
    while pos < S:
        n = int(rng.integers(1, 90))
        mod[pos:pos + n] = m
        pos += n
        m = (m + 1) % 8
    q, k, v = _rand_qkv(S, 4, 2, seed=21)
    ops = [C.dense(), C.ashape(4, 40), C.vslash(6, 5), C.grid(3, 12), C.trishape(2, 30, 10), C.sf_fixed(20, 9),
           C.sf_strided(16, 5), C.grid(8, 8, True, False, True)]
    cross = {(a, b): [C.none(), C.dense(), C.vert(7)][(a + b) % 3] for a in range(8) for b in range(8) if a != b}
    heads = [C.qboundary_head({m: ops[m] for m in range(8)}),
             C.boundary2d_head({m: ops[(m + 3) % 8] for m in range(8)}, cross),
             C.qboundary_head({m: ops[(m + 5) % 8] for m in range(8)}),
             C.boundary2d_head({m: ops[(m + 1) % 8] for m in range(8)},
                               {ab: C.vert(3) for ab in cross})]
    rep = full_check(ctx, S, 4, 2, mod, heads, q, k, v)
    say(f"  nnz={rep.nnz} ties={rep.ties} max|dO|={rep.max_o:.3g}")


def test_determinism(ctx):
    say("[gpu] determinism")
    from paper_2504_16083_amd import mmi
    wl = workloads.config0()
    q, k, v = (t.cuda() for t in generate.make_qkv(wl, "cpu"))
    outs = []
    for _ in range(2):
        prob = mmi.Problem(wl.S, wl.Hq, wl.Hkv, wl.modality)
        o = torch.empty_like(q)
        lse = torch.empty(wl.Hq, wl.S, device="cuda")
        plan = mmi.Plan(ctx, prob, wl.heads, q, k)
        plan.execute(q, k, v, o, lse)
        torch.cuda.synchronize()
        outs.append((o.clone(), lse.clone(), plan.export(0, "col_idx"), plan.export(0, "v")))
        plan.destroy()
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])
    assert np.array_equal(outs[0][2], outs[1][2]) and np.array_equal(outs[0][3], outs[1][3])


def test_side_stream_and_one_shot(ctx):
    """A plan created and executed on a side stream, the one-shot entry point
    and the default-stream plan give bitwise the same output; a plan executes
    twice with the same result; strided (non-packed) Q/K/V views give the
    same output as packed copies."""
    from paper_2504_16083_amd import mmi
    say("[gpu] side stream / one-shot / strides")
    wl = workloads.config2()
    S = 16384
    mod = wl.modality[:S].copy()
    heads = wl.heads[:8]
    q, k, v = _rand_qkv(S, 8, 2, seed=31, scale_k=2.0)
    prob = mmi.Problem(S, 8, 2, mod)
    ref = torch.empty_like(q)
    plan = mmi.Plan(ctx, prob, heads, q, k)
    plan.execute(q, k, v, ref)
    again = torch.empty_like(q)
    plan.execute(q, k, v, again)
    torch.cuda.synchronize()
    plan.destroy()
    assert torch.equal(ref, again)
    side = torch.cuda.Stream()
    o2 = torch.empty_like(q)
    with torch.cuda.stream(side):
        p2 = mmi.Plan(ctx, prob, heads, q, k, side)
        p2.execute(q, k, v, o2, None, side)
    side.synchronize()
    p2.destroy()
    assert torch.equal(ref, o2)
    o3 = torch.empty_like(q)
    mmi.mmi_attention(ctx, prob, heads, q, k, v, o3)
    torch.cuda.synchronize()
    assert torch.equal(ref, o3)
    # Q/K/V as views into wider buffers (token stride larger than H*128)
    big_q = torch.zeros(S, 10, 128, dtype=q.dtype, device="cuda")
    big_k = torch.zeros(S, 3, 128, dtype=k.dtype, device="cuda")
    big_v = torch.zeros(S, 3, 128, dtype=v.dtype, device="cuda")
    big_q[:, 1:9] = q
    big_k[:, :2] = k
    big_v[:, 1:3] = v
    qs, ks, vs = big_q[:, 1:9], big_k[:, :2], big_v[:, 1:3]
    probs = mmi.Problem(S, 8, 2, mod, strides={n: (t.stride(0), t.stride(1)) for n, t in
                                                (("q", qs), ("k", ks), ("v", vs))})
    o4 = torch.empty_like(q)
    p4 = mmi.Plan(ctx, probs, heads, qs, ks)
    p4.execute(qs, ks, vs, o4)
    torch.cuda.synchronize()
    p4.destroy()
    assert torch.equal(ref, o4)


def test_permute_roundtrip(ctx):
    say("[gpu] permute/unpermute")
    from paper_2504_16083_amd import mmi
    S = 5000
    x = torch.randn(S, 4, 128, device="cuda").to(torch.bfloat16)
    perm = torch.randperm(S, device="cuda").to(torch.int32)
    perm = torch.cat([perm, torch.full((40,), -1, device="cuda", dtype=torch.int32)])
    y = torch.empty(S + 40, 4, 128, device="cuda", dtype=torch.bfloat16)
    mmi.mmi_permute_rows(x, y, perm)
    z = torch.zeros_like(x)
    mmi.mmi_unpermute_rows(y, z, perm)
    torch.cuda.synchronize()
    assert torch.equal(y[:S], x[perm[:S].long()])
    assert torch.count_nonzero(y[S:]) == 0
    assert torch.equal(z, x)


@pytest.mark.parametrize("R", [1, 2, 4])
def test_row_group_variants(R, monkeypatch):
    """Every work-item shape (R query blocks per workgroup) against the oracle,
    with a small split chunk so long rows are merged by the combine kernel."""
    say(f"[gpu] row group R={R}")
    from paper_2504_16083_amd import mmi
    monkeypatch.setenv("MMI_ROW_GROUP", str(R))
    monkeypatch.setenv("MMI_CHUNK_BLOCKS", "5")
    c = mmi.Ctx(0)
    try:
        S = 3000
        mod = _mm_layout(S, 5)
        q, k, v = _rand_qkv(S, 4, 2, seed=13, scale_k=2.0)
        heads = [C.global_head(C.dense()), C.global_head(C.grid(20, 40)),
                 C.qboundary_head({0: C.ashape(32, 200), 1: C.vslash(30, 20)}),
                 C.boundary2d_head({0: C.ashape(32, 200), 1: C.grid(20, 40)},
                                   {(0, 1): C.vert(40), (1, 0): C.dense()})]
        rep = full_check(c, S, 4, 2, mod, heads, q, k, v)
        say(f"  nnz={rep.nnz} ties={rep.ties} max|dO|={rep.max_o:.3g}")
    finally:
        c.close()


@pytest.mark.parametrize("seed", range(24))
def test_random_configs(ctx, seed):
    """Seeded random layouts (1-4 modalities, segments of any length) and
    random heads of every kind and op (global ops incl. Grid and
    neighborhood attention, Q-Boundary incl. Grid modalities, 2D-Boundary
    with every cross kind) at random lengths up to 5000 tokens."""
    from random_cfg import random_head, random_layout
    rng = np.random.default_rng(1000 + seed)
    S = int(rng.integers(1, 5000))
    nmod = int(rng.integers(1, 5))
    mod = random_layout(rng, S, nmod) if nmod > 1 else None
    mods = sorted(set(mod.tolist())) if mod is not None else [0]
    heads = [random_head(rng, S, mods) for _ in range(4)]
    say(f"[gpu] random seed {seed}: S={S} modalities {mods} kinds {[h.kind for h in heads]}")
    q, k, v = _rand_qkv(S, 4, 2, seed=2000 + seed, scale_k=1.5)
    rows = None if S <= 2000 else np.unique(np.concatenate(
        [np.arange(S - 64, S), np.random.default_rng(seed).choice(S, 512, replace=False)]))
    rep = full_check(ctx, S, 4, 2, mod, heads, q, k, v, rows=rows)
    say(f"  nnz={rep.nnz} ties={rep.ties} max|dO|={rep.max_o:.3g}")


@pytest.mark.parametrize("Hq,Hkv", [(1, 1), (16, 2), (6, 6)])
def test_head_counts(ctx, Hq, Hkv):
    """One head, a GQA ratio of 8, and one KV head per query head."""
    say(f"[gpu] Hq={Hq} Hkv={Hkv}")
    S = 3000
    mod = _mm_layout(S, 9)
    q, k, v = _rand_qkv(S, Hq, Hkv, seed=40 + Hq, scale_k=1.5)
    kinds = [C.global_head(C.ashape(64, 300)), C.qboundary_head({0: C.ashape(32, 200), 1: C.vslash(30, 20)}),
             C.global_head(C.grid(20, 40)),
             C.boundary2d_head({0: C.ashape(32, 200), 1: C.grid(20, 40)}, {(0, 1): C.vert(40), (1, 0): C.dense()})]
    heads = [kinds[h % 4] for h in range(Hq)]
    rep = full_check(ctx, S, Hq, Hkv, mod, heads, q, k, v)
    say(f"  nnz={rep.nnz} ties={rep.ties} max|dO|={rep.max_o:.3g}")


@pytest.mark.parametrize("chunk", [None, "5"])
def test_output_without_lse(chunk, monkeypatch):
    """Without an LSE buffer the kernel skips the fp32 row sums; O (also of
    split rows, merged by the bf16-P sums) is bitwise the O of the run that
    writes the LSE, which the oracle tests check."""
    from paper_2504_16083_amd import mmi
    say(f"[gpu] O without LSE, chunk {chunk}")
    if chunk:
        monkeypatch.setenv("MMI_CHUNK_BLOCKS", chunk)
    c = mmi.Ctx(0)
    try:
        S = 3000
        mod = _mm_layout(S, 6)
        q, k, v = _rand_qkv(S, 4, 2, seed=23, scale_k=2.0)
        heads = [C.global_head(C.dense()), C.global_head(C.grid(20, 40)),
                 C.qboundary_head({0: C.ashape(32, 200), 1: C.vslash(30, 20)}),
                 C.boundary2d_head({0: C.ashape(32, 200), 1: C.grid(20, 40)},
                                   {(0, 1): C.vert(40), (1, 0): C.dense()})]
        prob = mmi.Problem(S, 4, 2, mod)
        plan = mmi.Plan(c, prob, heads, q, k)
        o1, o2 = torch.empty_like(q), torch.empty_like(q)
        lse = torch.empty(4, S, device="cuda")
        plan.execute(q, k, v, o1, lse)
        plan.execute(q, k, v, o2, None)
        torch.cuda.synchronize()
        split = sum(plan.stats(h).split_rows for h in range(4))
        plan.destroy()
        say(f"  split rows {split}")
        assert (split > 0) == bool(chunk)
        assert torch.equal(o1, o2)
        rep = full_check(c, S, 4, 2, mod, heads, q, k, v)
        say("  " + rep.line())
    finally:
        c.close()
