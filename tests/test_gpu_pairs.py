"""mmi_plan_pair_counts against the definition computed on the host from
the plan's exported block index and permutations: per selected block, the
live query rows times the live key rows at or below each of them (every
live pair for a bidirectional head); computed = selected blocks x 4096.
Causal heads of every kind (4K Grid workload, random mixes with boundary
heads) and bidirectional NATTEN heads."""
import numpy as np
import pytest
import torch

from synth import config as C
from synth import generate, workloads

from parity import say
from random_cfg import random_head, random_layout

pytestmark = pytest.mark.gpu


def host_counts(plan, h, S, causal=True):
    rp, col = plan.export(h, "row_ptr"), plan.export(h, "col_idx")
    qp = plan.export(h, "qperm").reshape(-1, 64)
    kp = plan.export(h, "kperm").reshape(-1, 64)
    useful = 0
    for i in range(len(rp) - 1):
        q = qp[i][qp[i] >= 0]
        if q.size == 0 or rp[i + 1] == rp[i]:
            continue
        for j in col[rp[i]:rp[i + 1]]:
            k = np.sort(kp[j][kp[j] >= 0])
            useful += int(np.searchsorted(k, q, side="right").sum()) if causal else q.size * k.size
    return useful, int(rp[-1]) * 4096


def _bidirectional(head):
    return head.kind == C.HEAD_GLOBAL and head.op.kind == C.OP_NATTEN


def _check(ctx, S, Hq, Hkv, modality, heads, q, k):
    from paper_2504_16083_amd import mmi
    plan = mmi.Plan(ctx, mmi.Problem(S, Hq, Hkv, modality), heads, q, k)
    try:
        for h in range(Hq):
            got = plan.pair_counts(h)
            want = host_counts(plan, h, S, not _bidirectional(heads[h]))
            say(f"  head {h}: useful {got[0]} of {got[1]} ({got[0] / max(1, got[1]):.3f})")
            assert got == want, (h, got, want)
    finally:
        plan.destroy()


@pytest.fixture(scope="module")
def ctx():
    from paper_2504_16083_amd import mmi
    c = mmi.Ctx(0)
    yield c
    c.close()


def test_pair_counts_grid_4k(ctx):
    wl = workloads.config0()
    q, k, _ = generate.make_qkv(wl, "cuda")
    say(f"[gpu] pair counts {wl.name}")
    _check(ctx, wl.S, wl.Hq, wl.Hkv, wl.modality, wl.heads, q, k)


@pytest.mark.parametrize("seed", [1, 2, 3, 4])
def test_pair_counts_random_mix(ctx, seed):
    """Random layouts and heads of every kind (the recipe of the random
    parity tests)."""
    rng = np.random.default_rng(3000 + seed)
    S = int(rng.integers(200, 4000))
    nmod = int(rng.integers(1, 4))
    mod = random_layout(rng, S, nmod) if nmod > 1 else None
    mods = sorted(set(mod.tolist())) if mod is not None else [0]
    heads = [random_head(rng, S, mods) for _ in range(4)]
    g = torch.Generator().manual_seed(seed)
    q = torch.randn(S, 4, 128, generator=g).to(torch.bfloat16).cuda()
    k = (1.5 * torch.randn(S, 2, 128, generator=g)).to(torch.bfloat16).cuda()
    say(f"[gpu] pair counts random case {seed}: S={S} modalities {mods} kinds {[h.kind for h in heads]}")
    _check(ctx, S, 4, 2, mod, heads, q, k)


def test_pair_counts_natten(ctx):
    S = 2880
    g = torch.Generator().manual_seed(3)
    q = torch.randn(S, 2, 128, generator=g).to(torch.bfloat16).cuda()
    k = torch.randn(S, 1, 128, generator=g).to(torch.bfloat16).cuda()
    heads = [C.global_head(C.natten((6, 20, 24), (3, 7, 9), (2, 4, 8))),
             C.global_head(C.natten((3, 30, 32), (1, 1, 1), (1, 4, 16)))]
    say("[gpu] pair counts NATTEN")
    _check(ctx, S, 2, 1, None, heads, q, k)


@pytest.mark.parametrize("S", [1, 63, 65])
def test_pair_counts_tiny(ctx, S):
    """One token to just over one block, every global op kind (padding rows
    and keys in the last block)."""
    g = torch.Generator().manual_seed(S)
    q = torch.randn(S, 8, 128, generator=g).to(torch.bfloat16).cuda()
    k = torch.randn(S, 2, 128, generator=g).to(torch.bfloat16).cuda()
    heads = [C.global_head(C.dense()), C.global_head(C.ashape(1, 4)), C.global_head(C.vslash(3, 2)),
             C.global_head(C.grid(1, 8)), C.global_head(C.trishape(1, 3, 2)), C.global_head(C.sf_fixed(5, 3)),
             C.global_head(C.sf_strided(2, 7)),
             C.global_head(C.natten((1, 1, S), (1, 1, 1 if S < 3 else 3), (1, 1, 64)))]
    say(f"[gpu] pair counts S={S}")
    _check(ctx, S, 8, 2, None, heads, q, k)
