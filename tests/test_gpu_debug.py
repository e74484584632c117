"""The debug checks on real plans: mmi_plan_check passes on the plans of
the 32K and 128K mixed workloads (every head kind, row groups of four),
Q-Boundary heads with Grid key layouts (one and two Grid layouts), and
bidirectional NATTEN heads; a context created with MMI_DEBUG=1 runs the
checks inside every plan creation and produces bitwise the same O as one
without."""
import numpy as np
import pytest
import torch

from synth import config as C
from synth import generate, workloads

from parity import say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ctx():
    from paper_2504_16083_amd import mmi
    c = mmi.Ctx(0)
    yield c
    c.close()


def _check_plan(ctx, S, Hq, Hkv, modality, heads, q, k):
    from paper_2504_16083_amd import mmi
    plan = mmi.Plan(ctx, mmi.Problem(S, Hq, Hkv, modality), heads, q, k)
    try:
        plan.check()
        t = plan.timing()
        say(f"  checked: {t['computed_blocks']} blocks, {t['loaded_blocks']} loaded, {t['work_items']} items")
    finally:
        plan.destroy()


@pytest.mark.parametrize("cid", [1, 2])
def test_plan_check_workloads(ctx, cid):
    wl = workloads.by_id(cid)
    say(f"[gpu] plan check {wl.name}")
    q, k, _ = generate.make_qkv(wl, "cuda")
    _check_plan(ctx, wl.S, wl.Hq, wl.Hkv, wl.modality, wl.heads, q, k)


def test_plan_check_layouts_and_natten(ctx):
    say("[gpu] plan check: Q-Boundary Grid layouts, NATTEN")
    S, F = 16384, 196
    rng = np.random.default_rng(23)
    segs, n, m = [], 0, 0
    while n < S:
        ln = min(int(rng.integers(300, 900)) if m == 0 else F * int(rng.integers(8, 30)), S - n)
        segs.append(np.full(ln, m, np.uint8))
        n += ln
        m ^= 1
    mod = np.concatenate(segs)
    g = torch.Generator().manual_seed(23)
    q = torch.randn(S, 4, 128, generator=g).to(torch.bfloat16).cuda()
    k = torch.randn(S, 2, 128, generator=g).to(torch.bfloat16).cuda()
    heads = [
        C.qboundary_head({0: C.ashape(128, 1024), 1: C.grid_frame(F)}),     # position order + one Grid layout
        C.qboundary_head({0: C.grid(8, 64), 1: C.grid_frame(F)}),           # two Grid layouts
        C.qboundary_head({0: C.vslash(100, 64), 1: C.grid_window(F)}),
        C.global_head(C.vslash(200, 32)),
    ]
    _check_plan(ctx, S, 4, 2, mod, heads, q, k)
    Sn = 2880
    qn = torch.randn(Sn, 3, 128, generator=g).to(torch.bfloat16).cuda()
    kn = torch.randn(Sn, 1, 128, generator=g).to(torch.bfloat16).cuda()
    nheads = [C.global_head(C.natten((6, 20, 24), (3, 7, 9), (2, 4, 8))),
              C.global_head(C.natten((1, 48, 60), (1, 11, 11), (1, 8, 8))),
              C.global_head(C.natten((3, 30, 32), (1, 1, 1), (1, 4, 16)))]
    _check_plan(ctx, Sn, 3, 1, None, nheads, qn, kn)


def test_debug_mode_same_output(monkeypatch):
    """MMI_DEBUG=1 at context creation: the plan of the 32K workload is
    checked inside mmi_attention, and O is bitwise that of a context
    without the debug mode."""
    from paper_2504_16083_amd import mmi
    wl = workloads.by_id(1)
    q, k, v = generate.make_qkv(wl, "cuda")
    prob = mmi.Problem(wl.S, wl.Hq, wl.Hkv, wl.modality)
    outs = []
    for dbg in ("1", None):
        if dbg:
            monkeypatch.setenv("MMI_DEBUG", dbg)
        else:
            monkeypatch.delenv("MMI_DEBUG", raising=False)
        c = mmi.Ctx(0)
        try:
            o = torch.empty(wl.S, wl.Hq, 128, dtype=torch.bfloat16, device="cuda")
            mmi.mmi_attention(c, prob, wl.heads, q, k, v, o)
            torch.cuda.synchronize()
            outs.append(o.view(torch.int16).cpu())
        finally:
            c.close()
    say(f"[gpu] debug mode: O bitwise equal {bool(torch.equal(outs[0], outs[1]))}")
    assert torch.equal(outs[0], outs[1])
