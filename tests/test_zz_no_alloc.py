"""mmi_attention_noalloc (the plan in the library's static device scratch)
against mmi_attention through the C-ABI: bitwise the same O and LSE on two
calls in a row, the second with a smaller problem (the scratch then still
holds the first call's contents), and a clear error, with O untouched, for a
problem whose plan does not fit the scratch."""
import numpy as np
import pytest
import torch

from synth import config as C
from synth import workloads

pytestmark = pytest.mark.gpu


def _qkv(S, Hq, Hkv, seed):
    g = torch.Generator().manual_seed(seed)
    return [(torch.randn(S, H, 128, generator=g) * s).to(torch.bfloat16).cuda()
            for H, s in ((Hq, 1.0), (Hkv, 1.5), (Hkv, 1.0))]


def _both(ctx, S, Hq, Hkv, mod, heads, seed):
    from paper_2504_16083_amd import mmi
    q, k, v = _qkv(S, Hq, Hkv, seed)
    prob = mmi.Problem(S, Hq, Hkv, mod)
    out = []
    for fn in (mmi.mmi_attention, mmi.mmi_attention_noalloc):
        o = torch.full_like(q, 3.0)
        lse = torch.full((Hq, S), float("nan"), device="cuda")
        fn(ctx, prob, heads, q, k, v, o, lse)
        torch.cuda.synchronize()
        out.append((o, lse))
    return out


def test_noalloc_matches_mmi_attention():
    from paper_2504_16083_amd import mmi
    print("[gpu] no-allocation entry point", flush=True)
    ctx = mmi.Ctx(0)
    try:
        wl = workloads.config2()
        S = 16384
        mod = wl.modality[:S].copy()
        (o1, l1), (o2, l2) = _both(ctx, S, 8, 2, mod, wl.heads[:8], seed=3)
        assert torch.equal(o1, o2) and torch.equal(l1, l2)
        assert not torch.isnan(l2).any()
        # smaller problem second: other head kinds, ragged length
        S2 = 3001
        mod2 = np.zeros(S2, np.uint8)
        mod2[1000:2200] = 1
        heads2 = [C.global_head(C.grid(20, 40)), C.global_head(C.vslash(30, 20)),
                  C.boundary2d_head({0: C.ashape(32, 200), 1: C.grid(20, 40)}, {(0, 1): C.vert(40), (1, 0): C.dense()}),
                  C.qboundary_head({0: C.ashape(32, 200), 1: C.vslash(30, 20)})]
        (o3, l3), (o4, l4) = _both(ctx, S2, 4, 2, mod2, heads2, seed=4)
        assert torch.equal(o3, o4) and torch.equal(l3, l4)
        assert not torch.isnan(l4).any()
    finally:
        ctx.close()


def test_noalloc_rejects_a_plan_beyond_the_scratch():
    """1M tokens, 8 dense heads: the per-head block bitmaps alone (32 MiB
    each) exceed the 256 MiB scratch; the call fails before the attention
    kernel and leaves O as it was."""
    from paper_2504_16083_amd import mmi
    print("[gpu] no-allocation entry point, too large", flush=True)
    ctx = mmi.Ctx(0)
    try:
        S, Hq = 1 << 20, 8
        q = torch.zeros(S, Hq, 128, dtype=torch.bfloat16, device="cuda")
        k = torch.zeros(S, 1, 128, dtype=torch.bfloat16, device="cuda")
        v = torch.zeros_like(k)
        o = torch.full_like(q, 3.0)
        with pytest.raises(mmi.MMIError) as ei:
            mmi.mmi_attention_noalloc(ctx, mmi.Problem(S, Hq, 1), [C.global_head(C.dense())] * Hq, q, k, v, o)
        torch.cuda.synchronize()
        assert ei.value.status == -2 and "no-allocation scratch" in str(ei.value)
        assert bool((o == 3.0).all())
        # the library still works afterwards, with and without the scratch
        (o1, l1), (o2, l2) = _both(ctx, 4096, 2, 1, None, [C.global_head(C.ashape(64, 512))] * 2, seed=5)
        assert torch.equal(o1, o2) and torch.equal(l1, l2)
    finally:
        ctx.close()
