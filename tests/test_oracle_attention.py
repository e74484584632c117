"""Pins of the oracle's attention and of the whole oracle pipeline.

* every causal block selected == textbook causal attention (torch fp64
  scaled_dot_product_attention, a library routine);
* attention evaluated in permuted slot space with the online-softmax block
  recurrence of Algorithms 5-7 == the direct masked softmax in original space;
* the planted grid of the 4096-token workload is recovered end to end.
"""
import numpy as np
import pytest
import torch

from oracle import attention as A
from oracle import numerics
from oracle import plan as P
from synth import config as C
from synth import generate, workloads


def _qkv(S, seed=0, D=128):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((S, D)), rng.standard_normal((S, D)) * 1.5,
            rng.standard_normal((S, D)))


def test_dense_plan_equals_torch_sdpa():
    S = 333
    Q, K, V = _qkv(S)
    hp = P.assemble(C.HEAD_GLOBAL, S, None, {"g": P.OpState(C.OP_DENSE, C.dense(), L=S)})
    rows = np.arange(S)
    O, L = A.head_rows(hp, Q, K, V, rows)
    t = lambda x: torch.from_numpy(x)[None, None]
    ref = torch.nn.functional.scaled_dot_product_attention(t(Q), t(K), t(V), is_causal=True)[0, 0].numpy()
    assert np.abs(O - ref).max() < 1e-12
    logits = (Q @ K.T) / np.sqrt(128)
    logits[np.triu_indices(S, 1)] = -np.inf
    from scipy.special import logsumexp
    assert np.abs(L - logsumexp(logits, axis=1)).max() < 1e-12


def _random_plans(S, seed):
    rng = np.random.default_rng(seed)
    mod = np.zeros(S, np.uint8)
    cut = sorted(rng.choice(np.arange(1, S), 3, replace=False))
    mod[cut[0]:cut[1]] = 1
    mod[cut[2]:] = 1
    T = {m: np.nonzero(mod == m)[0] for m in (0, 1)}
    vs = np.sort(rng.choice(S, 20, replace=False))
    ss = np.sort(rng.choice(S, 20, replace=False))
    yield P.assemble(C.HEAD_GLOBAL, S, None, {"g": P.grid_state(C.grid(11, 11), S, 11, 4)})
    yield P.assemble(C.HEAD_GLOBAL, S, None, {"g": P.grid_state(C.grid(70, 70, True, False, False), S, 70, 69)})
    yield P.assemble(C.HEAD_GLOBAL, S, None, {"g": P.OpState(C.OP_VSLASH, C.vslash(20, 20), vsel=vs, ssel=ss, L=S)})
    yield P.assemble(C.HEAD_QBOUNDARY, S, mod, {
        ("q", 0): P.OpState(C.OP_ASHAPE, C.ashape(16, 64), L=S),
        ("q", 1): P.OpState(C.OP_VSLASH, C.vslash(20, 20), vsel=vs, ssel=ss, L=S)})
    L1 = len(T[1])
    yield P.assemble(C.HEAD_2D, S, mod, {
        ("i", 0): P.OpState(C.OP_ASHAPE, C.ashape(16, 64), L=len(T[0])),
        ("i", 1): P.grid_state(C.grid(9, 9), L1, 9, 3),
        ("x", 0, 1): P.OpState(C.OP_VERT, C.vert(10), vsel=np.sort(rng.choice(L1, 10, replace=False)), L=L1),
        ("x", 1, 0): P.OpState(C.OP_DENSE, C.dense(), L=len(T[0]))})


@pytest.mark.parametrize("seed", [0, 1])
def test_permuted_blockwise_equals_masked_softmax(seed):
    S = 700
    Q, K, V = _qkv(S, seed)
    for hp in _random_plans(S, seed):
        O1, L1 = A.permuted_blockwise(hp, Q, K, V)
        rows = np.arange(S)
        O2, L2 = A.head_rows(hp, Q, K, V, rows)
        assert np.abs(O1 - O2).max() < 1e-12
        assert np.abs(L1 - L2).max() < 1e-12
        # the element mask always keeps the diagonal, never a future key
        for q in (0, 5, S - 1, S // 2):
            ks = P.element_mask_row(hp, q)
            assert q in ks and ks.max() <= q


def test_planted_grid_recovered_end_to_end():
    wl = workloads.config0()
    Q, K, V = generate.make_qkv(wl, "cpu")
    Q, K = numerics.torch_bf16_to_f64(Q), numerics.torch_bf16_to_f64(K)
    planted_phase = (64 + wl.structure.line_slot[0]) % 252      # 64 text tokens first
    for h in range(wl.Hq):
        hp = P.plan_head(wl.heads[h], wl.S, wl.modality, lambda r: Q[r, h], K[:, 0])
        st = hp.ops["g"]
        assert (st.sigma, st.p) == (252, planted_phase)


def test_planted_jittered_strides_recovered():
    """The 32K workload plants one stride per KV group (255 + U{-4..4}) and
    searches strides within 8 of 255: one Grid head of every KV group must
    find its group's stride, and the phase of its vertical line (128 text
    tokens come first)."""
    wl = workloads.config1()
    q, k, _ = generate.make_qkv(wl, "cpu")
    G = wl.Hq // wl.Hkv
    firsts = {}
    for h, c in enumerate(wl.heads):
        if c.op.kind == C.OP_GRID:
            firsts.setdefault(h // G, h)
    assert sorted(firsts) == list(range(wl.Hkv))
    assert len(set(wl.structure.sigma)) > 1                   # the strides do differ
    for g, h in firsts.items():
        sig = wl.structure.sigma[g]
        K = numerics.torch_bf16_to_f64(k[:, g])
        qh = q[:, h]
        hp = P.plan_head(wl.heads[h], wl.S, wl.modality,
                         lambda r: numerics.torch_bf16_to_f64(qh[torch.as_tensor(r)]), K)
        st = hp.ops["g"]
        assert (st.sigma, st.p) == (sig, (128 + wl.structure.line_slot[g]) % sig), (g, h)
