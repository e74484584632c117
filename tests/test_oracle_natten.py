"""Pins of the oracle's neighborhood attention (Appendix F, permuted 2D/3D
sliding windows): the window rule against a brute-force nearest-window
search, the tile permutation, closed-form blocks against token-pair
enumeration, and the bidirectional attention path against torch."""
import numpy as np
import pytest
import torch

from oracle import attention as A
from oracle import natten as N
from oracle import plan as P
from synth import config as C


def _plan(grid, win, tile):
    op = C.natten(grid, win, tile)
    S = int(np.prod(grid))
    return P.assemble(C.HEAD_GLOBAL, S, None, {"g": P.OpState(C.OP_NATTEN, op, L=S)})


def test_window_start_is_the_nearest_centred_window():
    for n in range(1, 24):
        for k in range(1, n + 1, 2):
            for c in range(n):
                # brute force: the k-window inside [0, n) whose centre is closest to c
                best = min(range(0, n - k + 1), key=lambda s: abs(s + k // 2 - c))
                s = int(N.window_start(c, n, k))
                assert s == best and s <= c < s + k


def test_tile_permutation_bijection():
    rng = np.random.default_rng(1)
    for _ in range(20):
        grid = (int(rng.integers(1, 5)), int(rng.integers(1, 20)), int(rng.integers(1, 20)))
        tile = C.natten_tiles()[int(rng.integers(0, len(C.natten_tiles())))]
        perm = N.permutation(grid, tile)
        assert len(perm) % 64 == 0
        live = perm[perm >= 0]
        assert sorted(live.tolist()) == list(range(int(np.prod(grid))))
        # inside a tile, tokens are in raster order
        for blk in perm.reshape(-1, 64):
            b = blk[blk >= 0]
            assert (np.diff(b) > 0).all()


def test_closed_form_equals_literal_lift():
    rng = np.random.default_rng(2)
    for _ in range(40):
        grid = (int(rng.integers(1, 6)), int(rng.integers(1, 26)), int(rng.integers(1, 26)))
        win = tuple(int(rng.integers(0, (n + 1) // 2)) * 2 + 1 for n in grid)
        tile = C.natten_tiles()[int(rng.integers(0, len(C.natten_tiles())))]
        hp = _plan(grid, win, tile)
        lifted = P.lift_blocks(hp)
        assert all(np.array_equal(a, b) for a, b in zip(hp.blocks, lifted)), (grid, win, tile)


def test_full_and_unit_windows():
    grid, tile = (3, 10, 12), (2, 4, 8)
    hp = _plan(grid, (3, 9, 11), tile)
    hp_full = _plan((3, 9, 11), (3, 9, 11), tile)
    assert all(len(b) == hp_full.nbq for b in hp_full.blocks)
    hp1 = _plan(grid, (1, 1, 1), tile)
    assert all(b.tolist() == [i] for i, b in enumerate(hp1.blocks))
    q = 77
    keys = P.element_mask_row(hp1, q)
    blk = hp1.kperm[(int(np.nonzero(hp1.qperm == q)[0][0]) // 64) * 64:][:64]
    assert np.array_equal(keys, np.sort(blk[blk >= 0]))
    assert hp.causal is False


def test_known_blocks_2d():
    """24 x 24 image, 8 x 8 tiles (3 x 3 tiles), 3 x 3 window. Tile (0, 0)
    covers rows/cols 0-7; its windows reach 8 -> key tiles (0..1) x (0..1)
    = {0, 1, 3, 4}. Tile (1, 1) covers 8-15, windows 7-16 -> all 9 tiles.
    Tile (2, 2) covers 16-23, windows 15-23 -> {4, 5, 7, 8}."""
    hp = _plan((1, 24, 24), (1, 3, 3), (1, 8, 8))
    assert hp.blocks[0].tolist() == [0, 1, 3, 4]
    assert hp.blocks[4].tolist() == list(range(9))
    assert hp.blocks[8].tolist() == [4, 5, 7, 8]
    assert hp.qperm[:10].tolist() == [0, 1, 2, 3, 4, 5, 6, 7, 24, 25]


def test_bidirectional_attention_matches_torch():
    """Full neighborhood = every token sees every token: the oracle's rows
    and its blockwise online-softmax path equal torch's non-causal SDPA."""
    rng = np.random.default_rng(3)
    grid = (3, 5, 7)
    S = 105
    hp = _plan(grid, grid, (1, 8, 8))
    Q, K, V = (rng.standard_normal((S, 128)) for _ in range(3))
    ref = torch.nn.functional.scaled_dot_product_attention(
        *(torch.from_numpy(x)[None, None] for x in (Q, K, V)), is_causal=False)[0, 0].numpy()
    O, L = A.head_rows(hp, Q, K, V, np.arange(S))
    assert np.abs(O - ref).max() < 1e-12
    O2, L2 = A.permuted_blockwise(hp, Q, K, V)
    assert np.abs(O2 - ref).max() < 1e-12 and np.abs(L2 - L).max() < 1e-12

