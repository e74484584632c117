"""Neighborhood attention over a token grid, made block-dense by a tile
permutation (Appendix F: 2D/3D sliding-window attention of DiT models turned
into dense blocks by permuting the tokens).

Token grid (T, H, W) in raster order: position x = (t * H + h) * W + w.
Neighborhood (reading): along each axis of length n with odd window k, the
window of coordinate c is the k consecutive coordinates starting at
start(c) = min(max(c - k // 2, 0), n - k): centred on c, shifted inside the
grid at the borders, so every token sees exactly k_t * k_h * k_w tokens.
Attention is bidirectional (no causal condition).

Permutation: the grid is cut into tiles of (tt, th, tw) tokens with
tt * th * tw = 64; tiles in raster order, tokens in raster order inside a
tile; a tile cut by the grid border is padded with -1 to 64 slots, so tile i
is block i for queries and keys alike.

Pinned in tests/test_oracle_natten.py: start() against the brute-force
nearest-window definition, the permutation is a bijection, closed-form
blocks == token-pair enumeration, full windows give every block.
"""
import numpy as np

B = 64


def window_start(c, n: int, k: int):
    """First coordinate of the window of coordinate(s) c on an axis of length n."""
    return np.minimum(np.maximum(np.asarray(c) - k // 2, 0), n - k)


def coords(pos, grid):
    T, H, W = grid
    pos = np.asarray(pos)
    return pos // (H * W), (pos // W) % H, pos % W


def predicate(qpos, kpos, grid, win):
    """Key in the query's neighborhood (broadcasting position arrays)."""
    out = None
    for qc, kc, n, k in zip(coords(qpos, grid), coords(kpos, grid), grid, win):
        s = window_start(qc, n, k)
        hit = (kc >= s) & (kc < s + k)
        out = hit if out is None else out & hit
    return out


def tile_counts(grid, tile):
    return tuple(-(-n // t) for n, t in zip(grid, tile))


def permutation(grid, tile):
    """slot -> position (-1 for padding), 64 slots per tile."""
    T, H, W = grid
    tt, th, tw = tile
    nt = tile_counts(grid, tile)
    out = np.full(nt[0] * nt[1] * nt[2] * B, -1, dtype=np.int64)
    x = 0
    for a in range(nt[0]):
        for b in range(nt[1]):
            for c in range(nt[2]):
                for i in range(tt):
                    for j in range(th):
                        for l in range(tw):
                            t, h, w = a * tt + i, b * th + j, c * tw + l
                            if t < T and h < H and w < W:
                                out[x] = (t * H + h) * W + w
                            x += 1
    return out


def tile_blocks(grid, win, tile, i: int):
    """Key tiles of query tile i: per axis the union of the windows of the
    tile's coordinates is one interval (start() is monotone and grows by at
    most 1 per step); the key tiles are those meeting the product of the
    intervals."""
    nt = tile_counts(grid, tile)
    idx = (i // (nt[1] * nt[2]), (i // nt[2]) % nt[1], i % nt[2])
    ranges = []
    for a, n, k, t in zip(idx, grid, win, tile):
        c0, c1 = a * t, min(n, a * t + t) - 1
        lo = int(window_start(c0, n, k))
        hi = int(window_start(c1, n, k)) + k - 1
        ranges.append(range(lo // t, hi // t + 1))
    return sorted((x * nt[1] + y) * nt[2] + z for x in ranges[0] for y in ranges[1] for z in ranges[2])
