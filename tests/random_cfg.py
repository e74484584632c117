"""Seeded random head configurations over every head kind and op (test
infrastructure: input recipes only, no arithmetic of the method)."""
import numpy as np

from synth import config as C


def random_layout(rng, S, nmod):
    mod = np.zeros(S, np.uint8)
    pos, m = 0, 0
    while pos < S:
        n = int(rng.integers(1, max(2, S // 3)))
        mod[pos:pos + n] = m
        pos += n
        m = (m + 1 + int(rng.integers(0, nmod - 1 if nmod > 1 else 1))) % nmod
    return mod


def random_op(rng, allow_grid=True, allow_vs=True):
    kinds = ["dense", "ashape", "trishape", "sf_fixed", "sf_strided"] + (["vslash"] if allow_vs else []) \
        + (["grid"] if allow_grid else [])
    k = kinds[int(rng.integers(0, len(kinds)))]
    r = lambda a, b: int(rng.integers(a, b))
    if k == "dense":
        return C.dense()
    if k == "ashape":
        return C.ashape(r(0, 200), r(1, 700))
    if k == "trishape":
        return C.trishape(r(0, 100), r(0, 500), r(0, 300))
    if k == "sf_fixed":
        return C.sf_fixed(r(1, 400), r(1, 400))
    if k == "sf_strided":
        return C.sf_strided(r(1, 300), r(1, 400))
    if k == "vslash":
        return C.vslash(r(0, 60), r(0, 60))
    lo = r(1, 120)
    h, v, s = (bool(rng.integers(0, 2)) for _ in range(3))
    return C.grid(lo, lo + r(0, 30), h, v, s)


def factor3(rng, S):
    """A (T, H, W) grid with T*H*W = S."""
    divs = [d for d in range(1, S + 1) if S % d == 0]
    T = divs[int(rng.integers(0, min(len(divs), 4)))]
    rest = S // T
    d2 = [d for d in range(1, rest + 1) if rest % d == 0]
    H = d2[int(rng.integers(0, len(d2)))]
    return T, H, rest // H


def random_head(rng, S, mods):
    k = int(rng.integers(0, 4 if len(mods) > 1 else 2))
    if k == 0:
        return C.global_head(random_op(rng))
    if k == 1:
        g = factor3(rng, S)
        win = tuple(int(rng.integers(0, (n + 1) // 2)) * 2 + 1 for n in g)
        tiles = C.natten_tiles()
        return C.global_head(C.natten(g, win, tiles[(7 * g[0] + 3 * g[1] + g[2]) % len(tiles)]))
    if k == 2:
        return C.qboundary_head({m: random_op(rng) for m in mods})
    cross = {}
    for a in mods:
        for b in mods:
            if a != b:
                x = int(rng.integers(0, 3))
                cross[(a, b)] = [C.none(), C.dense(), C.vert(int(rng.integers(1, 80)))][x]
    return C.boundary2d_head({m: random_op(rng) for m in mods}, cross)
