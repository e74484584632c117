"""Per-head pattern configuration: plain data, no arithmetic of the method.

The paper's offline search (Appendix A, Algorithm 4) outputs, for every
attention head, which sparse pattern to use and its parameters; at inference
that choice is an input (Section 3, opening paragraph). These dataclasses hold
that input. Both the HIP path (through the C-ABI marshalling) and the CPU
oracle read them; neither side computes anything here.

Search-space values come from the paper's Table "search space" (Appendix C.5):
Grid = (stride | frame_stride, use_hline, use_vline, use_slash, max_stride=1024),
A-shape = (sink, local), Vertical-Slash = (vertical_size, slash_size).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, Optional, Tuple

# Operation kinds (same integer codes as include/mmi.h MMI_OP_*).
OP_NONE, OP_DENSE, OP_ASHAPE, OP_VSLASH, OP_GRID, OP_VERT = 0, 1, 2, 3, 4, 5
OP_SF_FIXED, OP_SF_STRIDED, OP_TRISHAPE = 6, 7, 8      # static baselines (Section 4.1)
OP_NATTEN = 9              # 2D/3D neighborhood attention through a tile permutation (Appendix F)
OP_NAMES = {OP_NONE: "none", OP_DENSE: "dense", OP_ASHAPE: "ashape",
            OP_VSLASH: "vslash", OP_GRID: "grid", OP_VERT: "vert",
            OP_SF_FIXED: "sf_fixed", OP_SF_STRIDED: "sf_strided", OP_TRISHAPE: "trishape",
            OP_NATTEN: "natten"}
STATIC_OPS = (OP_DENSE, OP_ASHAPE, OP_SF_FIXED, OP_SF_STRIDED, OP_TRISHAPE)

# Head kinds (include/mmi.h MMI_HEAD_*): a global op over all rows (the
# No-Boundary / K-Boundary case of Section 3.2), Q-Boundary, 2D-Boundary.
HEAD_GLOBAL, HEAD_QBOUNDARY, HEAD_2D = 0, 1, 2
HEAD_NO_BOUNDARY = HEAD_K_BOUNDARY = HEAD_GLOBAL   # index continuous along queries (Appendix B.1)

MAX_STRIDE = 1024          # Table "search space": max stride
MAX_MODALITIES = 8
LAST_Q = 64                # Section 4.1: last_q = 64 for VS and Grid estimation


@dataclass(frozen=True)
class Op:
    kind: int = OP_DENSE
    sink: int = 0
    local: int = 0
    n_vertical: int = 0
    n_slash: int = 0
    stride_lo: int = 0
    stride_hi: int = 0
    use_h: bool = False
    use_v: bool = False
    use_s: bool = False
    bottom: int = 0
    grid: tuple = (0, 0, 0)        # NATTEN token grid (T, H, W), raster order, W fastest
    win: tuple = (0, 0, 0)         # NATTEN neighborhood size per axis (odd)
    tile: tuple = (0, 0, 0)        # NATTEN permutation tile, product 64


def dense() -> Op:
    return Op(OP_DENSE)


def none() -> Op:
    return Op(OP_NONE)


def ashape(sink: int, local: int) -> Op:
    return Op(OP_ASHAPE, sink=sink, local=local)


def vslash(n_vertical: int, n_slash: int) -> Op:
    return Op(OP_VSLASH, n_vertical=n_vertical, n_slash=n_slash)


def sf_fixed(segment: int, stride: int) -> Op:
    """Sparse Transformer "fixed": attend within the own segment of `segment`
    tokens and to every key at a multiple of `stride` (the segments' first
    tokens when stride == segment)."""
    return Op(OP_SF_FIXED, local=segment, stride_lo=stride)


def sf_strided(local: int, stride: int) -> Op:
    """Sparse Transformer "strided": a local window plus every key at a
    distance that is a multiple of `stride` (dilated slash lines)."""
    return Op(OP_SF_STRIDED, local=local, stride_lo=stride)


def trishape(sink: int, local: int, bottom: int) -> Op:
    """A-shape plus full attention for the final `bottom` queries."""
    return Op(OP_TRISHAPE, sink=sink, local=local, bottom=bottom)


def natten(grid, win, tile) -> Op:
    """Neighborhood attention over a (T, H, W) token grid (T = 1 for images),
    bidirectional: each token sees the win_t x win_h x win_w neighborhood
    around it, shifted inside the grid at the borders. Tokens are permuted
    tile by tile (tile_t x tile_h x tile_w = 64 tokens = one block); the tile
    shape is the caller's choice."""
    grid, win = tuple(int(x) for x in grid), tuple(int(x) for x in win)
    return Op(OP_NATTEN, grid=grid, win=win, tile=tuple(int(x) for x in tile))


def natten_tiles():
    """Tile shapes (powers of two, 64 tokens)."""
    return [(1 << a, 1 << b, 1 << (6 - a - b)) for a in range(7) for b in range(7 - a)]


def vert(n: int) -> Op:
    return Op(OP_VERT, n_vertical=n)


def grid(lo: int, hi: int, h: bool = True, v: bool = True, s: bool = True) -> Op:
    return Op(OP_GRID, stride_lo=lo, stride_hi=hi, use_h=h, use_v=v, use_s=s)


def grid_frame(frame: int, h=True, v=True, s=True) -> Op:
    """'frame_stride' entry of the search space: the stride is the frame size."""
    return grid(frame, frame, h, v, s)


def grid_window(frame: int, half: int = 8, h=True, v=True, s=True) -> Op:
    """'stride' entry of the search space: search strides around the frame size."""
    return grid(max(1, frame - half), min(MAX_STRIDE, frame + half), h, v, s)


@dataclass
class HeadCfg:
    kind: int = HEAD_GLOBAL
    op: Op = field(default_factory=dense)                  # HEAD_GLOBAL
    intra: Dict[int, Op] = field(default_factory=dict)      # modality -> op
    cross: Dict[Tuple[int, int], Op] = field(default_factory=dict)  # (mq, mk) -> op

    def intra_op(self, m: int) -> Op:
        return self.intra.get(m, dense())

    def cross_op(self, mq: int, mk: int) -> Op:
        return self.cross.get((mq, mk), none())


def global_head(op: Op) -> HeadCfg:
    return HeadCfg(HEAD_GLOBAL, op=op)


def no_boundary_head(op: Op) -> HeadCfg:
    """No modality boundary: the intra-modality op over all rows."""
    return HeadCfg(HEAD_NO_BOUNDARY, op=op)


def k_boundary_head(op: Op) -> HeadCfg:
    """Boundaries along the key axis only: the index is continuous along the
    query axis, so the intra-modality op applies over all rows (Appendix B.1)."""
    return HeadCfg(HEAD_K_BOUNDARY, op=op)


def qboundary_head(intra: Dict[int, Op]) -> HeadCfg:
    return HeadCfg(HEAD_QBOUNDARY, intra=dict(intra))


def boundary2d_head(intra: Dict[int, Op], cross: Dict[Tuple[int, int], Op]) -> HeadCfg:
    return HeadCfg(HEAD_2D, intra=dict(intra), cross=dict(cross))


@dataclass
class Problem:
    """Shape of one attention layer (batch 1, causal, head_dim 128, block 64)."""
    S: int
    Hq: int
    Hkv: int
    modality: Optional[object] = None   # numpy uint8 [S] or None (= all modality 0)
    D: int = 128
    block: int = 64
