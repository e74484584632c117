"""Inputs of the modality-aware pattern search (Appendix A, Algorithm 4;
Appendix C.5): the candidate lists and the FLOPs target. Data only.

Intra-modality candidates: the paper's Table "search space" — Grid
(frame_stride | stride, use_hline, use_vline, use_slash, max stride 1024),
A-shape (sink, local), Vertical-Slash (vertical size, slash size), values as
printed (3096 included). frame_stride: the stride is the frame size;
stride: strides searched within 8 of the frame size.

FLOPs target (Appendix C.5): the work of an A-shape head with 1k global
(sink) tokens and a 4k local window.

Cross-modality candidates (2D-Boundary pairs; the paper lists none, so this
is a reading): no keys, the n best key columns of the key modality for n in
256, 512, 1024, 2048, or every key.
"""
from __future__ import annotations

from typing import List, Tuple

from . import config as C

GRID_TABLE = [
    ("frame_stride", True, False, False, 1024), ("frame_stride", False, True, False, 1024),
    ("frame_stride", False, False, True, 1024), ("frame_stride", True, True, False, 1024),
    ("frame_stride", False, True, True, 1024), ("frame_stride", True, True, True, 1024),
    ("stride", True, False, False, 1024), ("stride", False, True, False, 1024),
    ("stride", False, False, True, 1024), ("stride", True, True, False, 1024),
    ("stride", False, True, True, 1024), ("stride", True, True, True, 1024),
]
ASHAPE_TABLE = [(128, 1024), (128, 2048), (128, 4096)]
VSLASH_TABLE = [(1000, 1024), (1000, 2048), (2000, 2048), (1000, 3096), (2000, 3096),
                (1000, 4096), (2000, 4096), (3500, 200), (1000, 2500)]
STRIDE_HALF_WINDOW = 8
BUDGET_SINK, BUDGET_LOCAL = 1024, 4096
CROSS_VERT_SIZES = [256, 512, 1024, 2048]


def intra_candidates(frame: int) -> List[Tuple[str, C.Op]]:
    """(name, op) in table order: Grid, A-shape, Vertical-Slash."""
    out = []
    for mode, h, v, s, mx in GRID_TABLE:
        assert mx == C.MAX_STRIDE
        op = C.grid_frame(frame, h, v, s) if mode == "frame_stride" else \
            C.grid_window(frame, STRIDE_HALF_WINDOW, h, v, s)
        out.append((f"grid_{mode}_{int(h)}{int(v)}{int(s)}", op))
    out += [(f"ashape_{a}_{b}", C.ashape(a, b)) for a, b in ASHAPE_TABLE]
    out += [(f"vslash_{a}_{b}", C.vslash(a, b)) for a, b in VSLASH_TABLE]
    return out


def cross_candidates() -> List[Tuple[str, C.Op]]:
    return ([("none", C.none())] + [(f"vert_{n}", C.vert(n)) for n in CROSS_VERT_SIZES]
            + [("dense", C.dense())])


def budget_op() -> C.Op:
    return C.ashape(BUDGET_SINK, BUDGET_LOCAL)
