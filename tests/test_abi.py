"""C-ABI checks that need no GPU: the library loads, exports every function
include/mmi.h declares, struct layouts agree, and host-side validation
returns the documented status codes without touching a device."""
import ctypes as ct
import os
import re

import numpy as np
import pytest

from paper_2504_16083_amd import mmi
from synth import config as C

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared():
    src = open(os.path.join(ROOT, "include", "mmi.h")).read()
    return sorted(set(re.findall(r"^\s*(?:int|const char\*)\s+(mmi_\w+)\s*\(", src, re.M)))


def test_every_declared_symbol_is_exported():
    names = declared()
    assert len(names) == 22 and set(names) == set(mmi.SYMBOLS)
    L = mmi.lib()
    for n in names:
        assert hasattr(L, n), n
    assert mmi.mmi_version() == 1
    assert mmi.mmi_status_str(0) == "ok"
    assert mmi.mmi_status_str(-3) == "bad head config"


def test_struct_sizes_match_header():
    # offsets of the trailing fields fix the layout of everything before them
    assert ct.sizeof(mmi.mmi_op) == 80
    assert ct.sizeof(mmi.mmi_head_cfg) == 4 + 80 + 8 * 80 + 64 * 80
    assert mmi.mmi_problem.modality.offset == 88 and ct.sizeof(mmi.mmi_problem) == 104
    assert mmi.mmi_index_view.union_ent.offset == 80 and ct.sizeof(mmi.mmi_index_view) == 88
    assert mmi.mmi_work_view.item_map.offset == 72 and ct.sizeof(mmi.mmi_work_view) == 80
    assert mmi.mmi_search_report.kind.offset == 152 and ct.sizeof(mmi.mmi_search_report) == 160


def _create(prob, heads, q=16, k=16):
    cfgs = mmi.head_cfgs(heads)
    h = ct.c_void_p()
    return mmi.lib().mmi_plan_create(None, ct.byref(prob.c), cfgs, ct.c_void_p(q), ct.c_void_p(k), None,
                                     ct.byref(h))


def test_search_arguments_without_device():
    """mmi_search refuses NULL pointers and bad candidate lists before it
    touches the context or the device."""
    L = mmi.lib()
    prob = mmi.Problem(100, 2, 1)
    tgt = mmi.op_struct(C.ashape(64, 256))
    cands = (mmi.mmi_op * 1)(mmi.op_struct(C.dense()))
    out = (mmi.mmi_head_cfg * 2)()
    dev = ct.c_void_p(1 << 20)                  # never dereferenced: the call fails first
    assert L.mmi_search(None, ct.byref(prob.c), dev, dev, dev, cands, 1, None, 0, ct.byref(tgt), None, out,
                        None) == -1
    assert "NULL" in mmi.mmi_last_error()
    assert L.mmi_search(None, ct.byref(prob.c), dev, dev, dev, cands, 1, None, 0, None, None, out,
                        None) == -1


def test_validation_codes_without_device():
    g = [C.global_head(C.dense())] * 2
    assert _create(mmi.Problem(100, 2, 1), g) == -1          # ctx NULL after valid args
    p = mmi.Problem(100, 2, 1); p.c.D = 64
    assert _create(p, g) == -2
    assert _create(mmi.Problem(100, 3, 2), [C.global_head(C.dense())] * 3) == -2
    assert _create(mmi.Problem(0, 2, 1), g) == -1
    assert _create(mmi.Problem((1 << 21) + 1, 2, 1), g) == -2
    assert _create(mmi.Problem(100, 2, 1), g, q=0) == -1
    assert _create(mmi.Problem(100, 2, 1), g, q=8) == -1      # misaligned
    assert _create(mmi.Problem(100, 2, 1), [C.global_head(C.grid(0, 5))] * 2) == -3
    assert _create(mmi.Problem(100, 2, 1), [C.global_head(C.grid(5, 2000))] * 2) == -3
    assert _create(mmi.Problem(100, 2, 1), [C.global_head(C.vert(5))] * 2) == -3
    mod = np.zeros(100, np.uint8); mod[50:] = 1
    assert _create(mmi.Problem(100, 2, 1, mod), [C.qboundary_head({1: C.grid(0, 8)})] * 2) == -3
    assert _create(mmi.Problem(100, 2, 1, mod), [C.qboundary_head({1: C.grid(4, 8)})] * 2) == -1  # valid
    big = np.zeros(1 << 21, np.uint8); big[1 << 20:] = 1      # 2 key layouts x 32768 blocks
    assert _create(mmi.Problem(1 << 21, 2, 1, big), [C.qboundary_head({1: C.grid(4, 8)})] * 2) == -2
    assert "key layouts" in mmi.mmi_last_error()
    assert _create(mmi.Problem(1 << 21, 2, 1, big), [C.qboundary_head({0: C.grid(4, 8), 1: C.grid(4, 8)})] * 2) == -2
    assert _create(mmi.Problem(1 << 20, 2, 1, big[1 << 19:3 << 19].copy()),       # 2 x 16384 blocks: fits
                   [C.qboundary_head({1: C.grid(4, 8)})] * 2) == -1
    nat = lambda grid, win, tile: [C.global_head(C.natten(grid, win, tile))] * 2
    assert _create(mmi.Problem(100, 2, 1), nat((1, 10, 10), (1, 3, 5), (1, 8, 8))) == -1       # valid
    assert _create(mmi.Problem(100, 2, 1), nat((1, 10, 10), (1, 4, 5), (1, 8, 8))) == -3       # even window
    assert _create(mmi.Problem(100, 2, 1), nat((1, 10, 10), (1, 3, 11), (1, 8, 8))) == -3      # window > axis
    assert _create(mmi.Problem(100, 2, 1), nat((1, 10, 11), (1, 3, 5), (1, 8, 8))) == -3       # grid != S
    assert _create(mmi.Problem(100, 2, 1), nat((1, 10, 10), (1, 3, 5), (1, 8, 4))) == -3       # tile != 64
    assert _create(mmi.Problem(100, 2, 1, mod), [C.qboundary_head({0: C.natten((1, 10, 10), (1, 3, 3), (1, 8, 8))})] * 2) == -3
    assert _create(mmi.Problem(1 << 20, 2, 1), nat((1, 1 << 10, 1 << 10), (1, 3, 3), (64, 1, 1))) == -2  # 2^20 tiles
    bad2d = C.boundary2d_head({0: C.dense(), 1: C.dense()}, {(0, 1): C.ashape(1, 1)})
    assert _create(mmi.Problem(100, 2, 1, mod), [bad2d] * 2) == -3
    assert "cross" in mmi.mmi_last_error()
    mod[3] = 9
    p = mmi.Problem(100, 2, 1, mod); p.c.n_modalities = 2
    assert _create(p, g) == -1
    # K/V token strides enter a 24-bit multiply in the attention kernel: at
    # most 2^23 - 8 elements (S = 100 keeps S x stride far below 2^31)
    for name in ("k", "v"):
        ok = mmi.Problem(100, 2, 1, strides={name: ((1 << 23) - 8, 128)})
        assert _create(ok, g) == -1                       # valid up to the ctx
        bad = mmi.Problem(100, 2, 1, strides={name: (1 << 23, 128)})
        assert _create(bad, g) == -2 and "2^23" in mmi.mmi_last_error()


def test_ctx_without_device_is_an_error():
    h = ct.c_void_p()
    rc = mmi.lib().mmi_ctx_create(0, ct.byref(h))
    try:
        import torch
        has_gpu = torch.cuda.is_available()
    except Exception:
        has_gpu = False
    if has_gpu:
        assert rc == 0
        mmi.lib().mmi_ctx_destroy(h)
    else:
        assert rc in (-1, -5) and mmi.mmi_last_error()


def test_stats_struct_matches_header():
    # kind, n_qblocks, n_kblocks (12) + pad (4) + 2 x int64 (16) + split_rows (4) + 2 x 8 int32 (64)
    assert mmi.mmi_head_stats.group_stride.offset == 100
    assert mmi.mmi_head_stats.loaded_blocks.offset == 104
    assert mmi.mmi_head_stats.blocks_by_modality.offset == 112
    assert ct.sizeof(mmi.mmi_head_stats) == 112 + 64 * 8


def test_head_cfg_marshalling_fills_every_op():
    """head_cfgs (a repeated config marshalled once, cross pairs only where
    set) writes the same bytes as filling every op of every head."""
    from synth import workloads

    def full(heads):
        arr = (mmi.mmi_head_cfg * len(heads))()
        for i, h in enumerate(heads):
            c = arr[i]
            c.kind = h.kind
            c.global_ = mmi.op_struct(h.op)
            for m in range(mmi.MAXM):
                c.intra[m] = mmi.op_struct(h.intra_op(m))
                for mk in range(mmi.MAXM):
                    c.cross[m][mk] = mmi.op_struct(h.cross_op(m, mk))
        return arr

    for cid in (2, 4):
        heads = workloads.by_id(cid).heads
        assert bytes(mmi.head_cfgs(heads)) == bytes(full(heads))


def test_head_cfg_cache_follows_values():
    """Marshalled configs are cached by value: a config changed in place
    marshals to its new value, equal configs to equal bytes."""
    h = C.global_head(C.ashape(128, 1024))
    a = bytes(mmi.head_cfgs([h, h]))
    h.op = C.ashape(128, 2048)
    b = bytes(mmi.head_cfgs([h, h]))
    assert a != b
    assert b == bytes(mmi.head_cfgs([C.global_head(C.ashape(128, 2048))] * 2))
    q = C.qboundary_head({1: C.grid(4, 8)})
    before = bytes(mmi.head_cfgs([q]))
    q.intra[0] = C.ashape(64, 512)
    assert bytes(mmi.head_cfgs([q])) != before
