"""ctypes binding of libmmi.so (include/mmi.h): argument marshalling only.

Every function here converts Python/torch arguments to the C structs and
device pointers of the C-ABI and calls the library; all computation runs in
the HIP kernels. Loading fails loudly when libmmi.so has not been built.
"""
from __future__ import annotations

import atexit
import ctypes as ct
import os
import weakref

import numpy as np

from synth import config as C

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmmi.so")

MAXM = 8
OK = 0
ERR_INTERNAL = -7
EXPORT = dict(qperm=0, kperm=1, row_ptr=2, col_idx=3, v=4, u=5, fold=6, vsel=7, ssel=8, params=9, est_lse=10,
              union_ptr=11, union=12)
_F32 = {"v", "u", "fold", "est_lse"}


class MMIError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"mmi status {status}: {msg}")
        self.status = status


class mmi_op(ct.Structure):
    _fields_ = [("kind", ct.c_int32), ("sink", ct.c_int32), ("local", ct.c_int32),
                ("n_vertical", ct.c_int32), ("n_slash", ct.c_int32),
                ("stride_lo", ct.c_int32), ("stride_hi", ct.c_int32),
                ("use_h", ct.c_int32), ("use_v", ct.c_int32), ("use_s", ct.c_int32), ("bottom", ct.c_int32),
                ("grid_t", ct.c_int32), ("grid_h", ct.c_int32), ("grid_w", ct.c_int32),
                ("win_t", ct.c_int32), ("win_h", ct.c_int32), ("win_w", ct.c_int32),
                ("tile_t", ct.c_int32), ("tile_h", ct.c_int32), ("tile_w", ct.c_int32)]


class mmi_head_cfg(ct.Structure):
    _fields_ = [("kind", ct.c_int32), ("global_", mmi_op), ("intra", mmi_op * MAXM),
                ("cross", (mmi_op * MAXM) * MAXM)]


class mmi_problem(ct.Structure):
    _fields_ = [("S", ct.c_int64), ("Hq", ct.c_int32), ("Hkv", ct.c_int32), ("D", ct.c_int32),
                ("block", ct.c_int32),
                ("q_stride_s", ct.c_int64), ("q_stride_h", ct.c_int64),
                ("k_stride_s", ct.c_int64), ("k_stride_h", ct.c_int64),
                ("v_stride_s", ct.c_int64), ("v_stride_h", ct.c_int64),
                ("o_stride_s", ct.c_int64), ("o_stride_h", ct.c_int64),
                ("modality", ct.POINTER(ct.c_uint8)), ("n_modalities", ct.c_int32)]


class mmi_head_stats(ct.Structure):
    _fields_ = [("kind", ct.c_int32), ("n_qblocks", ct.c_int32), ("n_kblocks", ct.c_int32),
                ("nnz_blocks", ct.c_int64), ("causal_blocks", ct.c_int64), ("split_rows", ct.c_int32),
                ("sigma", ct.c_int32 * MAXM), ("phase", ct.c_int32 * MAXM), ("group_stride", ct.c_int32),
                ("loaded_blocks", ct.c_int64), ("blocks_by_modality", (ct.c_int64 * MAXM) * MAXM)]


class mmi_plan_timing(ct.Structure):
    _fields_ = [("est_ms", ct.c_float), ("select_ms", ct.c_float), ("index_ms", ct.c_float),
                ("attn_ms", ct.c_float), ("combine_ms", ct.c_float), ("computed_blocks", ct.c_int64),
                ("work_items", ct.c_int64), ("loaded_blocks", ct.c_int64), ("device_bytes", ct.c_int64)]


I32P = ct.POINTER(ct.c_int32)


class mmi_index_view(ct.Structure):
    _fields_ = [("S", ct.c_int32), ("n_qblocks", ct.c_int32), ("n_kblocks", ct.c_int32),
                ("n_layouts", ct.c_int32), ("causal", ct.c_int32), ("qperm", I32P), ("kperm", I32P),
                ("row_ptr", I32P), ("col_idx", I32P), ("group_size", ct.c_int32), ("group_stride", ct.c_int32),
                ("n_groups", ct.c_int32), ("union_ptr", I32P), ("union_ent", I32P)]


class mmi_work_view(ct.Structure):
    _fields_ = [("n_heads", ct.c_int32), ("n_groups", I32P), ("union_ptr", ct.POINTER(I32P)),
                ("n_items", ct.c_int64), ("items", I32P), ("n_parts", ct.c_int64), ("n_splits", ct.c_int64),
                ("splits", I32P), ("map_len", ct.c_int64), ("item_map", I32P)]


I64P, F64P = ct.POINTER(ct.c_int64), ct.POINTER(ct.c_double)


class mmi_search_report(ct.Structure):
    _fields_ = [("n_mod", ct.c_int32), ("mods", ct.c_int32 * MAXM), ("plans", ct.c_int64),
                ("budget1", I64P), ("step1_cost", I64P), ("step1_err", F64P), ("intra", I32P),
                ("step2_cost", I64P), ("step2_err", F64P), ("cross", I32P), ("budget3", I64P),
                ("step3g_cost", I64P), ("step3g_err", F64P), ("global_", I32P), ("step3_cost", I64P),
                ("step3_err", F64P), ("kind", I32P)]


SYMBOLS = ["mmi_search", "mmi_plan_timing_get", "mmi_version", "mmi_status_str", "mmi_last_error", "mmi_ctx_create", "mmi_ctx_destroy",
           "mmi_plan_create", "mmi_plan_execute", "mmi_plan_stats", "mmi_plan_export",
           "mmi_plan_destroy", "mmi_attention", "mmi_dense_attention", "mmi_permute_rows",
           "mmi_unpermute_rows", "mmi_output_sqerr", "mmi_attention_noalloc", "mmi_check_index",
           "mmi_check_work", "mmi_plan_check", "mmi_plan_pair_counts"]

_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: run __graft_entry__.build() first")
        L = ct.CDLL(LIB_PATH)
        vp, i32, i64, sz = ct.c_void_p, ct.c_int, ct.c_int64, ct.c_size_t
        sig = {
            "mmi_version": ([], i32), "mmi_status_str": ([i32], ct.c_char_p),
            "mmi_last_error": ([], ct.c_char_p),
            "mmi_ctx_create": ([i32, ct.POINTER(vp)], i32), "mmi_ctx_destroy": ([vp], i32),
            "mmi_plan_create": ([vp, ct.POINTER(mmi_problem), ct.POINTER(mmi_head_cfg), vp, vp, vp,
                                 ct.POINTER(vp)], i32),
            "mmi_plan_execute": ([vp, vp, vp, vp, vp, vp, vp], i32),
            "mmi_plan_stats": ([vp, i32, ct.POINTER(mmi_head_stats)], i32),
            "mmi_plan_export": ([vp, i32, i32, i32, vp, sz, ct.POINTER(sz)], i32),
            "mmi_plan_destroy": ([vp], i32),
            "mmi_plan_timing_get": ([vp, ct.POINTER(mmi_plan_timing)], i32),
            "mmi_attention": ([vp, ct.POINTER(mmi_problem), ct.POINTER(mmi_head_cfg), vp, vp, vp, vp, vp,
                               vp], i32),
            "mmi_attention_noalloc": ([vp, ct.POINTER(mmi_problem), ct.POINTER(mmi_head_cfg), vp, vp, vp, vp,
                                       vp, vp], i32),
            "mmi_dense_attention": ([vp, ct.POINTER(mmi_problem), vp, vp, vp, vp, vp, vp], i32),
            "mmi_permute_rows": ([vp, i64, vp, i64, vp, i64, i64, vp], i32),
            "mmi_unpermute_rows": ([vp, i64, vp, i64, vp, i64, i64, vp], i32),
            "mmi_output_sqerr": ([ct.POINTER(mmi_problem), vp, vp, vp, i32, vp, vp], i32),
            "mmi_check_index": ([ct.POINTER(mmi_index_view)], i32),
            "mmi_check_work": ([ct.POINTER(mmi_work_view)], i32),
            "mmi_plan_check": ([vp], i32),
            "mmi_plan_pair_counts": ([vp, i32, ct.POINTER(ct.c_int64), ct.POINTER(ct.c_int64)], i32),
            "mmi_search": ([vp, ct.POINTER(mmi_problem), vp, vp, vp, ct.POINTER(mmi_op), i32, ct.POINTER(mmi_op),
                            i32, ct.POINTER(mmi_op), vp, ct.POINTER(mmi_head_cfg),
                            ct.POINTER(mmi_search_report)], i32),
        }
        for name, (args, res) in sig.items():
            f = getattr(L, name)
            f.argtypes, f.restype = args, res
        _lib = L
    return _lib


def _check(status):
    if status != OK:
        raise MMIError(status, lib().mmi_last_error().decode(errors="replace"))


def _ptr(t):
    return None if t is None else ct.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        import torch
        stream = torch.cuda.current_stream()
    return ct.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def mmi_version() -> int:
    return lib().mmi_version()


def mmi_status_str(s: int) -> str:
    return lib().mmi_status_str(s).decode()


def mmi_last_error() -> str:
    return lib().mmi_last_error().decode(errors="replace")


# ------------------------------------------------------------------ marshalling
def op_struct(op: C.Op) -> mmi_op:
    return mmi_op(op.kind, op.sink, op.local, op.n_vertical, op.n_slash, op.stride_lo, op.stride_hi,
                  int(op.use_h), int(op.use_v), int(op.use_s), op.bottom, *op.grid, *op.win, *op.tile)


def _head_cfg(h) -> mmi_head_cfg:
    c = mmi_head_cfg()                 # zero-filled: every op not set below is MMI_OP_NONE
    c.kind = h.kind
    c.global_ = op_struct(h.op)
    for m in range(MAXM):
        c.intra[m] = op_struct(h.intra_op(m))
    for (mq, mk), op in h.cross.items():
        c.cross[mq][mk] = op_struct(op)
    return c


def _cfg_key(h):
    """Value of a head config (its ops are immutable; the config itself may
    be changed between calls, so it is keyed by what it holds)."""
    return (h.kind, h.op, tuple(sorted(h.intra.items())), tuple(sorted(h.cross.items())))


_cfg_cache = {}      # value of one head config -> marshalled mmi_head_cfg
_cfgs_cache = {}     # values of a head list -> marshalled array
_CACHE_MAX = 256


def head_cfgs(heads) -> ct.Array:
    """mmi_head_cfg array for the heads. Marshalled configs are cached by
    value (the library reads the array only during the call it is passed to,
    so one array may serve several plans)."""
    keys = tuple(_cfg_key(h) for h in heads)
    arr = _cfgs_cache.get(keys)
    if arr is None:
        arr = (mmi_head_cfg * len(heads))()
        for i, (h, key) in enumerate(zip(heads, keys)):
            c = _cfg_cache.get(key)
            if c is None:
                if len(_cfg_cache) >= _CACHE_MAX:
                    _cfg_cache.clear()
                c = _cfg_cache[key] = _head_cfg(h)
            arr[i] = c
        if len(_cfgs_cache) >= _CACHE_MAX:
            _cfgs_cache.clear()
        _cfgs_cache[keys] = arr
    return arr


class Problem:
    """mmi_problem for packed [S, H, 128] tensors (or explicit strides)."""

    def __init__(self, S, Hq, Hkv, modality=None, strides=None):
        self.mod = None if modality is None else np.ascontiguousarray(modality, dtype=np.uint8)
        p = mmi_problem()
        p.S, p.Hq, p.Hkv, p.D, p.block = S, Hq, Hkv, 128, 64
        for name, (ss, sh) in (strides or {}).items():
            setattr(p, f"{name}_stride_s", ss)
            setattr(p, f"{name}_stride_h", sh)
        if self.mod is not None:
            p.modality = self.mod.ctypes.data_as(ct.POINTER(ct.c_uint8))
            p.n_modalities = int(self.mod.max()) + 1
        self.c = p


_live_ctx = weakref.WeakSet()


class Ctx:
    """mmi_ctx; closing it first destroys every plan still alive on it."""

    def __init__(self, device: int = 0):
        h = ct.c_void_p()
        _check(lib().mmi_ctx_create(device, ct.byref(h)))
        self.h = h
        self.plans = weakref.WeakSet()
        _live_ctx.add(self)

    def close(self):
        if self.h:
            for p in list(self.plans):
                p.destroy()
            _check(lib().mmi_ctx_destroy(self.h))
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def mmi_ctx_create(device: int = 0) -> Ctx:
    return Ctx(device)


class Plan:
    def __init__(self, ctx: Ctx, prob: Problem, heads, q, k, stream=None):
        self.ctx, self.prob = ctx, prob
        self.cfgs = head_cfgs(heads)
        h = ct.c_void_p()
        _check(lib().mmi_plan_create(ctx.h, ct.byref(prob.c), self.cfgs, _ptr(q), _ptr(k), _stream(stream),
                                     ct.byref(h)))
        self.h = h
        ctx.plans.add(self)

    def execute(self, q, k, v, o, lse=None, stream=None):
        _check(lib().mmi_plan_execute(self.h, _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), _stream(stream)))

    def stats(self, head: int) -> mmi_head_stats:
        s = mmi_head_stats()
        _check(lib().mmi_plan_stats(self.h, head, ct.byref(s)))
        return s

    def timing(self) -> dict:
        t = mmi_plan_timing()
        _check(lib().mmi_plan_timing_get(self.h, ct.byref(t)))
        return {f: getattr(t, f) for f, _ in mmi_plan_timing._fields_}

    def export(self, head: int, what: str, slot: int = 0) -> np.ndarray:
        need = ct.c_size_t()
        code = EXPORT[what]
        _check(lib().mmi_plan_export(self.h, head, code, slot, None, 0, ct.byref(need)))
        dt = np.float32 if what in _F32 else np.int32
        out = np.zeros(need.value // 4, dtype=dt)
        if need.value:
            _check(lib().mmi_plan_export(self.h, head, code, slot, out.ctypes.data_as(ct.c_void_p), need.value,
                                         ct.byref(need)))
        return out

    def pair_counts(self, head: int):
        """(useful, computed) query-key pairs of the head's selected blocks."""
        u, c = ct.c_int64(), ct.c_int64()
        _check(lib().mmi_plan_pair_counts(self.h, head, ct.byref(u), ct.byref(c)))
        return u.value, c.value

    def check(self):
        """Consistency check of the plan's tables on the host (raises MMIError)."""
        _check(lib().mmi_plan_check(self.h))

    def destroy(self):
        if self.h:
            _check(lib().mmi_plan_destroy(self.h))
            self.h = None

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass


def mmi_plan_create(ctx, prob, heads, q, k, stream=None) -> Plan:
    return Plan(ctx, prob, heads, q, k, stream)


def mmi_plan_execute(plan: Plan, q, k, v, o, lse=None, stream=None):
    plan.execute(q, k, v, o, lse, stream)


def mmi_plan_stats(plan: Plan, head: int):
    return plan.stats(head)


def mmi_plan_export(plan: Plan, head: int, what: str, slot: int = 0):
    return plan.export(head, what, slot)


def mmi_plan_timing_get(plan: Plan) -> dict:
    return plan.timing()


def mmi_plan_destroy(plan: Plan):
    plan.destroy()


def mmi_attention(ctx, prob, heads, q, k, v, o, lse=None, stream=None):
    cfgs = head_cfgs(heads)
    _check(lib().mmi_attention(ctx.h, ct.byref(prob.c), cfgs, _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse),
                               _stream(stream)))


def mmi_attention_noalloc(ctx, prob, heads, q, k, v, o, lse=None, stream=None):
    cfgs = head_cfgs(heads)
    _check(lib().mmi_attention_noalloc(ctx.h, ct.byref(prob.c), cfgs, _ptr(q), _ptr(k), _ptr(v), _ptr(o),
                                       _ptr(lse), _stream(stream)))


def mmi_dense_attention(ctx, prob, q, k, v, o, lse=None, stream=None):
    _check(lib().mmi_dense_attention(ctx.h, ct.byref(prob.c), _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse),
                                     _stream(stream)))


def mmi_permute_rows(src, dst, perm, stream=None):
    """dst[x] = src[perm[x]] row-wise (rows = first dim, contiguous rows)."""
    rb = src[0].numel() * src.element_size()
    _check(lib().mmi_permute_rows(_ptr(src), src.stride(0) * src.element_size(), _ptr(dst),
                                  dst.stride(0) * dst.element_size(), _ptr(perm), perm.numel(), rb,
                                  _stream(stream)))


def mmi_unpermute_rows(src, dst, perm, stream=None):
    """dst[perm[x]] = src[x] row-wise."""
    rb = src[0].numel() * src.element_size()
    _check(lib().mmi_unpermute_rows(_ptr(src), src.stride(0) * src.element_size(), _ptr(dst),
                                    dst.stride(0) * dst.element_size(), _ptr(perm), perm.numel(), rb,
                                    _stream(stream)))


def mmi_output_sqerr(prob, a, b, cls, n_class, out, stream=None):
    """out[h * n_class + c] (device float64) = squared difference of outputs a
    and b summed over the positions of class c."""
    _check(lib().mmi_output_sqerr(ct.byref(prob.c), _ptr(a), _ptr(b), _ptr(cls), int(n_class), _ptr(out),
                                  _stream(stream)))


def mmi_search(ctx, prob, q, k, v, cands, xc, target, stream=None):
    """Algorithm 4 for every head (the C call mmi_search). cands / xc: ops in
    table order; target: the FLOPs target op. Returns (the chosen
    mmi_head_cfg per head, the report's arrays as numpy arrays)."""
    Hq = prob.c.Hq
    nc, nx = len(cands), len(xc)
    ca = (mmi_op * max(nc, 1))(*[op_struct(o) for o in cands])
    xa = (mmi_op * max(nx, 1))(*[op_struct(o) for o in xc])
    tgt = op_struct(target)
    out = (mmi_head_cfg * Hq)()
    arrays = {"budget1": (np.int64, (Hq, MAXM)), "step1_cost": (np.int64, (Hq, nc, MAXM)),
              "step1_err": (np.float64, (Hq, nc, MAXM)), "intra": (np.int32, (Hq, MAXM)),
              "step2_cost": (np.int64, (Hq, MAXM - 1, nx, MAXM)), "step2_err": (np.float64, (Hq, MAXM - 1, nx, MAXM)),
              "cross": (np.int32, (Hq, MAXM, MAXM)), "budget3": (np.int64, (Hq,)),
              "step3g_cost": (np.int64, (Hq, nc)), "step3g_err": (np.float64, (Hq, nc)),
              "global_": (np.int32, (Hq,)), "step3_cost": (np.int64, (Hq, 3)), "step3_err": (np.float64, (Hq, 3)),
              "kind": (np.int32, (Hq,))}
    rep = mmi_search_report()
    got = {}
    for name, (dt, shape) in arrays.items():
        a = got[name] = np.zeros(shape, dt)
        ptype = {np.int64: I64P, np.int32: I32P, np.float64: F64P}[dt]
        setattr(rep, name, a.ctypes.data_as(ptype))
    _check(lib().mmi_search(ctx.h, ct.byref(prob.c), _ptr(q), _ptr(k), _ptr(v), ca, nc, xa, nx, ct.byref(tgt),
                            _stream(stream), out, ct.byref(rep)))
    got["n_mod"], got["mods"], got["plans"] = rep.n_mod, list(rep.mods)[:rep.n_mod], rep.plans
    return list(out), got


def _i32(a):
    """int32 C-contiguous copy (kept alive by the caller) and its pointer, or (None, None)."""
    if a is None:
        return None, None
    arr = np.ascontiguousarray(a, dtype=np.int32)
    return arr, arr.ctypes.data_as(I32P)


def mmi_check_index(S, n_qblocks, n_kblocks, row_ptr, col_idx, qperm=None, kperm=None, n_layouts=1, causal=True,
                    group_size=0, group_stride=1, union_ptr=None, union_ent=None):
    """Host consistency check of one head's block index (raises MMIError);
    union_ptr None skips the row-group checks."""
    keep = [_i32(x) for x in (qperm, kperm, row_ptr, col_idx, union_ptr, union_ent)]
    v = mmi_index_view(S=S, n_qblocks=n_qblocks, n_kblocks=n_kblocks, n_layouts=n_layouts, causal=int(causal),
                       qperm=keep[0][1], kperm=keep[1][1], row_ptr=keep[2][1], col_idx=keep[3][1],
                       group_size=group_size, group_stride=group_stride,
                       n_groups=0 if union_ptr is None else len(union_ptr) - 1,
                       union_ptr=keep[4][1], union_ent=keep[5][1])
    _check(lib().mmi_check_index(ct.byref(v)))


def mmi_check_work(union_ptrs, items, n_parts, splits, item_map):
    """Host consistency check of a work list: union_ptrs per head, items
    [n][5] (head, group, e0, e1, partial slot), splits [n][4], item_map [8][len]."""
    ups = [_i32(u) for u in union_ptrs]
    ng = np.array([len(u) - 1 for u in union_ptrs], dtype=np.int32)
    up_arr = (I32P * max(1, len(ups)))(*[p for _, p in ups])
    it, itp = _i32(np.asarray(items).reshape(-1))
    sp, spp = _i32(np.asarray(splits).reshape(-1))
    im = np.asarray(item_map)
    mp, mpp = _i32(im.reshape(-1))
    w = mmi_work_view(n_heads=len(ups), n_groups=ng.ctypes.data_as(I32P), union_ptr=up_arr,
                      n_items=len(it) // 5, items=itp, n_parts=n_parts, n_splits=len(sp) // 4, splits=spp,
                      map_len=im.shape[1] if im.ndim == 2 else 0, item_map=mpp)
    _check(lib().mmi_check_work(ct.byref(w)))


def mmi_plan_check(plan: Plan):
    plan.check()


def mmi_plan_pair_counts(plan: Plan, head: int):
    return plan.pair_counts(head)


@atexit.register
def _close_all():
    """Release plans and contexts before the HIP runtime shuts down."""
    for c in list(_live_ctx):
        try:
            c.close()
        except Exception:
            pass
