"""Parity driver: run the HIP path through the C-ABI, export what it chose and
computed, and compare every checked head with the oracle (test
infrastructure). The per-head comparison and its five layers are in
parity_core.py; this module holds the GPU side and the fan-out of heads over
worker processes for the full-size workloads.
"""
from __future__ import annotations

import multiprocessing as mp
import os
import shutil
import sys
import tempfile
import time
from concurrent.futures import ProcessPoolExecutor
from dataclasses import dataclass, field

import numpy as np
import torch

import parity_core as PC
from oracle import layout as OL
from oracle import numerics as ON
from synth import config as C

O_TOL, LSE_TOL, SCORE_RTOL, TIE_RTOL = PC.O_TOL, PC.LSE_TOL, PC.SCORE_RTOL, PC.TIE_RTOL
ROWS_PER_HEAD = 4096


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@dataclass
class Report:
    ties: list = field(default_factory=list)
    heads: list = field(default_factory=list)
    max_o: float = 0.0
    max_o_excess: float = 0.0
    max_lse: float = 0.0
    score_err: float = 0.0
    rows: int = 0
    nnz: dict = field(default_factory=dict)

    def add(self, r):
        self.heads.append(r["head"])
        self.ties += [(r["head"],) + tuple(t) for t in r["ties"]]
        self.max_o = max(self.max_o, r["max_o"])
        self.max_o_excess = max(self.max_o_excess, r["max_o_excess"])
        self.max_lse = max(self.max_lse, r["max_lse"])
        self.score_err = max(self.score_err, r["score_err"])
        self.rows += r["rows"]
        self.nnz[r["head"]] = r["nnz"]

    def line(self):
        return (f"heads={len(self.heads)} rows={self.rows} ties={self.ties} score_err={self.score_err:.2e} "
                f"max|dO|={self.max_o:.3g} (excess {self.max_o_excess:.3g}) lse={self.max_lse:.3g}")


def run_gpu(ctx, S, Hq, Hkv, modality, heads, q, k, v):
    from paper_2504_16083_amd import mmi
    prob = mmi.Problem(S, Hq, Hkv, modality)
    o = torch.empty_like(q)
    lse = torch.full((Hq, S), float("nan"), device=q.device, dtype=torch.float32)
    plan = mmi.Plan(ctx, prob, heads, q, k)
    plan.execute(q, k, v, o, lse)
    torch.cuda.synchronize()
    return plan, o, lse


def export_head(plan, h, cfg, S, modality):
    """Everything the comparison needs from the library for one head."""
    gpu = dict(qperm=plan.export(h, "qperm"), kperm=plan.export(h, "kperm"),
               row_ptr=plan.export(h, "row_ptr"), col_idx=plan.export(h, "col_idx"), slots={})
    for key, op in PC.op_keys(cfg, S, modality):
        s = PC.slot_of(key)
        d = dict(params=plan.export(h, "params", s), v=plan.export(h, "v", s), est_lse=plan.export(h, "est_lse", s))
        if op.kind == C.OP_GRID:
            d["fold"] = plan.export(h, "fold", s)
        else:
            d["vsel"] = plan.export(h, "vsel", s)
        if op.kind == C.OP_VSLASH:
            d["u"] = plan.export(h, "u", s)
            d["ssel"] = plan.export(h, "ssel", s)
        gpu["slots"][key] = d
    return gpu


def full_check(ctx, S, Hq, Hkv, modality, heads, q, k, v, rows=None, heads_to_check=None):
    """GPU run + layered comparison of every head (or heads_to_check) in this
    process, on all rows or the given rows. q/k/v: CUDA bf16 tensors."""
    plan, o, lse = run_gpu(ctx, S, Hq, Hkv, modality, heads, q, k, v)
    Q, K, V = (ON.torch_bf16_to_f64(t) for t in (q, k, v))
    O = ON.torch_bf16_to_f64(o)
    LSE = lse.cpu().double().numpy()
    G = Hq // Hkv
    rr = np.arange(S) if rows is None else np.asarray(rows, dtype=np.int64)
    rep = Report()
    try:
        for h in (heads_to_check if heads_to_check is not None else range(Hq)):
            gpu = export_head(plan, h, heads[h], S, modality)
            r = PC.check_head(h, heads[h], S, modality, lambda x, h=h: Q[x, h], K[:, h // G], V[:, h // G], gpu,
                              rr, O[rr, h], LSE[h, rr])
            rep.add(r)
    finally:
        plan.destroy()
    return rep


def _workers():
    """Oracle worker processes: the host's cores, at most 12 (a one-GPU host
    share holds about 16 cores; this process keeps the GPU)."""
    n = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    return max(1, min(12, n))


def _scratch_dir():
    for base in ("/dev/shm", tempfile.gettempdir()):
        try:
            st = os.statvfs(base)
            if st.f_bavail * st.f_frsize > (8 << 30):
                return tempfile.mkdtemp(prefix="mmi_parity_", dir=base)
        except OSError:
            continue
    return tempfile.mkdtemp(prefix="mmi_parity_")


def _bits(t):
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def run_tasks(tasks, workers=None, t0=None):
    """parity_core.run_task over the tasks, in fresh oracle worker processes
    (spawn: they import numpy and the oracle only, never the GPU), with one
    BLAS thread each. Returns the merged Report."""
    t0 = time.time() if t0 is None else t0
    rep = Report()
    nw = workers or _workers()
    if nw <= 1 or len(tasks) <= 1:
        for t in tasks:
            rep.add(PC.run_task(t))
        return rep
    env_old = {x: os.environ.get(x) for x in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS")}
    for x in env_old:
        os.environ[x] = "1"
    try:
        with ProcessPoolExecutor(max_workers=min(nw, len(tasks)), mp_context=mp.get_context("spawn")) as ex:
            for r in ex.map(PC.run_task, tasks):
                rep.add(r)
                say(f"  [parity] head {r['head']}: nnz {r['nnz']} ties {r['ties']} "
                    f"|dO| {r['max_o']:.3g} score {r['score_err']:.2e} ({time.time() - t0:.0f} s)")
    finally:
        for x, val in env_old.items():
            if val is None:
                os.environ.pop(x, None)
            else:
                os.environ[x] = val
    return rep


def sampled_check(ctx, wl, q, k, v, heads_to_check, n_rows=ROWS_PER_HEAD, seed=0, workers=None,
                  max_hline_blocks=None):
    """Full-size parity: the GPU plan of the whole layer, then for every head
    in heads_to_check all five layers (scores, choices re-derived, block index
    bit-exact, choices against the oracle with ties re-checked under the
    GPU's choice, O/LSE) on n_rows stratified rows per head. Heads are
    spread over oracle worker processes, started fresh (spawn): they import
    numpy and the oracle only and never touch the GPU; K and V reach them
    through bf16 bit files, each head's query and output rows through the
    task itself."""
    S, Hq, Hkv = wl.S, wl.Hq, wl.Hkv
    G = Hq // Hkv
    t0 = time.time()
    plan, o, lse = run_gpu(ctx, S, Hq, Hkv, wl.modality, wl.heads, q, k, v)
    tmp = _scratch_dir()
    tasks = []
    try:
        path_k, path_v = os.path.join(tmp, "k.npy"), os.path.join(tmp, "v.npy")
        np.save(path_k, _bits(k.transpose(0, 1)))
        np.save(path_v, _bits(v.transpose(0, 1)))
        mod = OL.modality_array(S, wl.modality)
        T = OL.positions_of(mod)
        est_rows = {"g": OL.global_rows(S)}
        est_rows.update({m: OL.final_run_rows(T[m]) for m in T})
        for h in heads_to_check:
            cfg = wl.heads[h]
            gpu = export_head(plan, h, cfg, S, wl.modality)
            rows = PC.sample_rows(S, wl.modality, cfg, gpu, n_target=n_rows, seed=seed * 1000 + h,
                                  max_hline_blocks=max_hline_blocks)
            qpos = np.union1d(rows, np.concatenate(list(est_rows.values())))
            dev = torch.as_tensor(qpos, device=q.device)
            drow = torch.as_tensor(rows, device=q.device)
            tasks.append(dict(h=h, g=h // G, cfg=cfg, S=S, modality=wl.modality, gpu=gpu, q_pos=qpos,
                              q_bits=_bits(q[dev, h]), rows=rows, o_bits=_bits(o[drow, h]),
                              lse=lse[h, drow].cpu().double().numpy(), path_k=path_k, path_v=path_v))
        plan.destroy()
        plan = None
        tasks.sort(key=lambda t: t["g"])
        say(f"  [parity] GPU plan, exports and row gathers: {time.time() - t0:.1f} s, {len(tasks)} heads")
        return run_tasks(tasks, workers, t0)
    finally:
        if plan is not None:
            plan.destroy()
        shutil.rmtree(tmp, ignore_errors=True)
