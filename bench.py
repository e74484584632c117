"""Prefill sparse-attention benchmark on one MI355X.

One step = the whole hot path for one layer (all heads): estimation, choices,
permutations, block index, block-sparse attention and the output scatter
(mmi_plan_create + mmi_plan_execute + mmi_plan_destroy through the C-ABI),
on seeded synthetic inputs already resident in HBM, producing the attention
output O (with --lse also each row's log-sum-exp). Prints ONE JSON line.

Also measured in the same run:
  * dense baseline: every causal block through the same kernel
    (mmi_dense_attention), for the speedup over dense on this GPU;
  * roofline of the dominant kernel (block-sparse attention): algorithmic
    flops = computed blocks x 4*64*64*128, divided by the kernel's duration
    from HIP events recorded on the stream it runs on;
  * cpu_baseline: the CPU oracle timed on a bounded sample of the same
    workload on this host's cores, extrapolated to ms/layer;
  * with --sdpa, as context only: PyTorch's flash scaled-dot-product
    attention (dense causal, one call per KV group with GQA) on the same
    tensors.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
FLOP_PER_BLOCK = 4 * 64 * 64 * 128

# HBM traffic of one k_attention launch on the 1M workload, from two rocprofv3
# --pmc passes (FETCH_SIZE, then WRITE_SIZE, KiB per dispatch) scaled by what
# the same counters read for a plain 1 GiB copy (read x1.939, write x1.000).
# Keyed by the SHA-256 prefix of the sources that decide the launch's memory
# traffic (the kernel, the block index and work list, the runtime that orders
# them): once any of them changes the counters are stale and `traffic` is
# reported as null.
TRAFFIC_SOURCES = ("k_attention.hip", "k_blocks.hip", "runtime.hip")
TRAFFIC = {
    "b01aa7b3395f3a7b": {"workload": "cfg4_mm_1m", "fetch_kib": 542877060, "write_kib": 7698770,
                         "fetch_scale": 1.939, "write_scale": 1.000},
}


def pattern_head(pattern: str, tpf: int):
    """One head configuration for every head: the paper's baselines with the
    hyperparameters of its baseline table (tpf = tokens per frame), or
    Q-Boundary heads with A-shape text and Grid video."""
    from synth import config as C
    return {"ashape": C.global_head(C.ashape(128, 4096)),
            "trishape": C.global_head(C.trishape(128, 4096, 128)),
            "sf_fixed": C.global_head(C.sf_fixed(tpf, tpf)),
            "sf_strided": C.global_head(C.sf_strided(tpf, tpf)),
            "vslash": C.global_head(C.vslash(1000, 1024)),
            "grid": C.global_head(C.grid_window(tpf)),
            "qb_grid": C.qboundary_head({0: C.ashape(128, 4096), 1: C.grid_window(tpf)})}[pattern]


def traffic_key():
    import hashlib
    h = hashlib.sha256()
    for name in TRAFFIC_SOURCES:
        with open(os.path.join(ROOT, "paper_2504_16083_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def attention_traffic(workload: str):
    t = TRAFFIC.get(traffic_key())
    if t is None or t["workload"] != workload:
        return None
    return (t["fetch_kib"] * t["fetch_scale"] + t["write_kib"] * t["write_scale"]) * 1024.0


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", type=int, default=4, help="workload id 0-4 (4 = 1M tokens)")
    ap.add_argument("--workload", default="mm", choices=["mm", "natten", "search", "permute"],
                    help="mm: the multi-modal prefill workloads (--config); natten: neighborhood "
                         "attention over a video DiT token grid (Appendix F), bidirectional; search: "
                         "the modality-aware pattern search (Algorithm 4) on its calibration sample; "
                         "permute: the Q/K/V permutation and the inverse permutation of O as explicit "
                         "passes (mmi_permute_rows / mmi_unpermute_rows) for the workload's permuted "
                         "heads, the alternative to the attention kernel's fused gathers")
    ap.add_argument("--dense-reps", type=int, default=3, help="dense baseline runs (median reported)")
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--sdpa", action="store_true",
                    help="also time PyTorch's flash SDPA (dense causal) on the same inputs, as context")
    ap.add_argument("--cpu-blocks", type=int, default=4,
                    help="query blocks per sampled head whose rows the cpu_baseline oracle computes")
    ap.add_argument("--lse", action="store_true",
                    help="also ask for each row's log-sum-exp (the prefill layer itself needs only O)")
    ap.add_argument("--no-128k", action="store_true",
                    help="skip the 128K workload that the default 1M run also reports (metric_128k)")
    ap.add_argument("--pattern", default="method",
                    choices=["method", "ashape", "trishape", "sf_fixed", "sf_strided", "vslash", "grid", "qb_grid"],
                    help="every head on one pattern instead of the workload's per-head patterns: one of "
                         "the paper's baselines (Section 4.1, baseline hyperparameter table), grid (Grid "
                         "heads, strides within 8 of the frame size), or qb_grid (Q-Boundary heads, A-shape "
                         "text and Grid video)")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="run one plain copy of this many MiB (k_permute, identity) before the steps, "
                         "as the reference dispatch for HBM byte counters")
    return ap.parse_args()


def _scratch_dir():
    import tempfile
    for base in ("/dev/shm", tempfile.gettempdir()):
        try:
            st = os.statvfs(base)
            if st.f_bavail * st.f_frsize > (16 << 30):
                return tempfile.mkdtemp(prefix="mmi_bench_", dir=base)
        except OSError:
            continue
    return tempfile.mkdtemp(prefix="mmi_bench_")


def _oracle_head(t):
    """One head of the cpu_baseline sample, in a worker process (one BLAS
    thread): the oracle's full plan (estimation, choices, permutations, every
    block row), then every row of a few uniformly drawn permuted query
    blocks. Returns the CPU seconds of each part and the selected key blocks
    of the sampled query blocks and of the whole head."""
    import numpy as np

    from oracle import attention as OA
    from oracle import numerics as ON
    from oracle import plan as OP
    qb = np.load(t["path_q"], mmap_mode="r")[t["qi"]]
    K = ON.bf16_bits_to_f64(np.asarray(np.load(t["path_k"], mmap_mode="r")[t["kvi"]]))
    V = ON.bf16_bits_to_f64(np.asarray(np.load(t["path_v"], mmap_mode="r")[t["kvi"]]))

    def q_rows(r):
        return ON.bf16_bits_to_f64(np.asarray(qb[np.asarray(r, dtype=np.int64)]))

    c0 = time.process_time()
    hp = OP.plan_head(t["cfg"], t["S"], t["modality"], q_rows, K)
    c1 = time.process_time()
    rng = np.random.default_rng(t["seed"])
    live = [i for i in range(hp.nbq) if (hp.qperm[i * 64:(i + 1) * 64] >= 0).any()]
    pick = rng.choice(live, size=min(t["blocks"], len(live)), replace=False)
    rows = np.concatenate([hp.qperm[i * 64:(i + 1) * 64] for i in pick])
    rows = np.sort(rows[rows >= 0])
    c2 = time.process_time()
    OA.head_rows(hp, q_rows, K, V, rows)
    c3 = time.process_time()
    return dict(h=t["h"], plan_s=c1 - c0, rows_s=c3 - c2, rows=len(rows),
                nnz_sample=int(sum(len(hp.blocks[i]) for i in pick)), nnz=int(sum(len(b) for b in hp.blocks)))


def cpu_baseline(wl, q, k, v, blocks_per_head, max_workers=16):
    """The oracle (numpy fp64) on a bounded sample of the layer, timed on this
    host's cores: one worker process per sampled head (the first `cores`
    heads, every head kind among them), each running the full oracle plan of
    its head and every row of `blocks_per_head` random query blocks. Layer
    CPU time = sum over all heads of (plan time + row time per selected key
    block x selected key blocks), each head taking the mean of the sampled
    heads of its configuration; the value is that time spread over the
    workers (heads and rows are independent)."""
    import multiprocessing as mp
    import shutil
    from concurrent.futures import ProcessPoolExecutor

    import numpy as np
    import torch
    G = wl.Hq // wl.Hkv
    n = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    cores = max(1, min(max_workers, n, wl.Hq))
    heads = list(range(cores))
    kvs = sorted({h // G for h in heads})
    t0 = time.perf_counter()
    tmp = _scratch_dir()
    try:
        bits = lambda x: x.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
        paths = {nm: os.path.join(tmp, nm + ".npy") for nm in ("q", "k", "v")}
        np.save(paths["q"], bits(q[:, heads].transpose(0, 1)))
        np.save(paths["k"], bits(k[:, kvs].transpose(0, 1)))
        np.save(paths["v"], bits(v[:, kvs].transpose(0, 1)))
        tasks = [dict(h=h, qi=i, kvi=kvs.index(h // G), cfg=wl.heads[h], S=wl.S, modality=wl.modality,
                      blocks=blocks_per_head, seed=h, path_q=paths["q"], path_k=paths["k"], path_v=paths["v"])
                 for i, h in enumerate(heads)]
        env_old = {x: os.environ.get(x) for x in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS")}
        for x in env_old:
            os.environ[x] = "1"
        try:
            with ProcessPoolExecutor(max_workers=cores, mp_context=mp.get_context("spawn")) as ex:
                res = list(ex.map(_oracle_head, tasks))
        finally:
            for x, val in env_old.items():
                if val is None:
                    os.environ.pop(x, None)
                else:
                    os.environ[x] = val
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
    wall = time.perf_counter() - t0

    def kind(h):
        c = wl.heads[h]
        return (c.kind, c.op, tuple(sorted(c.intra.items())), tuple(sorted(c.cross.items())))
    by_kind = {}
    for r in res:
        by_kind.setdefault(kind(r["h"]), []).append(r)
    layer_s = 0.0
    for h in range(wl.Hq):
        rs = by_kind[kind(h)]
        layer_s += np.mean([r["plan_s"] + r["rows_s"] / max(r["nnz_sample"], 1) * r["nnz"] for r in rs])
    sample_cpu = sum(r["plan_s"] + r["rows_s"] for r in res)
    return {"value": layer_s / cores * 1e3, "unit": "ms/layer", "cores": cores, "kind": "oracle",
            "sample": (f"heads 0-{cores - 1} (every head configuration of the layer), one worker process "
                       f"each: full oracle plan + all rows of {blocks_per_head} random query blocks "
                       f"({sum(r['rows'] for r in res)} rows); {sample_cpu:.1f} CPU s in {wall:.1f} s "
                       f"wall incl. input staging; layer = sum over heads of plan time + row time per "
                       f"selected key block x selected key blocks, spread over the {cores} cores"),
            "cpu_s_per_layer": layer_s}


def sdpa_context(wl, q, k, v, sparse_ms):
    """PyTorch's flash SDPA, dense causal, on the same tensors: one call per
    KV group (its G query heads against one K/V head, GQA), inputs copied to
    [1, H, S, D] before timing. The math fallback is disabled (at these
    lengths it would build the S x S matrix); if flash is unavailable the
    result says so. Reported as context, not as a baseline of this method."""
    import torch
    import torch.nn.functional as F
    from torch.nn.attention import SDPBackend, sdpa_kernel
    G = wl.Hq // wl.Hkv
    groups = []
    for g in range(wl.Hkv):
        groups.append((q[:, g * G:(g + 1) * G].permute(1, 0, 2).contiguous().unsqueeze(0),
                       k[:, g].contiguous()[None, None], v[:, g].contiguous()[None, None]))
    torch.cuda.synchronize()

    def run():
        with sdpa_kernel([SDPBackend.FLASH_ATTENTION]):
            return [F.scaled_dot_product_attention(a, b, c, is_causal=True, enable_gqa=True)
                    for a, b, c in groups]
    try:
        run()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        run()
        e1.record()
        torch.cuda.synchronize()
    except RuntimeError as err:
        return {"backend": "torch flash SDPA", "error": str(err)[:200]}
    t = e0.elapsed_time(e1)
    useful = 4.0 * 128 * wl.Hq * wl.S * (wl.S + 1) / 2      # causal q.k pairs only
    return {"backend": f"torch {torch.__version__} flash SDPA, per KV group", "ms": t,
            "tflops_causal_pairs": useful / (t * 1e-3) / 1e12, "sparse_speedup": t / sparse_ms}


def search_main(args):
    """Algorithm 4 on its calibration sample, all heads, the paper's search
    space; one step = one whole search. cpu_baseline: the oracle scoring a
    bounded sample of the same candidate plans for one head, extrapolated."""
    import numpy as np
    import torch

    from paper_2504_16083_amd import mmi
    from paper_2504_16083_amd import search as GS
    from synth import config as C
    from synth import generate, workloads
    from synth import search_space as SP

    wl = workloads.search_calibration()
    torch.cuda.set_device(0)
    q, k, v = generate.make_qkv(wl, "cuda")
    cands, xc, target = SP.intra_candidates(wl.frame), SP.cross_candidates(), SP.budget_op()
    ctx = mmi.Ctx(0)
    for _ in range(args.warmup):
        GS.search(ctx, wl.S, wl.Hq, wl.Hkv, wl.modality, q, k, v, cands, xc, target)
        log("warmup search done")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        heads, reps, nplans = GS.search(ctx, wl.S, wl.Hq, wl.Hkv, wl.modality, q, k, v, cands, xc, target)
        log(f"search done: {nplans} plans")
    torch.cuda.synchronize()
    sec = (time.perf_counter() - t0) / args.steps
    kinds = {}
    for r in reps:
        key = r.kind + ":" + (r.global_op[0] if r.kind == "global" else
                              ",".join(f"{m}={r.intra[m][0]}" for m in sorted(r.intra)))
        kinds[key] = kinds.get(key, 0) + 1
    cpu = None
    if not args.no_cpu:
        from oracle import attention as OA
        from oracle import numerics as ON
        from oracle import plan as OP
        Q, K, V = (ON.torch_bf16_to_f64(t[:, 0]) for t in (q, k, v))
        t1 = time.perf_counter()
        n = 3
        for name, op in cands[:n]:
            hp = OP.plan_head(C.global_head(op), wl.S, wl.modality, lambda r: Q[r], K)
            O, _ = OA.permuted_blockwise(hp, Q, K, V)
        per = (time.perf_counter() - t1) / n
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
        cpu = {"value": per * nplans * wl.Hq, "unit": "s/search", "cores": threads, "kind": "oracle",
               "sample": f"oracle plan + blockwise attention of {n} global candidates for head 0 "
                         f"({per:.1f} s each), extrapolated x {nplans} plans x {wl.Hq} heads"}
    out = {"metric": "pattern search seconds (Algorithm 4, all heads, one calibration sample)",
           "value": sec, "unit": "s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
           "ms_per_step": sec * 1e3, "higher_is_better": False, "scaling": "weak", "vs_baseline": None,
           "dtype": "bf16", "data": "synthetic (seeded Q/K/V with planted grid/text structure)",
           "config": {"workload": wl.name, "S": wl.S, "Hq": wl.Hq, "Hkv": wl.Hkv, "head_dim": 128,
                      "candidates": len(cands), "cross_candidates": len(xc), "plans": nplans},
           "chosen": kinds, "cpu_baseline": cpu}
    print(json.dumps(out), flush=True)
    ctx.close()


def permute_main(args):
    """The permutation steps of the hot path done as separate passes: for
    every head whose plan permutes queries or keys, gather its Q rows by
    qperm and its K and V rows by kperm into slot order, and scatter an
    output in slot order back to token order by qperm (what the attention
    kernel otherwise does inside its loads and its epilogue). Bytes = rows
    read + rows written (256 B each); reported against the 8 TB/s HBM peak."""
    import numpy as np
    import torch

    from paper_2504_16083_amd import mmi
    from synth import generate, workloads
    wl = workloads.by_id(args.config)
    torch.cuda.set_device(0)
    q, k, v = generate.make_qkv(wl, "cuda")
    ctx = mmi.Ctx(0)
    stream = torch.cuda.current_stream()
    plan = mmi.Plan(ctx, mmi.Problem(wl.S, wl.Hq, wl.Hkv, wl.modality), wl.heads, q, k, stream)
    G = wl.Hq // wl.Hkv
    jobs = []
    for h in range(wl.Hq):
        qp, kp = plan.export(h, "qperm"), plan.export(h, "kperm")
        ident = len(qp) >= wl.S and np.array_equal(qp[:wl.S], np.arange(wl.S)) and (qp[wl.S:] < 0).all() \
            and len(kp) == len(qp) and np.array_equal(kp, qp)
        if not ident:
            jobs.append((h, torch.as_tensor(qp, device="cuda"), torch.as_tensor(kp, device="cuda")))
    plan.destroy()
    nq = max(len(j[1]) for j in jobs)
    nk = max(len(j[2]) for j in jobs)
    qs = torch.empty(nq, 128, dtype=q.dtype, device="cuda")
    ks = torch.empty(nk, 128, dtype=q.dtype, device="cuda")
    vs = torch.empty(nk, 128, dtype=q.dtype, device="cuda")
    o = torch.empty_like(q)

    def step():
        for h, qp, kp in jobs:
            mmi.mmi_permute_rows(q[:, h], qs[:len(qp)], qp, stream)
            mmi.mmi_permute_rows(k[:, h // G], ks[:len(kp)], kp, stream)
            mmi.mmi_permute_rows(v[:, h // G], vs[:len(kp)], kp, stream)
            mmi.mmi_unpermute_rows(qs[:len(qp)], o[:, h], qp, stream)   # slot-order rows back to tokens

    row = 256

    def moved(qp, kp):        # rows read + rows written (a -1 slot writes zeros, reads nothing)
        lq, lk = int((qp >= 0).sum().item()), int((kp >= 0).sum().item())
        return (lq + len(qp)) + 2 * (lk + len(kp)) + 2 * lq
    nbytes = row * sum(moved(qp, kp) for _, qp, kp in jobs)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    gbs = nbytes / (ms * 1e-3) / 1e9
    out = {"metric": "explicit permutation passes ms/layer (Q, K, V gathers and O scatter of the permuted heads)",
           "value": ms, "unit": "ms/layer", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
           "ms_per_step": ms, "higher_is_better": False, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
           "data": "synthetic (seeded Q/K/V with planted grid/text/sink structure)",
           "config": {"workload": wl.name, "S": wl.S, "Hq": wl.Hq, "Hkv": wl.Hkv, "permuted_heads": len(jobs)},
           "roofline": {"bound": "hbm", "kernel": "k_permute", "achieved": gbs, "peak": 8000.0, "unit": "GB/s",
                        "frac": gbs / 8000.0, "traffic": None, "bytes_per_step": nbytes},
           "cpu_baseline": None}
    print(json.dumps(out), flush=True)
    ctx.close()


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this library and benchmark run on exactly one GPU; multi-GPU sharding "
                                   "is a design note only (heads shard with no exchange)", "n_gpus": args.gpus}))
        sys.exit(2)
    if args.workload == "search":
        search_main(args)
        return
    if args.workload == "permute":
        permute_main(args)
        return
    import torch

    from paper_2504_16083_amd import mmi
    from synth import workloads

    wl = workloads.natten_video() if args.workload == "natten" else workloads.by_id(args.config)
    if args.pattern != "method":
        wl.heads = [pattern_head(args.pattern, wl.frame or 256)] * wl.Hq
        wl.name = f"{wl.name}+{args.pattern}"
    torch.cuda.set_device(0)
    ctx = mmi.Ctx(0)
    stream = torch.cuda.current_stream()
    if args.calib_copy_mib > 0:
        rows = args.calib_copy_mib * 1024 * 1024 // 256
        src = torch.empty(rows, 128, device="cuda", dtype=torch.bfloat16).fill_(1.0)
        dst = torch.empty_like(src)
        ident = torch.arange(rows, device="cuda", dtype=torch.int32)
        mmi.mmi_permute_rows(src, dst, ident, stream)
        torch.cuda.synchronize()
        log(f"calibration copy: {rows * 256} bytes read and written")
        del src, dst, ident

    res, q, k, v = measure(wl, args, ctx, stream, sdpa=args.sdpa and args.workload == "mm")
    cpu = None
    if not args.no_cpu:
        log("cpu baseline")
        cpu = cpu_baseline(wl, q, k, v, args.cpu_blocks)
        log(f"cpu baseline done: {cpu['sample']}")
    del q, k, v
    extra = {}
    if args.workload == "mm" and args.pattern == "method" and args.config == 4 and not args.no_128k:
        # the metric's other size: the 128K mixed-modality workload, same steps
        torch.cuda.empty_cache()
        r2, *_ = measure(workloads.by_id(2), args, ctx, stream, sdpa=False)
        extra["metric_128k"] = {"workload": r2["workload"], "ms_per_layer": r2["ms"],
                                "stages_ms": r2["stages_ms"], "blocks": r2["blocks"],
                                "roofline": {"achieved": r2["tflops"], "frac": r2["tflops"] / PEAK_BF16_TFLOPS,
                                             "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s"},
                                "dense": r2["dense"],
                                "speedup_vs_dense": None if r2["dense"] is None
                                else r2["dense"]["speedup_sparse_vs_dense"]}
    out = {
        "metric": ("neighborhood attention ms/layer (bidirectional, all heads, index + attention)"
                   if args.workload == "natten" else
                   "prefill attention ms/layer (sparse, all heads, estimation + index + attention)"),
        "value": res["ms"], "unit": "ms/layer", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": res["ms"], "higher_is_better": False, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16",
        "data": ("synthetic (seeded N(0,1) Q/K/V)" if args.workload == "natten"
                 else "synthetic (seeded Q/K/V with planted grid/text/sink structure)"),
        "config": {"workload": wl.name, "S": wl.S, "Hq": wl.Hq, "Hkv": wl.Hkv, "head_dim": 128,
                   "block": 64, "parallelism": "single GPU", "outputs": "O and LSE" if args.lse else "O",
                   **({k2: wl.extra[k2] for k2 in ("grid", "win", "tile")} if args.workload == "natten" else {})},
        "stages_ms": res["stages_ms"],
        "blocks": res["blocks"],
        "roofline": {"bound": "mfma", "kernel": "k_attention", "achieved": res["tflops"],
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": res["tflops"] / PEAK_BF16_TFLOPS,
                     "traffic": attention_traffic(wl.name)},
        "dense": res["dense"],
        "speedup_vs_dense": None if res["dense"] is None else res["dense"]["speedup_sparse_vs_dense"],
        **({"sdpa_context": res["sdpa"]} if res["sdpa"] is not None else {}),
        **extra,
        "cpu_baseline": cpu,
        "wall_s": res["wall"],
    }
    print(json.dumps(out), flush=True)
    ctx.close()


def measure(wl, args, ctx, stream, sdpa=False):
    """K timed steps of the whole layer (after W warmup steps) on one
    workload, with the attention kernel's HIP-event time of each step; then
    the dense baseline (median of --dense-reps runs) and, if asked, SDPA."""
    import numpy as np
    import torch

    from paper_2504_16083_amd import mmi
    from synth import config as C
    from synth import generate
    log(f"workload {wl.name}: S={wl.S} Hq={wl.Hq} Hkv={wl.Hkv}")
    q, k, v = generate.make_qkv(wl, "cuda")
    torch.cuda.synchronize()
    log("inputs generated")
    o = torch.empty_like(q)
    lse = torch.empty(wl.Hq, wl.S, device="cuda", dtype=torch.float32) if args.lse else None
    prob = mmi.Problem(wl.S, wl.Hq, wl.Hkv, wl.modality)

    def step():
        plan = mmi.Plan(ctx, prob, wl.heads, q, k, stream)
        plan.execute(q, k, v, o, lse, stream)
        t = plan.timing()
        plan.destroy()
        return t

    for _ in range(args.warmup):
        step()
        log("warmup step done")
    torch.cuda.synchronize()
    timings = []
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    wall0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        timings.append(step())
        log(f"step done: {timings[-1]}")
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms = ev0.elapsed_time(ev1) / args.steps
    avg = {key: float(np.mean([t[key] for t in timings])) for key in timings[0]}
    blocks = int(timings[-1]["computed_blocks"])
    loaded = int(timings[-1]["loaded_blocks"])
    attn_tflops = blocks * FLOP_PER_BLOCK / (avg["attn_ms"] * 1e-3) / 1e12
    nb = (wl.S + 63) // 64
    causal_blocks = nb * (nb + 1) // 2 * wl.Hq
    dense_heads = [C.global_head(C.dense())] * wl.Hq
    natten = wl.heads[0].op.kind == C.OP_NATTEN
    if natten:
        # bidirectional baseline: the same op with windows as large as the grid
        # allows (odd), which selects every (query tile, key tile) pair
        g, t = wl.extra["grid"], wl.extra["tile"]
        full = C.natten(g, tuple(n if n % 2 else n - 1 for n in g), t)
        dense_heads = [C.global_head(full)] * wl.Hq
        ntiles = 1
        for n, x in zip(g, t):
            ntiles *= -(-n // x)
        causal_blocks = ntiles * ntiles * wl.Hq

    # causal-useful share of the computed pairs (outside the timed region)
    plan = mmi.Plan(ctx, prob, wl.heads, q, k, stream)
    useful = computed_pairs = 0
    for h in range(wl.Hq):
        u, c = plan.pair_counts(h)
        useful += u
        computed_pairs += c
    plan.destroy()
    log(f"pairs: {useful} of {computed_pairs} computed are used")

    dense = None
    if not args.no_dense:
        dense_ms = []
        for _ in range(args.dense_reps):
            plan = mmi.Plan(ctx, prob, dense_heads, q, k, stream)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            plan.execute(q, k, v, o, lse, stream)
            e1.record(stream)
            plan.destroy()
            torch.cuda.synchronize()
            dense_ms.append(e0.elapsed_time(e1))
            log(f"dense done: {dense_ms[-1]:.2f} ms")
        dms = float(np.median(dense_ms))
        dense = {"ms_attention": dms, "runs_ms": dense_ms, "blocks": causal_blocks,
                 "tflops": causal_blocks * FLOP_PER_BLOCK / (dms * 1e-3) / 1e12,
                 "speedup_sparse_vs_dense": dms / ms}
    sd = None
    if sdpa:
        sd = sdpa_context(wl, q, k, v, ms)
        log(f"sdpa done: {sd}")
    del o, lse
    return (dict(workload=wl.name, lse=bool(args.lse), ms=ms, wall=wall, tflops=attn_tflops, dense=dense, sdpa=sd,
                 stages_ms={k2: avg[k2] for k2 in ("est_ms", "select_ms", "index_ms", "attn_ms", "combine_ms")},
                 blocks={"computed": blocks, "loaded": loaded,
                         ("all_pairs" if natten else "causal"): causal_blocks,
                         "density": blocks / causal_blocks, "computed_per_load": blocks / max(loaded, 1),
                         "useful_pair_fraction": useful / max(computed_pairs, 1)}),
            q, k, v)


if __name__ == "__main__":
    main()
