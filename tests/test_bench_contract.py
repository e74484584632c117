"""bench.py's command-line contract that needs no GPU: more than one GPU is
refused with one JSON line and exit status 2, and the traffic table is keyed
by a kernel-source hash in the form bench.py computes."""
import json
import os
import re
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    lines = [l for l in r.stdout.splitlines() if l.strip()]
    assert len(lines) == 1
    out = json.loads(lines[0])
    assert out["n_gpus"] == 2 and "one GPU" in out["error"]


def test_traffic_table_entries_are_well_formed():
    sys.path.insert(0, ROOT)
    import bench
    for key, t in bench.TRAFFIC.items():
        assert re.fullmatch(r"[0-9a-f]{16}", key)
        assert t["fetch_kib"] > 0 and t["write_kib"] > 0 and t["fetch_scale"] > 0 and t["write_scale"] > 0
    v = bench.attention_traffic("cfg4_mm_1m")
    assert v is None or v > 0


def test_cpu_baseline_sample_and_extrapolation():
    """The cpu_baseline leg on the 4096-token workload (CPU tensors): one
    worker per sampled head, every head configuration sampled, a positive
    extrapolated layer time spread over the workers it used."""
    sys.path.insert(0, ROOT)
    import bench
    from synth import generate, workloads
    wl = workloads.config0()
    q, k, v = generate.make_qkv(wl, "cpu")
    r = bench.cpu_baseline(wl, q, k, v, blocks_per_head=2, max_workers=2)
    assert r["kind"] == "oracle" and r["unit"] == "ms/layer" and r["cores"] == 2
    assert r["value"] > 0 and abs(r["value"] - r["cpu_s_per_layer"] / 2 * 1e3) < 1e-6
    assert "(256 rows)" in r["sample"]          # 2 heads x 2 blocks x 64 rows
