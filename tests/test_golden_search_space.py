"""The paper's printed search space (Appendix C.5) maps onto the op schema."""
import json
import os

from synth import config as C

HERE = os.path.dirname(__file__)


def test_search_space_table_maps_to_ops():
    t = json.load(open(os.path.join(HERE, "golden", "search_space.json")))
    assert len(t["grid"]) == 12 and len(t["ashape"]) == 3 and len(t["vslash"]) == 9
    for mode, h, v, s, mx in t["grid"]:
        assert mx == C.MAX_STRIDE
        op = C.grid_frame(256, h, v, s) if mode == "frame_stride" else C.grid_window(256, 8, h, v, s)
        assert op.kind == C.OP_GRID and (op.use_h, op.use_v, op.use_s) == (h, v, s)
        assert 1 <= op.stride_lo <= op.stride_hi <= mx
    for sink, local in t["ashape"]:
        op = C.ashape(sink, local)
        assert (op.sink, op.local) == (sink, local)
    for nv, ns in t["vslash"]:
        op = C.vslash(nv, ns)
        assert (op.n_vertical, op.n_slash) == (nv, ns)
    assert t["last_q"]["value"] == C.LAST_Q


def test_workload_layouts_match_sequence_length():
    from synth import workloads
    for cid in range(5):
        wl = workloads.by_id(cid)
        assert len(wl.modality) == wl.S and wl.Hq % wl.Hkv == 0 and len(wl.heads) == wl.Hq


def test_bench_baselines_follow_the_printed_table():
    """bench.py --pattern uses the baseline hyperparameters the paper prints
    (Appendix, Table 'impl_details'); MInference takes its smallest sizes."""
    import bench
    t = json.load(open(os.path.join(HERE, "golden", "baselines.json")))
    tpf = 196
    op = bench.pattern_head("ashape", tpf).op
    assert (op.sink, op.local) == (t["ashape"]["sink"], t["ashape"]["local"])
    op = bench.pattern_head("trishape", tpf).op
    assert (op.sink, op.local, op.bottom) == (t["trishape"]["sink"], t["trishape"]["local"], t["trishape"]["bottom"])
    for name in ("sf_fixed", "sf_strided"):
        op = bench.pattern_head(name, tpf).op
        assert t[name] == {"local": "token_per_frame", "vline_stride": "token_per_frame"}
        assert (op.local, op.stride_lo) == (tpf, tpf)
    op = bench.pattern_head("vslash", tpf).op
    assert (op.n_vertical, op.n_slash) == (min(t["minference"]["vertical_size"]), min(t["minference"]["slash_size"]))
