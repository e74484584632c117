"""The five synthetic workloads (layout, per-head configs, planted structure).

Each is one attention layer, batch 1, head_dim 128, bf16, causal, block 64.
Layouts follow the paper's inputs: frames of 252/255/196/256 tokens, text
segments between frames, up to 1M tokens (Section 4.1; Appendix D).
Random choices (stride jitter, segment lengths, head patterns, line slots)
come from numpy's PCG64 seeded with 20250416 + config id; tensors are drawn
by generate.make_qkv with the same seed.
"""
from __future__ import annotations

import numpy as np

from . import config as C
from .generate import Structure, Workload

SEED0 = 20250416


def _rng(cid):
    return np.random.default_rng(SEED0 + cid)


def _layout(segments):
    """[(modality, length), ...] -> uint8 modality array."""
    return np.concatenate([np.full(n, m, dtype=np.uint8) for m, n in segments])


def _line_slots(rng, sigmas):
    return [int(rng.integers(0, s)) for s in sigmas]


def config0() -> Workload:
    """4096 = 64 text + 16 frames x 252; 2 query heads / 1 KV head; Grid(frame 252);
    the slot embedding on Q, K and V."""
    rng = _rng(0)
    mod = _layout([(0, 64), (1, 16 * 252)])
    st = Structure(sigma=[252], amp=2.0, v_embed=True)
    st.line_slot = _line_slots(rng, st.sigma)
    heads = [C.global_head(C.grid_frame(252)) for _ in range(2)]
    return Workload("cfg0_grid_4k", 4096, 2, 1, mod, heads, st, SEED0 + 0, frame=252)


def config1() -> Workload:
    """32768 = 128 text + 128 frames x 255; 28/4; stride 255+U{-4..4} per KV group;
    per-head pattern drawn from {Grid(window), A-shape(128,1024), VS(1000,1024)};
    the slot embedding on Q, K and V."""
    rng = _rng(1)
    mod = _layout([(0, 128), (1, 128 * 255)])
    sig = [255 + int(rng.integers(-4, 5)) for _ in range(4)]
    st = Structure(sigma=sig, amp=2.0, v_embed=True)
    st.line_slot = _line_slots(rng, sig)
    choices = [C.grid_window(255), C.ashape(128, 1024), C.vslash(1000, 1024)]
    heads = [C.global_head(choices[int(rng.integers(0, 3))]) for _ in range(28)]
    return Workload("cfg1_mixed_32k", 32768, 28, 4, mod, heads, st, SEED0 + 1, frame=255)


def qb_head(frame):
    return C.qboundary_head({0: C.ashape(128, 1024), 1: C.vslash(1000, 1024)})


def b2d_head(frame):
    return C.boundary2d_head({0: C.ashape(128, 1024), 1: C.grid_frame(frame)},
                             {(0, 1): C.vert(256), (1, 0): C.vert(256)})


def config2() -> Workload:
    """131072 tokens: T V T V T V T V, text U{512..4096}, video = whole 196-token frames."""
    rng = _rng(2)
    S, F = 131072, 196
    text = [int(rng.integers(512, 4097)) for _ in range(4)]
    vid_total = S - sum(text)
    nf = vid_total // F
    text[-1] += vid_total - nf * F
    cuts = np.sort(rng.choice(np.arange(1, nf), size=3, replace=False))
    frames = np.diff(np.concatenate([[0], cuts, [nf]])).tolist()
    segs = []
    for t, f in zip(text, frames):
        segs += [(0, t), (1, f * F)]
    mod = _layout(segs)
    assert len(mod) == S
    sig = [F] * 4
    st = Structure(sigma=sig, amp=2.0, text_amp=1.0)
    st.line_slot = _line_slots(rng, sig)
    kinds = [qb_head(F), b2d_head(F), C.global_head(C.grid_window(F)),
             C.global_head(C.vslash(1000, 1024))]
    heads = [kinds[h % 4] for h in range(28)]
    return Workload("cfg2_mm_128k", S, 28, 4, mod, heads, st, SEED0 + 2, frame=F,
                    extra={"text": text, "frames": frames})


def config3() -> Workload:
    """262144 = 256 text + 1023 frames x 256 (the stated "256 text + 1024 frames"
    is 256 tokens over 2^18; the frame count gives way); 32/8; amp 1.5; 1% sinks;
    per-head Grid / A-shape / Vertical-Slash at about 5% mean block density."""
    rng = _rng(3)
    mod = _layout([(0, 256), (1, 1023 * 256)])
    sig = [256] * 8
    st = Structure(sigma=sig, amp=1.5, sink_frac=0.01)
    st.line_slot = _line_slots(rng, sig)
    # op sizes set for a mean block density of about 5% over the 32 heads
    # (measured per head: Grid 1.2%, A-shape(128, 8192) 6.3%, VS(200, 64) ~5.6%)
    choices = [C.grid_window(256), C.ashape(128, 8192), C.vslash(200, 64)]
    heads = [C.global_head(choices[int(rng.integers(0, 3))]) for _ in range(32)]
    return Workload("cfg3_256k", 262144, 32, 8, mod, heads, st, SEED0 + 3, frame=256)


def config4() -> Workload:
    """1048576 = 4 x 512 text at seeded frame boundaries + 4088 frames x 256; 28/4."""
    rng = _rng(4)
    F, nf = 256, 4088
    at = np.sort(rng.choice(np.arange(0, nf), size=4, replace=False))
    segs, prev = [], 0
    for b in at:
        if b > prev:
            segs.append((1, int(b - prev) * F))
        segs.append((0, 512))
        prev = int(b)
    if nf > prev:
        segs.append((1, (nf - prev) * F))
    mod = _layout(segs)
    S = len(mod)
    assert S == 1048576
    sig = [F] * 4
    st = Structure(sigma=sig, amp=2.0)
    st.line_slot = _line_slots(rng, sig)
    kinds = [C.global_head(C.grid_window(F)), C.global_head(C.ashape(128, 4096)),
             C.global_head(C.vslash(1000, 1024)), qb_head(F), b2d_head(F)]
    heads = [kinds[h % 5] for h in range(28)]
    return Workload("cfg4_mm_1m", S, 28, 4, mod, heads, st, SEED0 + 4, frame=F,
                    extra={"text_at_frames": at.tolist()})


def search_calibration() -> Workload:
    """Calibration sample of the pattern search (Appendix C.5: one sample of
    at most 25K tokens): 24,576 tokens, T V T V with text U{512..2048} and
    whole 196-token frames, 28/4 heads, the 128K workload's planted
    structure."""
    rng = _rng(6)
    S, F = 24576, 196
    text = [int(rng.integers(512, 2049)) for _ in range(2)]
    nf = (S - sum(text)) // F
    text[-1] += S - sum(text) - nf * F
    cut = int(rng.integers(nf // 4, 3 * nf // 4))
    segs = [(0, text[0]), (1, cut * F), (0, text[1]), (1, (nf - cut) * F)]
    mod = _layout(segs)
    assert len(mod) == S
    st = Structure(sigma=[F] * 4, amp=2.0, text_amp=1.0)
    st.line_slot = _line_slots(rng, st.sigma)
    heads = [C.global_head(C.dense())] * 28
    return Workload("search_calib_24k", S, 28, 4, mod, heads, st, SEED0 + 6, frame=F)


def natten_video() -> Workload:
    """Neighborhood attention stand-in for one video DiT layer (Appendix F):
    a 33 x 45 x 80 token grid (118,800 tokens: the latent of a 129-frame
    720p clip under 4x temporal / 8x spatial compression and 2 x 2 patches),
    24 heads without GQA, 9 x 15 x 15 windows (about 1.7% of the tokens per
    query), tiles of 2 x 4 x 8 tokens (the power-of-two tile with the fewest
    selected tile pairs for these windows). Plain N(0, 1) Q/K/V: the
    pattern is static, nothing is estimated from the data."""
    grid, win, H = (33, 45, 80), (9, 15, 15), 24
    S = grid[0] * grid[1] * grid[2]
    op = C.natten(grid, win, (2, 4, 8))
    st = Structure(sigma=[1] * H, amp=0.0)
    return Workload("natten_video_119k", S, H, H, np.zeros(S, np.uint8), [C.global_head(op)] * H, st,
                    SEED0 + 5, extra={"grid": grid, "win": win, "tile": op.tile})


ALL = [config0, config1, config2, config3, config4]


def by_id(cid: int) -> Workload:
    wl = ALL[cid]()
    assert len(wl.modality) == wl.S, (wl.name, len(wl.modality), wl.S)
    return wl
