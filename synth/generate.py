"""Seeded synthetic Q/K/V with the structure of the paper's video/text workloads.

The paper measures on real VLM activations of long videos (Section 4.1,
Appendix D); those models and datasets are not available, so these seeded
inputs stand in for them. They take the paper's shapes: tokens per frame
(196 for VideoChat-Flash, Section 4.5; 256 in Figure "motivations_sparsity"),
frame counts up to about 1M tokens (V-NIAH, Section 4.1), text inserted
between frames (MM-NIAH, Section 4.1), grid heads whose period is the frame
size (Section 2.2) and text with local/sink structure (Section 2.2).

This module draws random numbers only; it holds none of the method's
arithmetic. The same tensors feed the HIP path and the CPU oracle.

Structure planted per KV group g (added to Q of every query head of g and
to K of head g; to V only where v_embed is set):
  * slot embedding  E_g[s] ~ amp * N(0, I)  at video tokens whose video-local
    index is s mod sigma_g  (the same-spatial-slot lines of the grid); with
    v_embed the same embedding is added to V as well (Q, K and V share the
    per-position embedding, so outputs reach |O| of several units);
  * one line slot p*_g: keys of that slot get  line_k * w_g  and every video
    query gets  line_q * w_g  (the vertical lines of the grid);
  * text: a causal exponential-filter (AR(1)-like) bias of amplitude
    text_amp on text Q/K (local-window structure);
  * sinks: a fraction of key positions get  3 * u_g, all queries 0.5 * u_g.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np
import torch

from .config import HeadCfg


@dataclass
class Structure:
    sigma: List[int]                  # planted stride per KV group
    amp: float = 2.0                  # slot-embedding per-element std
    line_q: float = 1.0
    line_k: float = 4.0
    text_amp: float = 0.0             # text local bias amplitude (0 = off)
    text_rho: float = 0.95
    sink_frac: float = 0.0
    line_slot: Optional[List[int]] = None   # filled by make_workload (seeded)
    v_embed: bool = False             # add the slot embedding to V too


@dataclass
class Workload:
    name: str
    S: int
    Hq: int
    Hkv: int
    modality: np.ndarray              # uint8 [S]; 0 = text, 1 = video
    heads: List[HeadCfg]
    structure: Structure
    seed: int
    frame: int = 0                    # tokens per frame of the video modality
    note: str = ""
    extra: dict = field(default_factory=dict)


def video_index(modality: np.ndarray) -> np.ndarray:
    """Positions of video tokens (modality 1), ascending."""
    return np.nonzero(modality == 1)[0]


def segments(modality: np.ndarray):
    """Maximal runs [(modality, start, end)] of the layout."""
    m = np.asarray(modality)
    cut = np.nonzero(np.diff(m.astype(np.int16)))[0] + 1
    starts = np.concatenate([[0], cut])
    ends = np.concatenate([cut, [len(m)]])
    return [(int(m[a]), int(a), int(b)) for a, b in zip(starts, ends)]


def _periodic(E, first, n):
    """Rows E[(first + i) mod len(E)] for i < n, built from copies only."""
    sig = E.shape[0]
    reps = (n + sig - 1) // sig + 1
    return torch.roll(E, -first, 0).repeat(reps, 1)[:n]


def make_qkv(wl: Workload, device="cpu", dtype=torch.bfloat16):
    """Q [S,Hq,128], K [S,Hkv,128], V [S,Hkv,128] (bf16) for the workload.

    Deterministic for a given (workload seed, device type). Large tensors are
    only ever updated through contiguous or strided slices."""
    S, Hq, Hkv, D = wl.S, wl.Hq, wl.Hkv, 128
    if len(wl.modality) != S:
        raise ValueError(f"layout has {len(wl.modality)} tokens, S = {S}")
    G = Hq // Hkv
    dev = torch.device(device)
    gen = torch.Generator(device=dev)
    gen.manual_seed(int(wl.seed))

    def randn(*shape):
        return torch.randn(*shape, generator=gen, device=dev, dtype=torch.float32)

    Q = randn(S, Hq, D)
    K = randn(S, Hkv, D)
    V = randn(S, Hkv, D)
    st = wl.structure
    segs = segments(wl.modality)
    vsegs, vloc = [], 0
    for m, a, b in segs:
        if m == 1:
            vsegs.append((a, b, vloc))
            vloc += b - a
    if vsegs:
        for g in range(Hkv):
            sig = int(st.sigma[g])
            E = st.amp * randn(sig, D)
            w = randn(D)
            p_star = int(st.line_slot[g]) if st.line_slot else 0
            for a, b, v0 in vsegs:
                e = _periodic(E, v0 % sig, b - a)
                K[a:b, g] += e
                Q[a:b, g * G:(g + 1) * G] += e[:, None, :]
                if st.v_embed:
                    V[a:b, g] += e
                first = (p_star - v0) % sig
                K[a + first:b:sig, g] += st.line_k * w
                Q[a:b, g * G:(g + 1) * G] += st.line_q * w
    tsegs = [(a, b) for m, a, b in segs if m == 0]
    n_txt = sum(b - a for a, b in tsegs)
    if st.text_amp > 0 and n_txt > 1:
        taps = 128
        kern = torch.tensor([st.text_rho ** t for t in range(taps)], device=dev,
                            dtype=torch.float32) * math.sqrt(1 - st.text_rho ** 2)
        for g in range(Hkv):
            z = randn(1, D, n_txt + taps - 1)
            z = torch.nn.functional.conv1d(z.reshape(D, 1, -1), kern.flip(0).reshape(1, 1, -1))
            z = z.reshape(D, n_txt).t() * st.text_amp
            off = 0
            for a, b in tsegs:
                K[a:b, g] += z[off:off + b - a]
                Q[a:b, g * G:(g + 1) * G] += z[off:off + b - a, None, :]
                off += b - a
    if st.sink_frac > 0:
        nsink = max(1, int(round(st.sink_frac * S)))
        perm = torch.randperm(S, generator=gen, device=dev)[:nsink]
        for g in range(Hkv):
            u = randn(D)
            K[:, g].index_add_(0, perm, (3.0 * u).expand(nsink, D).contiguous())
            Q[:, g * G:(g + 1) * G] += 0.5 * u
    return Q.to(dtype), K.to(dtype), V.to(dtype)
