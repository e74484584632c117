"""Masked softmax attention in fp64 (the computation of Algorithms 5-7).

For a query at position q with the element mask M(q) of its head plan
(selected blocks, causal by original positions unless the head is
bidirectional):
    O[q]   = sum_{k in M(q)} softmax_k(tau * q.k) V[k]
    LSE[q] = ln sum_{k in M(q)} exp(tau * q.k)
Skipped keys contribute exactly zero. This is the plain definition; the
online-softmax recurrence of the kernels (running max m, running sum l,
rescale alpha) reaches the same value up to rounding.

Pinned in tests/test_oracle_attention.py: with every causal block selected
it equals torch's fp64 scaled_dot_product_attention (causal); every softmax
row sums to 1; LSE equals scipy's logsumexp over the masked logits.
"""
import math

import numpy as np

from . import estimate, plan as P


def attend(qvec, K, V, keys, scale):
    s = scale * (K[keys] @ qvec)
    m = s.max()
    e = np.exp(s - m)
    l = e.sum()
    return (e / l) @ V[keys], m + math.log(l)


def head_rows(hp: P.HeadPlan, Qh, K, V, rows, scale=None):
    """O [len(rows), D] and LSE [len(rows)] for the given query positions.

    Qh: fp64 [S, D] or a callable positions -> rows; K, V: fp64 [S, D].
    Rows of one permuted query block share that block's selected key
    blocks, so their logits come from one product with the union of those
    keys; each row then keeps only its own causal keys (k <= q) and takes
    the plain softmax over them."""
    scale = estimate.tau(K.shape[1]) if scale is None else scale
    rows = np.asarray(rows, dtype=np.int64)
    qv = Qh(rows) if callable(Qh) else Qh[rows]
    O = np.zeros((len(rows), V.shape[1]))
    L = np.zeros(len(rows))
    slot_of = np.full(hp.S, -1, dtype=np.int64)
    valid = hp.qperm >= 0
    slot_of[hp.qperm[valid]] = np.nonzero(valid)[0]
    qblk = slot_of[rows] // P.B
    blocks = np.unique(qblk)
    # gathered key rows go to buffers allocated once (sized for the largest
    # key set) and reused by every block
    nmax = max((len(hp.blocks[i]) for i in blocks), default=0) * P.B
    kbuf, vbuf = np.empty((nmax, K.shape[1])), np.empty((nmax, V.shape[1]))
    for i in blocks:
        sel = np.nonzero(qblk == i)[0]
        ks = np.concatenate([hp.kperm[j * P.B:(j + 1) * P.B] for j in hp.blocks[i]])
        keys = np.sort(ks[ks >= 0])
        Kk = np.take(K, keys, axis=0, out=kbuf[:len(keys)], mode="clip")   # keys are in range
        Vk = np.take(V, keys, axis=0, out=vbuf[:len(keys)], mode="clip")
        s = scale * (qv[sel] @ Kk.T)                            # [rows of block i, keys]
        if hp.causal:
            s = np.where(keys[None, :] <= rows[sel][:, None], s, -np.inf)
        m = s.max(axis=1)
        e = np.exp(s - m[:, None])                              # masked keys give exactly 0
        l = e.sum(axis=1)
        O[sel] = (e / l[:, None]) @ Vk
        L[sel] = m + np.log(l)
    return O, L


def dense_causal_rows(Qh, K, V, rows, scale=None):
    """Plain causal attention (every k <= q) for the given rows."""
    scale = estimate.tau(K.shape[1]) if scale is None else scale
    O = np.zeros((len(rows), V.shape[1]))
    L = np.zeros(len(rows))
    for n, q in enumerate(rows):
        qv = Qh(np.array([q]))[0] if callable(Qh) else Qh[q]
        O[n], L[n] = attend(qv, K, V, np.arange(q + 1), scale)
    return O, L


def permuted_blockwise(hp: P.HeadPlan, Qh, K, V, scale=None):
    """The same result computed the way Algorithms 5-7 do: gather Q/K/V into
    slot order through the permutations, walk each query block's selected key
    blocks with the online-softmax recurrence (running max m, sum l, rescale
    alpha), mask causally by the carried original positions, normalise by l
    and scatter each row back to its position. Returns O [S, D], LSE [S]."""
    scale = estimate.tau(K.shape[1]) if scale is None else scale
    S, D = hp.S, V.shape[1]
    O = np.zeros((S, D))
    LSE = np.zeros(S)
    for i in range(hp.nbq):
        qpos = hp.qperm[i * P.B:(i + 1) * P.B]
        live = qpos >= 0
        qc = np.where(live[:, None], Qh[np.maximum(qpos, 0)], 0.0)
        m = np.full(P.B, -np.inf)
        l = np.zeros(P.B)
        acc = np.zeros((P.B, D))
        for j in hp.blocks[i]:
            kpos = hp.kperm[j * P.B:(j + 1) * P.B]
            kc = K[np.maximum(kpos, 0)]
            vc = V[np.maximum(kpos, 0)]
            s = scale * (qc @ kc.T)
            ok = (kpos[None, :] >= 0) & live[:, None]
            if hp.causal:
                ok &= kpos[None, :] <= qpos[:, None]
            s = np.where(ok, s, -np.inf)
            m_new = np.maximum(m, s.max(axis=1))
            safe = np.where(np.isfinite(m_new), m_new, 0.0)
            p = np.exp(s - safe[:, None])
            alpha = np.where(np.isfinite(m), np.exp(m - safe), 0.0)
            l = alpha * l + p.sum(axis=1)
            acc = alpha[:, None] * acc + p @ vc
            m = m_new
        rows = qpos[live]
        O[rows] = acc[live] / l[live, None]
        LSE[rows] = m[live] + np.log(l[live])
    return O, LSE
