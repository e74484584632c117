"""The host consistency checks of the C-ABI (mmi_check_index, mmi_check_work)
on the CPU: hand-built valid block indices, row-group unions and work lists
pass, and each planted corruption of them (a duplicated or missing position,
an out-of-range or unordered key block, a wrong select or mask bit, a gap or
overlap in the work list, a reused partial slot, an item missing from the
item map) is reported with its table and index. The same checks on real
plans, and the MMI_DEBUG mode that runs them, are GPU tests
(test_gpu_debug.py)."""
import numpy as np
import pytest

from paper_2504_16083_amd import mmi

BIG = 0x7FFFFFFF


def _index(seed, S=1000, R=4, rho=2, causal=True, layouts=1, identity=False):
    """A consistent head index: random permutations with padding slots, a
    random block selection per query block (its own diagonal blocks always
    in), and the row-group unions rebuilt by their definition."""
    rng = np.random.default_rng(seed)
    nb = (S + 63) // 64 + 2                      # two blocks of padding slots
    def perm():
        p = np.full(nb * 64, -1, np.int32)
        slots = rng.choice(nb * 64, S, replace=False)
        p[slots] = rng.permutation(S).astype(np.int32)
        return p
    qp = None if identity else perm()
    kps = [perm() for _ in range(layouts)]
    kp = None if identity and layouts == 1 else np.concatenate(kps)
    nbq, nbk = (S + 63) // 64 if identity else nb, ((S + 63) // 64 if identity else nb) * layouts
    qs = (qp if qp is not None else np.where(np.arange(nbq * 64) < S, np.arange(nbq * 64), -1)).reshape(nbq, 64)
    ks = (kp if kp is not None else np.where(np.arange(nbk * 64) < S, np.arange(nbk * 64), -1)).reshape(nbk, 64)
    rows = []
    for i in range(nbq):
        pick = set(np.flatnonzero(rng.random(nbk) < 0.3).tolist())
        live = qs[i][qs[i] >= 0]
        for j in range(nbk):                    # blocks holding a query's own key
            if np.isin(ks[j], live).any():
                pick.add(j)
        rows.append(sorted(pick))
    rp = np.zeros(nbq + 1, np.int32)
    rp[1:] = np.cumsum([len(r) for r in rows])
    col = np.array([j for r in rows for j in r], np.int32)
    kmax = np.where((ks < 0).any(axis=1), BIG, ks.max(axis=1))
    qmin = np.where(qs >= 0, qs, BIG).min(axis=1)
    ng = (nbq + R * rho - 1) // (R * rho) * rho
    uptr, ent = [0], []
    for g in range(ng):
        mem = [(g // rho) * (R * rho) + g % rho + r * rho for r in range(R)]
        lists = [set(rows[i]) if i < nbq else set() for i in mem]
        exist = [lists[r] for r in range(R) if mem[r] < nbq]
        common = set.intersection(*exist) if exist else set()
        for j in sorted(common) + sorted(set().union(*lists) - common):
            sel = sum(1 << r for r in range(R) if j in lists[r])
            need = [mem[r] < nbq and ((kmax[j] > qmin[mem[r]]) if causal else kmax[j] == BIG) for r in range(R)]
            msk = sum(1 << r for r in range(R) if j in lists[r] and need[r])
            ent.append(np.uint32(j | (sel << 16) | (msk << 24)).view(np.int32))
        uptr.append(len(ent))
    return dict(S=S, n_qblocks=nbq, n_kblocks=nbk, row_ptr=rp, col_idx=col, qperm=qp, kperm=kp, n_layouts=layouts,
                causal=causal, group_size=R, group_stride=rho, union_ptr=np.array(uptr, np.int32),
                union_ent=np.array(ent, np.int32))


def _fails(ix, fragment):
    with pytest.raises(mmi.MMIError) as e:
        mmi.mmi_check_index(**ix)
    assert e.value.status == mmi.ERR_INTERNAL and fragment in str(e.value), str(e.value)


@pytest.mark.parametrize("kw", [dict(), dict(identity=True), dict(causal=False), dict(layouts=2), dict(R=2, rho=1),
                                dict(R=1, rho=1), dict(S=64 * 9, rho=4)])
def test_valid_index_passes(kw):
    mmi.mmi_check_index(**_index(3, **kw))


def test_index_corruptions_are_reported():
    base = _index(5)
    def mod(**upd):
        d = {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in base.items()}
        for k, f in upd.items():
            f(d[k])
        return d
    live = np.flatnonzero(base["qperm"] >= 0)
    _fails(mod(qperm=lambda a: a.__setitem__(live[1], a[live[0]])), "qperm: position")
    _fails(mod(qperm=lambda a: a.__setitem__(live[0], base["S"])), "qperm[")
    _fails(mod(kperm=lambda a: a.__setitem__(np.flatnonzero(a >= 0)[7], -1)), "kperm: position")
    _fails(mod(row_ptr=lambda a: a.__setitem__(3, a[2] - 1)), "row_ptr decreases")
    _fails(mod(col_idx=lambda a: a.__setitem__(0, base["n_kblocks"])), "not a key block")
    r = next(i for i in range(base["n_qblocks"]) if base["row_ptr"][i + 1] - base["row_ptr"][i] >= 2)
    a0 = base["row_ptr"][r]
    _fails(mod(col_idx=lambda a: a.__setitem__(slice(a0, a0 + 2), a[a0:a0 + 2][::-1].copy())), "not ascending")
    ent = base["union_ent"].view(np.uint32)

    def set_ent(x, val):
        return lambda a: a.__setitem__(x, np.uint32(val).view(np.int32))
    _fails(mod(union_ent=set_ent(0, (ent[0] & ~np.uint32(0xFFFF)) | np.uint32(base["n_kblocks"]))), "key block")
    # a select bit of a member past the last query block (the last group's last member)
    g = len(base["union_ptr"]) - 2
    x = base["union_ptr"][g]
    mem = [(g // 2) * 8 + g % 2 + r * 2 for r in range(4)]
    assert mem[-1] >= base["n_qblocks"] and base["union_ptr"][g + 1] > x
    _fails(mod(union_ent=set_ent(x, int(ent[x]) | (1 << 19))), "select bits")
    # mask bit cleared / set against the positions (identity order: blocks
    # below a member's query block need no mask, those from it on do)
    idn = _index(6, identity=True)
    ient = idn["union_ent"].view(np.uint32)
    for x, flip in ((int(np.flatnonzero((ient >> 24) & 1)[0]), 1 << 24),
                    (int(np.flatnonzero(((ient >> 16) & 1) & ~((ient >> 24) & 1))[0]), 1 << 24)):
        d = dict(idn, union_ent=idn["union_ent"].copy())
        d["union_ent"][x] = np.uint32(int(ient[x]) ^ flip).view(np.int32)
        _fails(d, "mask bit")
    # a member's select bit removed from an entry other members keep
    xs = int(np.flatnonzero((((ent >> 16) & 0xF) != 1) & ((ent >> 16) & 1))[0])
    _fails(mod(union_ent=set_ent(xs, int(ent[xs]) & ~(1 << 16) & ~(1 << 24))), "")
    # one key block twice in a group, and the common part out of order
    g2 = next(g for g in range(len(base["union_ptr"]) - 1) if base["union_ptr"][g + 1] - base["union_ptr"][g] >= 3)
    a, b = base["union_ptr"][g2], base["union_ptr"][g2 + 1]
    _fails(mod(union_ent=set_ent(a + 1, ent[a])), "")
    d = mod()
    d["union_ent"][a:b] = d["union_ent"][a:b][::-1].copy()
    _fails(d, "group")


def _work(seed, nheads=3, chunk=3):
    """A consistent work list: per head, groups with random union sizes cut
    into items of `chunk` entries; split groups get consecutive partial slots
    and a split row; the items dealt over 8 XCD rows of the item map."""
    rng = np.random.default_rng(seed)
    uptrs, items, splits, nparts = [], [], [], 0
    for h in range(nheads):
        sizes = rng.integers(0, 10, int(rng.integers(3, 9)))
        up = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
        uptrs.append(up)
        for g, n in enumerate(sizes):
            if n == 0:
                continue
            nch = (int(n) + chunk - 1) // chunk
            p0 = nparts if nch > 1 else -1
            for c in range(nch):
                e0 = int(up[g]) + c * chunk
                items.append([h, g, e0, min(e0 + chunk, int(up[g + 1])), p0 + c if nch > 1 else -1])
            if nch > 1:
                splits.append([h, g, p0, nch])
                nparts += nch
    order = rng.permutation(len(items))
    L = (len(items) + 7) // 8 + 1
    imap = np.full((8, L), -1, np.int32)
    for k, it in enumerate(order):
        imap[k % 8, k // 8] = it
    return dict(union_ptrs=uptrs, items=np.array(items, np.int32), n_parts=nparts,
                splits=np.array(splits, np.int32).reshape(-1, 4), item_map=imap)


def _work_fails(w, fragment):
    with pytest.raises(mmi.MMIError) as e:
        mmi.mmi_check_work(**w)
    assert e.value.status == mmi.ERR_INTERNAL and fragment in str(e.value), str(e.value)


def test_valid_work_passes():
    for seed in range(4):
        mmi.mmi_check_work(**_work(seed))


def test_work_corruptions_are_reported():
    base = _work(11)
    assert len(base["splits"]) >= 2
    def mod():
        return {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in base.items()}
    it = base["items"]
    s = next(i for i in range(len(it)) if it[i, 4] >= 0 and i + 1 < len(it) and it[i + 1, 4] == it[i, 4] + 1)
    w = mod(); w["items"][s + 1, 2] += 1
    _work_fails(w, "entries")                       # a gap between two items of a group
    w = mod(); w["items"][s, 3] -= 1
    _work_fails(w, "entries")                       # the next item no longer starts where this one ends
    w = mod(); w["items"][s + 1, 4] = w["items"][s, 4]
    _work_fails(w, "partial slot")                  # a partial slot used twice
    w = mod(); w["items"][[s, s + 1]] = w["items"][[s + 1, s]]
    _work_fails(w, "entries")                       # two items of a group swapped
    w = mod(); w["splits"][0, 3] += 1
    _work_fails(w, "split row")
    w = mod(); w["splits"] = w["splits"][1:]
    _work_fails(w, "split rows")
    w = mod(); w["item_map"][w["item_map"] == 0] = -1
    _work_fails(w, "not in the item map")
    w = mod(); w["item_map"][w["item_map"] == 1] = 0
    _work_fails(w, "item map entry")
    single = next(i for i in range(len(it)) if it[i, 4] < 0)
    w = mod(); w["items"][single, 4] = base["n_parts"] - 1
    _work_fails(w, "partial slot")
    # a group whose union entries no item covers
    w = mod()
    drop = single
    keep = np.array([i for i in range(len(it)) if i != drop])
    remap = {int(o): n for n, o in enumerate(keep)}
    w["items"] = it[keep]
    w["item_map"] = np.array([[remap.get(int(x), -1) if x >= 0 else -1 for x in row] for row in base["item_map"]],
                             np.int32)
    _work_fails(w, "in no item")
