// Host-side consistency checks of a plan's tables (the debug mode of the
// runtime, and mmi_check_index / mmi_check_work of the C-ABI). Every index the attention
// kernel derives from these tables (permutation slots, key blocks, union
// entries, work items, partial slots, the item map) is in bounds when they
// pass, so a plan that passes cannot make the kernel read or write outside
// its buffers. Each check returns an empty string, or the first violation.
#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <string>
#include <vector>

#include "device.hpp"
#include "internal.hpp"

namespace mmi {

namespace {

std::string msg(const char* fmt, ...) {
  char buf[256];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  return buf;
}

// A permutation table of nslots slots: every entry -1 (padding) or a
// position in [0, S), each position exactly once.
std::string check_perm(const char* name, const int32_t* perm, int64_t nslots, int S) {
  if (!perm) {
    if (nslots < S) return msg("%s: identity over %lld slots does not hold %d positions", name, (long long)nslots, S);
    return {};
  }
  std::vector<int64_t> seen(S, -1);
  for (int64_t x = 0; x < nslots; ++x) {
    const int32_t p = perm[x];
    if (p == -1) continue;
    if (p < 0 || p >= S) return msg("%s[%lld] = %d: not a position of [0, %d)", name, (long long)x, p, S);
    if (seen[p] >= 0) return msg("%s: position %d in slots %lld and %lld", name, p, (long long)seen[p], (long long)x);
    seen[p] = x;
  }
  for (int p = 0; p < S; ++p)
    if (seen[p] < 0) return msg("%s: position %d in no slot", name, p);
  return {};
}

int32_t slot_of(const int32_t* perm, int64_t x, int S) { return perm ? perm[x] : (x < S ? (int32_t)x : -1); }

}  // namespace

std::string check_index(const mmi_index_view& v) {
  const int S = v.S, nbq = v.n_qblocks, nbk = v.n_kblocks;
  if (S < 1 || nbq < 1 || nbk < 1 || nbk > 0x10000 || (int64_t)nbq * B < S || (int64_t)nbk * B < S)
    return msg("sizes: S %d, %d query blocks, %d key blocks", S, nbq, nbk);
  if (!v.row_ptr || !v.col_idx) return "row_ptr / col_idx missing";
  const int nlay = v.n_layouts;
  if (nlay < 1 || nbk % nlay != 0 || (int64_t)(nbk / nlay) * B < S || (nlay > 1 && !v.kperm))
    return msg("%d key layouts of %d key blocks", nlay, nbk);
  std::string e = check_perm("qperm", v.qperm, (int64_t)nbq * B, S);
  for (int l = 0; l < nlay && e.empty(); ++l) {
    const int64_t per = (int64_t)(nbk / nlay) * B;
    e = check_perm(l == 0 ? "kperm" : "kperm (a later layout)", v.kperm ? v.kperm + l * per : nullptr, per, S);
  }
  if (!e.empty()) return e;
  if (v.row_ptr[0] != 0) return msg("row_ptr[0] = %d", v.row_ptr[0]);
  for (int i = 0; i < nbq; ++i) {
    const int a = v.row_ptr[i], b = v.row_ptr[i + 1];
    if (b < a) return msg("row_ptr decreases at row %d (%d -> %d)", i, a, b);
    for (int x = a; x < b; ++x) {
      const int j = v.col_idx[x];
      if (j < 0 || j >= nbk) return msg("col_idx[%d] = %d (row %d): not a key block of [0, %d)", x, j, i, nbk);
      if (x > a && j <= v.col_idx[x - 1]) return msg("row %d: col_idx not ascending at entry %d", i, x);
    }
  }
  if (v.n_groups <= 0) return {};
  const int R = v.group_size, rho = v.group_stride, ng = v.n_groups;
  if (R != 1 && R != 2 && R != 4) return msg("group size %d", R);
  if (rho < 1 || ng < groups_for(nbq, R, rho)) return msg("%d groups with stride %d hold fewer than %d query blocks", ng, rho, nbq);
  if (!v.union_ptr || !v.union_ent) return "union_ptr / union_ent missing";
  if (v.union_ptr[0] != 0) return msg("union_ptr[0] = %d", v.union_ptr[0]);
  // smallest query position of each query block, largest key position of each
  // key block (INT_BIG when it holds padding): the mask bits follow from them
  std::vector<int32_t> qmin(nbq, INT_BIG), kmax(nbk, -1);
  for (int64_t x = 0; x < (int64_t)nbq * B; ++x) {
    const int32_t p = slot_of(v.qperm, x, S);
    if (p >= 0 && p < qmin[x / B]) qmin[x / B] = p;
  }
  for (int64_t x = 0; x < (int64_t)nbk * B; ++x) {
    const int32_t p = slot_of(v.kperm, x, S);
    int32_t& m = kmax[x / B];
    m = p < 0 ? INT_BIG : (m == INT_BIG ? m : std::max(m, p));
  }
  std::vector<int32_t> mark(nbk, -1);      // key block -> entry of the current group
  for (int g = 0; g < ng; ++g) {
    const int a = v.union_ptr[g], b = v.union_ptr[g + 1];
    if (b < a) return msg("union_ptr decreases at group %d", g);
    int rows[4], live = 0;
    for (int r = 0; r < R; ++r) {
      rows[r] = group_row(g, r, R, rho);
      if (rows[r] < nbq) live |= 1 << r;
    }
    bool common = true;                    // still in the part every live member selects
    int prev = -1;
    for (int x = a; x < b; ++x) {
      const uint32_t en = (uint32_t)v.union_ent[x];
      const int j = (int)(en & 0xffffu), sel = (int)((en >> 16) & 0xffu), msk = (int)(en >> 24);
      if (j >= nbk) return msg("group %d entry %d: key block %d of %d", g, x, j, nbk);
      if (sel == 0 || (sel & ~live)) return msg("group %d entry %d: select bits 0x%x, live members 0x%x", g, x, sel, live);
      if (msk & ~sel) return msg("group %d entry %d: mask bits 0x%x outside select bits 0x%x", g, x, msk, sel);
      if (mark[j] >= a) return msg("group %d: key block %d in entries %d and %d", g, j, mark[j], x);
      mark[j] = x;
      const bool all = sel == live;
      if (all && !common) return msg("group %d entry %d: a block of every member after the others", g, x);
      if (!all && common) { common = false; prev = -1; }
      if (j <= prev) return msg("group %d entry %d: key blocks not ascending", g, x);
      prev = j;
      for (int r = 0; r < R; ++r) {
        if (!((sel >> r) & 1)) continue;
        const bool need = v.causal ? kmax[j] > qmin[rows[r]] : kmax[j] == INT_BIG;
        if (need != (bool)((msk >> r) & 1))
          return msg("group %d entry %d: mask bit of member %d is %d, the block %s a mask", g, x, r, (msk >> r) & 1,
                     need ? "needs" : "needs no");
      }
    }
    // every member's select bits mark exactly its query block's key blocks
    for (int r = 0; r < R; ++r) {
      if (!((live >> r) & 1)) continue;
      const int i = rows[r];
      int n = 0;
      for (int x = v.row_ptr[i]; x < v.row_ptr[i + 1]; ++x) {
        const int j = v.col_idx[x];
        if (mark[j] < a || !(((uint32_t)v.union_ent[mark[j]] >> (16 + r)) & 1))
          return msg("group %d: key block %d of query block %d has no select bit %d", g, j, i, r);
        ++n;
      }
      int m = 0;
      for (int x = a; x < b; ++x) m += ((uint32_t)v.union_ent[x] >> (16 + r)) & 1;
      if (m != n) return msg("group %d: member %d selects %d key blocks, query block %d lists %d", g, r, m, i, n);
    }
  }
  return {};
}

std::string check_work(const mmi_work_view& w) {
  const int64_t n = w.n_items;
  if (w.n_heads < 0 || n < 0 || w.n_parts < 0 || w.n_splits < 0 || w.map_len < 0) return "negative sizes";
  if ((n > 0 && !w.items) || (w.n_heads > 0 && (!w.n_groups || !w.union_ptr)) || (w.n_splits > 0 && !w.splits) ||
      (w.map_len > 0 && !w.item_map))
    return "work view arrays missing";
  for (int h = 0; h < w.n_heads; ++h)
    if (w.n_groups[h] < 0 || (w.n_groups[h] > 0 && !w.union_ptr[h])) return msg("head %d: %d groups", h, w.n_groups[h]);
  // the items of a row group follow each other and tile its union in order
  std::vector<std::vector<int>> items_of(w.n_heads);   // [head][group] -> number of items
  for (int h = 0; h < w.n_heads; ++h) items_of[h].assign(w.n_groups[h], 0);
  std::vector<uint8_t> part_used(w.n_parts, 0);
  int lh = -1, lg = -1, cursor = 0, nch = 0, part0 = -1;
  auto close_group = [&]() -> std::string {
    if (lh < 0) return {};
    const int end = w.union_ptr[lh][lg + 1];
    if (cursor != end) return msg("head %d group %d: items end at entry %d, its union at %d", lh, lg, cursor, end);
    items_of[lh][lg] = nch;
    return {};
  };
  for (int64_t i = 0; i < n; ++i) {
    const int32_t* it = w.items + 5 * i;
    const int head = it[0], group = it[1], e0 = it[2], e1 = it[3], part = it[4];
    if (head < 0 || head >= w.n_heads) return msg("item %lld: head %d", (long long)i, head);
    if (group < 0 || group >= w.n_groups[head]) return msg("item %lld: group %d of %d", (long long)i, group, w.n_groups[head]);
    if (head != lh || group != lg) {
      std::string e = close_group();
      if (!e.empty()) return e;
      if (head < lh || (head == lh && group < lg) || items_of[head][group] != 0)
        return msg("item %lld: head %d group %d out of order", (long long)i, head, group);
      lh = head; lg = group; cursor = w.union_ptr[lh][lg]; nch = 0; part0 = part;
    }
    const int end = w.union_ptr[lh][lg + 1];
    if (e0 != cursor || e1 < e0 || e1 > end)
      return msg("item %lld: entries [%d, %d), expected from %d up to %d", (long long)i, e0, e1, cursor, end);
    cursor = e1;
    if (part >= 0) {
      if (part >= w.n_parts || part_used[part] || part != part0 + nch)
        return msg("item %lld: partial slot %d (of %lld)", (long long)i, part, (long long)w.n_parts);
      part_used[part] = 1;
    } else if (part != -1 || part0 >= 0) {
      return msg("item %lld: partial slot %d in a group whose first item has %d", (long long)i, part, part0);
    }
    ++nch;
  }
  std::string e = close_group();
  if (!e.empty()) return e;
  int64_t nsplit = 0;
  for (int h = 0; h < w.n_heads; ++h)
    for (int g = 0; g < w.n_groups[h]; ++g) {
      if (items_of[h][g] == 0 && w.union_ptr[h][g + 1] != w.union_ptr[h][g])
        return msg("head %d group %d: union entries [%d, %d) in no item", h, g, w.union_ptr[h][g], w.union_ptr[h][g + 1]);
      nsplit += items_of[h][g] > 1;
    }
  for (int64_t i = 0; i < n; ++i) {   // a group of several items writes partials, a single item writes O
    const int32_t* it = w.items + 5 * i;
    if ((items_of[it[0]][it[1]] > 1) != (it[4] >= 0))
      return msg("item %lld: partial slot %d in a group of %d items", (long long)i, it[4], items_of[it[0]][it[1]]);
  }
  if (w.n_splits != nsplit) return msg("%lld split rows for %lld split groups", (long long)w.n_splits, (long long)nsplit);
  std::vector<std::vector<uint8_t>> split_seen(w.n_heads);
  for (int h = 0; h < w.n_heads; ++h) split_seen[h].assign(w.n_groups[h], 0);
  for (int64_t s = 0; s < w.n_splits; ++s) {
    const int32_t* sr = w.splits + 4 * s;
    const int head = sr[0], group = sr[1], p0 = sr[2], np = sr[3];
    if (head < 0 || head >= w.n_heads || group < 0 || group >= w.n_groups[head] || split_seen[head][group] ||
        items_of[head][group] != np || np < 2 || p0 < 0 || (int64_t)p0 + np > w.n_parts)
      return msg("split row %lld: head %d group %d partials [%d, +%d)", (long long)s, head, group, p0, np);
    split_seen[head][group] = 1;
  }
  // the item map: [8][map_len], every item once, -1 elsewhere
  if (n > 8 * w.map_len) return msg("%lld items, item map of 8 x %lld", (long long)n, (long long)w.map_len);
  std::vector<uint8_t> seen(n, 0);
  for (int64_t x = 0; x < 8 * w.map_len; ++x) {
    const int32_t it = w.item_map[x];
    if (it == -1) continue;
    if (it < 0 || it >= n || seen[it]) return msg("item map entry %lld = %d", (long long)x, it);
    seen[it] = 1;
  }
  for (int64_t i = 0; i < n; ++i)
    if (!seen[i]) return msg("item %lld not in the item map", (long long)i);
  return {};
}

}  // namespace mmi
