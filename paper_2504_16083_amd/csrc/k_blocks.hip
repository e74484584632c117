// Block-index construction: the causal block lift of every head's token
// predicate ("sparse loading, dense computation": whole 64x64 blocks are
// loaded and computed), plus the key block holding each query's own key.
// The mask-index building of the 2D-Boundary head (Section 3.2) and the
// vertical/slash -> block conversion of the VS head (Appendix C.3) are the
// same operation here.
//
// k_key_summaries: per key block the smallest key position (kminpos) and,
//   per VS / VERT op, the position and key block of every selected vertical
//   (selpb: a query block tests at most n_vertical selections instead of
//   every key block).
// k_blocks_count: one workgroup per (head, query block) sets the selected key
//   blocks in an LDS bitmap with closed-form rules (ranges, per-block
//   threshold tests, slash offsets), then stores the bitmap and its
//   popcount. Bit setting is an OR, so the result is order independent.
// k_group_count / k_group_fill: the union of the key-block sets of R
//   query blocks (a row group), with a per-query-block flag on every entry
//   (the attention kernel loads each key block once for all R query blocks).
// k_blocks_scan: per head, prefix sums of counts (CSR row pointers), of the
//   group unions and of work-item counts.
// k_blocks_fill: ascending column lists from the bitmaps.
// k_work_fill: work items (a row group and <= chunk union entries each) and
//   the split-group table for the combine kernel.
#include "device.hpp"
#include "internal.hpp"

namespace mmi {

__global__ __launch_bounds__(256) void k_kminpos(const HeadDev* heads) {
  const HeadDev hd = heads[blockIdx.x];
  const int j = blockIdx.y * 256 + threadIdx.x;
  if (!hd.kminpos || j >= hd.nbk) return;
  int mn = INT_BIG, mx = -1;
  bool pad = false;
  for (int x = 0; x < B; ++x) {
    const int slot = j * B + x;
    const int p = hd.kperm ? hd.kperm[slot] : (slot < hd.S ? slot : -1);
    if (p >= 0) { mn = min(mn, p); mx = max(mx, p); }
    else pad = true;
  }
  hd.kminpos[j] = mn;
  if (hd.kmaxpos) hd.kmaxpos[j] = pad ? INT_BIG : mx;
}

// Position and key block of every selected vertical: a query block selects
// key block b for the verticals iff some selection in b has a position at or
// below the block's largest query position.
__global__ __launch_bounds__(256) void k_sel_blocks(OpDev* ops) {
  const OpDev op = ops[blockIdx.x];
  const int i = blockIdx.y * 256 + threadIdx.x;
  if (!op.selpb || i >= op.nv) return;
  const int kap = op.vsel[i];
  const int pos = op.keymap ? op.keymap[kap] : kap;
  int local = kap;
  if (op.kgrid && op.kparams[0] > 0) local = grid_slot(grid_geo(op.L, op.kparams[0], op.kparams[1]), kap);
  op.selpb[i] = make_int2(pos, local / B);
}

hipError_t launch_key_summaries(const HeadDev* heads, int nheads, OpDev* ops, int nops, Groups g,
                                int max_nbk, int max_sel, hipStream_t st) {
  (void)g;
  if (nheads > 0 && max_nbk > 0)
    hipLaunchKernelGGL(k_kminpos, dim3(nheads, (max_nbk + 255) / 256), dim3(256), 0, st, heads);
  if (nops > 0 && max_sel > 0)
    hipLaunchKernelGGL(k_sel_blocks, dim3(nops, (max_sel + 255) / 256), dim3(256), 0, st, ops);
  return hipGetLastError();
}

// ---------------------------------------------------------------- bitmap rules
struct RowInfo {
  int nvalid;        // valid rows (a prefix of the block)
  int maxpos;        // largest original position among the rows
  int nruns;         // runs of consecutive coordinates
};

__device__ __forceinline__ void set_bit(uint32_t* bm, int j) { atomicOr(&bm[j >> 5], 1u << (j & 31)); }

// all threads call with the same (a, b)
__device__ __forceinline__ void set_range(uint32_t* bm, int a, int b) {
  if (b < a) return;
  const int w0 = a >> 5, w1 = b >> 5;
  for (int w = w0 + (int)threadIdx.x; w <= w1; w += blockDim.x) {
    uint32_t m = 0xffffffffu;
    if (w == w0) m &= 0xffffffffu << (a & 31);
    if (w == w1) m &= 0xffffffffu >> (31 - (b & 31));
    atomicOr(&bm[w], m);
  }
}

// one thread sets the bits [a, b]
__device__ __forceinline__ void set_range_one(uint32_t* bm, int a, int b) {
  for (int w = a >> 5; w <= (b >> 5); ++w) {
    uint32_t m = 0xffffffffu;
    if (w == (a >> 5)) m &= 0xffffffffu << (a & 31);
    if (w == (b >> 5)) m &= 0xffffffffu >> (31 - (b & 31));
    atomicOr(&bm[w], m);
  }
}

// key blocks [kbase, kbase + n) whose threshold value thr[j - kbase] <= lim
__device__ __forceinline__ void set_threshold(uint32_t* bm, const int32_t* thr, int kbase, int n, int lim,
                                              bool identity_blocks) {
  for (int jj = threadIdx.x; jj < n; jj += blockDim.x) {
    const int t = identity_blocks ? (kbase + jj) * B : thr[jj];
    if (t <= lim) set_bit(bm, kbase + jj);
  }
}

// key blocks kbase + b of the selected verticals whose position is <= lim
__device__ __forceinline__ void set_verticals(uint32_t* bm, const OpDev& op, int kbase, int lim) {
  for (int i = threadIdx.x; i < op.nv; i += blockDim.x) {
    const int2 sb = op.selpb[i];
    if (sb.x <= lim) set_bit(bm, kbase + sb.y);
  }
}

// dense / A-shape / VS / static baselines over coordinates whose keys sit at
// key block kbase + c / 64 (row coordinates as runs [ra, rb])
__device__ void identity_rules(uint32_t* bm, const OpDev& op, const int* ra, const int* rb, int nruns,
                               int maxpos, int kbase) {
  const int qmax = rb[nruns - 1];
  if (op.kind == MMI_OP_DENSE || (op.kind == MMI_OP_GRID) ||    // GRID here = dense fallback
      (op.kind == MMI_OP_TRISHAPE && qmax >= op.L - op.bottom)) {  // a final query sees every key
    set_range(bm, kbase, kbase + qmax / B);
  } else if (op.kind == MMI_OP_ASHAPE || op.kind == MMI_OP_TRISHAPE) {
    if (op.sink > 0) set_range(bm, kbase, kbase + min(op.sink - 1, qmax) / B);
    if (op.local > 0)
      for (int r = 0; r < nruns; ++r) set_range(bm, kbase + max(0, ra[r] - op.local + 1) / B, kbase + rb[r] / B);
  } else if (op.kind == MMI_OP_SF_FIXED) {
    // own segment: keys [floor(q/l) l, q] over the run's rows
    for (int r = 0; r < nruns; ++r) set_range(bm, kbase + ra[r] / op.local * op.local / B, kbase + rb[r] / B);
    // segment heads: keys at multiples of the stride up to the last row
    for (int m = threadIdx.x; m <= qmax / op.stride; m += blockDim.x) set_bit(bm, kbase + m * op.stride / B);
  } else if (op.kind == MMI_OP_SF_STRIDED) {
    for (int r = 0; r < nruns; ++r) {
      set_range(bm, kbase + max(0, ra[r] - op.local + 1) / B, kbase + rb[r] / B);
      if (rb[r] - ra[r] + 1 >= op.stride) {
        set_range(bm, kbase, kbase + rb[r] / B);     // the run covers every residue mod stride
      } else {
        // keys q - m*stride for the run's rows q: [ra - m s, rb - m s] for every m
        for (int m = threadIdx.x; m <= rb[r] / op.stride; m += blockDim.x) {
          const int lo = max(0, ra[r] - m * op.stride) / B, hi = (rb[r] - m * op.stride) / B;
          for (int j = lo; j <= hi; ++j) set_bit(bm, kbase + j);
        }
      }
    }
  } else if (op.kind == MMI_OP_VSLASH) {
    set_verticals(bm, op, kbase, maxpos);
    for (int idx = threadIdx.x; idx < op.ns; idx += blockDim.x) {
      const int o = op.ssel[idx];
      for (int r = 0; r < nruns; ++r) {
        if (rb[r] < o) continue;
        const int lo = max(0, ra[r] - o) / B, hi = (rb[r] - o) / B;
        for (int j = lo; j <= hi; ++j) set_bit(bm, kbase + j);
      }
    }
  }
}

// Grid closed forms in the slot space [0, L) of one group (key blocks kbase + ...)
__device__ void grid_rules(uint32_t* bm, const OpDev& op, int sig, int ph, int L, int il, int kbase,
                           const int* rpos, const int32_t* kminpos, bool identity_k, int* sh_maxc) {
  const GridGeo geo = grid_geo(L, sig, ph);
  const int lo = il * B, hi = min(lo + B, L) - 1;
  if (threadIdx.x == 0) *sh_maxc = -1;
  __syncthreads();
  if ((int)threadIdx.x <= hi - lo) atomicMax(sh_maxc, grid_coord(geo, lo + threadIdx.x));
  __syncthreads();
  const int maxc = *sh_maxc;
  const int g0p = grid_g0(geo, ph);
  if (op.use_s) {
    const int cf = grid_coord(geo, lo);
    set_range(bm, kbase + grid_g0(geo, cf % sig) / B, kbase + il);
  }
  if (op.use_v && maxc >= ph) {
    const int f = (maxc - ph) / sig;
    set_range(bm, kbase + g0p / B, kbase + (g0p + f) / B);
  }
  if (op.use_h && hi >= g0p) {
    const int qh = rpos[hi - lo];
    set_threshold(bm, kminpos + kbase, kbase, (L + B - 1) / B, qh, identity_k);
  }
  __syncthreads();
}

// Neighborhood attention, query tile qb (tiles in raster order, one block
// each): per axis the union of the windows of the tile's coordinates is one
// interval; every key tile meeting the product of the intervals is selected.
__device__ void natten_rules(uint32_t* bm, const OpDev& op, int qb) {
  int nt[3], lo[3], hi[3];
  for (int a = 0; a < 3; ++a) nt[a] = (op.grid[a] + op.tile[a] - 1) / op.tile[a];
  const int idx[3] = {qb / (nt[1] * nt[2]), (qb / nt[2]) % nt[1], qb % nt[2]};
  for (int a = 0; a < 3; ++a) {
    const int n = op.grid[a], k = op.win[a], t = op.tile[a];
    const int c0 = idx[a] * t, c1 = min(n, c0 + t) - 1;
    lo[a] = min(max(c0 - k / 2, 0), n - k) / t;
    hi[a] = (min(max(c1 - k / 2, 0), n - k) + k - 1) / t;
  }
  const int rows = (hi[0] - lo[0] + 1) * (hi[1] - lo[1] + 1);
  for (int r = threadIdx.x; r < rows; r += blockDim.x) {      // one run of key tiles per (t, h) tile row
    const int x = lo[0] + r / (hi[1] - lo[1] + 1), y = lo[1] + r % (hi[1] - lo[1] + 1);
    set_range_one(bm, (x * nt[1] + y) * nt[2] + lo[2], (x * nt[1] + y) * nt[2] + hi[2]);
  }
}

// Q-Boundary Grid: query rows rpos[0, nvalid) of one modality in phase
// order (global positions), keys in the Grid order of all S positions at key
// block kbase + slot / 64 (coordinate c sits at slot g0(c mod s) + c / s).
__device__ void qb_grid_rules(uint32_t* bm, const OpDev& op, int sig, int ph, int S, const int* rpos, int nvalid,
                              int maxpos, const int32_t* kminpos, int kbase, int* sh_qh) {
  const GridGeo geo = grid_geo(S, sig, ph);
  if (threadIdx.x == 0) *sh_qh = -1;
  __syncthreads();
  const int r = threadIdx.x;
  if (r < nvalid) {
    const int q = rpos[r], f = q % sig;
    const int g0f = grid_g0(geo, f);
    set_bit(bm, kbase + (g0f + q / sig) / B);                        // the row's own key
    // rows of one phase are contiguous and ascending: the last one reaches furthest
    if (op.use_s && (r + 1 == nvalid || rpos[r + 1] % sig != f))     // same phase, k <= q
      set_range_one(bm, kbase + g0f / B, kbase + (g0f + q / sig) / B);
    if (f == ph) atomicMax(sh_qh, q);
  }
  if (op.use_v && maxpos >= ph) {                                    // phase-p keys, k <= q
    const int g0p = grid_g0(geo, ph);
    set_range(bm, kbase + g0p / B, kbase + (g0p + (maxpos - ph) / sig) / B);
  }
  __syncthreads();
  const int qh = *sh_qh;
  if (op.use_h && qh >= 0) set_threshold(bm, kminpos + kbase, kbase, (S + B - 1) / B, qh, false);
  __syncthreads();
}

__global__ __launch_bounds__(256) void k_blocks_count(const HeadDev* heads, const OpDev* ops, Groups g) {
  const HeadDev hd = heads[blockIdx.x];
  const int qb = blockIdx.y;
  if (qb >= hd.nbq) return;
  __shared__ uint32_t bm[MMI_MAX_SEQ / B / 32 + 8];   // + one block per padded group
  __shared__ int rpos[B], rc[B], ra[B], rb[B];
  __shared__ int sh_nvalid, sh_maxpos, sh_nruns, sh_count, sh_maxc;
  const int tid = threadIdx.x;
  for (int w = tid; w < hd.nwords; w += blockDim.x) bm[w] = 0;
  int gi = -1, li0 = 0;
  if (hd.kind != MMI_HEAD_GLOBAL) {
    const int x = qb * B;
    for (int i = 0; i < g.n; ++i) {
      const int padded = (g.len[i] + B - 1) / B * B;
      if (x >= g.off[i] && x < g.off[i] + padded) gi = i;
    }
    if (gi < 0) return;      // not reachable: every slot < nbq*64 lies in a group
    li0 = x - g.off[gi];
  }
  if (tid < B) {
    const int slot = qb * B + tid;
    const int p = hd.qperm ? hd.qperm[slot] : (slot < hd.S ? slot : -1);
    rpos[tid] = p;
    rc[tid] = hd.kind == MMI_HEAD_2D ? li0 + tid : p;   // coordinate of the row for identity-order rules
  }
  __syncthreads();
  if (tid < B) {
    // wave 0, one row per lane: the leading valid rows, their largest
    // position and their runs of consecutive coordinates [ra, rb]
    const int r = tid;
    const uint64_t vm = __ballot(rpos[r] >= 0);
    const int nv = ~vm ? __builtin_ctzll(~vm) : B;
    const bool in = r < nv;
    const bool start = in && (r == 0 || rc[r] != rc[r - 1] + 1);
    const bool end = in && (r + 1 == nv || rc[r + 1] != rc[r] + 1);
    const uint64_t sm = __ballot(start);
    const uint64_t upto = r == B - 1 ? ~0ull : ((1ull << (r + 1)) - 1);
    const int run = __popcll(sm & upto) - 1;          // the run row r belongs to
    if (start) ra[run] = rc[r];
    if (end) rb[run] = rc[r];
    int mp = in ? rpos[r] : -1;
    for (int off = 32; off > 0; off >>= 1) mp = max(mp, __shfl_xor(mp, off, 64));
    if (r == 0) {
      sh_nvalid = nv;
      sh_maxpos = mp;
      sh_nruns = __popcll(sm);
      sh_count = 0;
    }
  }
  __syncthreads();
  const int maxpos = sh_maxpos, nruns = sh_nruns;
  if (hd.kind == MMI_HEAD_GLOBAL) {
    const OpDev op = ops[hd.op0];
    const int sig = op.kind == MMI_OP_GRID ? op.params[0] : 0;
    if (op.kind == MMI_OP_NATTEN)
      natten_rules(bm, op, qb);
    else if (sig > 0)
      grid_rules(bm, op, sig, op.params[1], hd.S, qb, 0, rpos, hd.kminpos, false, &sh_maxc);
    else
      identity_rules(bm, op, ra, rb, nruns, maxpos, 0);
    if (tid == 0) set_bit(bm, qb);
  } else if (hd.kind == MMI_HEAD_QBOUNDARY) {
    const OpDev op = ops[hd.op0 + gi];
    const int sig = op.kind == MMI_OP_GRID ? op.params[0] : 0;
    if (sig > 0) {
      qb_grid_rules(bm, op, sig, op.params[1], hd.S, rpos, sh_nvalid, maxpos, hd.kminpos, op.kbase, &sh_maxc);
    } else {
      identity_rules(bm, op, ra, rb, nruns, maxpos, op.kbase);
      for (int r = 0; r < nruns; ++r) set_range(bm, op.kbase + ra[r] / B, op.kbase + rb[r] / B);
    }
  } else {
    for (int gk = 0; gk < g.n; ++gk) {
      const OpDev op = ops[hd.op0 + gi * g.n + gk];
      const int kbase = g.off[gk] / B;
      const int nk = (g.len[gk] + B - 1) / B;
      if (gk == gi) {
        const int sig = op.kind == MMI_OP_GRID ? op.params[0] : 0;
        if (sig > 0)
          grid_rules(bm, op, sig, op.params[1], g.len[gi], li0 / B, kbase, rpos, hd.kminpos, false, &sh_maxc);
        else
          identity_rules(bm, op, ra, rb, nruns, maxpos, kbase);
      } else if (op.kind == MMI_OP_DENSE) {
        set_threshold(bm, hd.kminpos + kbase, kbase, nk, maxpos, false);
      } else if (op.kind == MMI_OP_VERT) {
        set_verticals(bm, op, kbase, maxpos);
      }
    }
    if (tid == 0) set_bit(bm, qb);
  }
  __syncthreads();
  int cnt = 0;
  uint32_t* gbm = hd.bitmap + (int64_t)qb * hd.nwords;
  for (int w = tid; w < hd.nwords; w += blockDim.x) {
    const uint32_t v = bm[w];
    gbm[w] = v;
    cnt += __popc(v);
  }
  atomicAdd(&sh_count, cnt);
  __syncthreads();
  if (tid == 0) hd.counts[qb] = sh_count;
}

hipError_t launch_blocks_count(const HeadDev* heads, int nheads, const OpDev* ops, Groups g, int max_nbq,
                               hipStream_t st) {
  if (nheads <= 0 || max_nbq <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_blocks_count, dim3(nheads, max_nbq), dim3(256), 0, st, heads, ops, g);
  return hipGetLastError();
}

// Union size of the key-block sets of a group's members.
__device__ int union_count(const HeadDev& hd, int g, int R, int rho) {
  int cnt = 0;
  for (int w = threadIdx.x; w < hd.nwords; w += blockDim.x) {
    uint32_t u = 0;
    for (int r = 0; r < R; ++r) {
      const int row = group_row(g, r, R, rho);
      if (row < hd.nbq) u |= hd.bitmap[(int64_t)row * hd.nwords + w];
    }
    cnt += __popc(u);
  }
  return cnt;
}

__global__ void k_zero64(int64_t* p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

// Candidate row strides: 1, 2, 4, 8 and the head's extra ones (0 = none).
__device__ __forceinline__ int rho_candidate(const HeadDev& hd, int c) {
  return c < 4 ? 1 << c : hd.rho_alt[c - 4];
}

// Union size of every group for the candidate strides from c0 on
// (gcnt[head][c][g]), and their per-head totals (cand).
__global__ __launch_bounds__(256) void k_group_eval(const HeadDev* heads, int R, int64_t* cand, int32_t* gcnt,
                                                    int max_groups, int c0) {
  const HeadDev hd = heads[blockIdx.x];
  const int g = blockIdx.y;
  __shared__ int sh;
  for (int c = c0; c < NRHO; ++c) {
    const int rho = rho_candidate(hd, c);
    if (rho <= 0) continue;
    if (g >= groups_for(hd.nbq, R, rho)) continue;      // uniform over the block
    if (threadIdx.x == 0) sh = 0;
    __syncthreads();
    atomicAdd(&sh, union_count(hd, g, R, rho));
    __syncthreads();
    if (threadIdx.x == 0) {
      atomicAdd(reinterpret_cast<unsigned long long*>(&cand[blockIdx.x * NRHO + c]), (unsigned long long)sh);
      gcnt[((int64_t)blockIdx.x * NRHO + c) * max_groups + g] = sh;
    }
    __syncthreads();
  }
}

// The same for row groups of four and the strides 1, 2, 4 and 8 in one pass:
// those groups lie inside aligned spans of 32 query blocks (span s holds
// groups 8s .. 8s + 7 of every one of them, group 8s + l starting at block
// 32s + (l / rho) 4 rho + l mod rho), so each bitmap word of a span is read
// once for all four strides. One workgroup per (head, span).
__global__ __launch_bounds__(256) void k_group_eval4(const HeadDev* heads, int64_t* cand, int32_t* gcnt,
                                                     int max_groups) {
  const HeadDev hd = heads[blockIdx.x];
  const int q0 = blockIdx.y * 32;
  if (q0 >= hd.nbq) return;
  __shared__ int red[4][32];            // per wave: counts of [stride c][group l]
  int cnt[32];
#pragma unroll
  for (int k = 0; k < 32; ++k) cnt[k] = 0;
  for (int w = threadIdx.x; w < hd.nwords; w += blockDim.x) {
    uint32_t x[32];
#pragma unroll
    for (int b = 0; b < 32; ++b) x[b] = q0 + b < hd.nbq ? hd.bitmap[(int64_t)(q0 + b) * hd.nwords + w] : 0u;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int rho = 1 << c;
#pragma unroll
      for (int l = 0; l < 8; ++l) {
        const int b0 = (l / rho) * 4 * rho + l % rho;
        cnt[c * 8 + l] += __popc(x[b0] | x[b0 + rho] | x[b0 + 2 * rho] | x[b0 + 3 * rho]);
      }
    }
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int k = 0; k < 32; ++k) {
    int v = cnt[k];
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    if (lane == 0) red[wave][k] = v;
  }
  __syncthreads();
  if (threadIdx.x < 32) {
    const int k = threadIdx.x, c = k >> 3, g = blockIdx.y * 8 + (k & 7);
    const int tot = red[0][k] + red[1][k] + red[2][k] + red[3][k];
    if (g < groups_for(hd.nbq, 4, 1 << c)) {
      gcnt[((int64_t)blockIdx.x * NRHO + c) * max_groups + g] = tot;
      atomicAdd(reinterpret_cast<unsigned long long*>(&cand[blockIdx.x * NRHO + c]), (unsigned long long)tot);
    }
  }
}

__global__ void k_group_pick(const HeadDev* heads, int nheads, int R, const int64_t* cand) {
  const int h = blockIdx.x * blockDim.x + threadIdx.x;
  if (h >= nheads) return;
  const HeadDev hd = heads[h];
  int best = 0;
  for (int c = 1; c < NRHO; ++c)
    if (rho_candidate(hd, c) > 0 && cand[h * NRHO + c] < cand[h * NRHO + best]) best = c;
  hd.gp[0] = rho_candidate(hd, best);
  hd.gp[1] = groups_for(hd.nbq, R, hd.gp[0]);
  hd.gp[2] = best;
}

hipError_t launch_group_stride(const HeadDev* heads, int nheads, int R, int max_groups, int max_nbq, bool extra,
                               int64_t* cand, int32_t* gcnt, hipStream_t st) {
  if (nheads <= 0 || max_groups <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_zero64, dim3((nheads * NRHO + 255) / 256), dim3(256), 0, st, cand, nheads * NRHO);
  if (R == 4) {
    hipLaunchKernelGGL(k_group_eval4, dim3(nheads, (max_nbq + 31) / 32), dim3(256), 0, st, heads, cand, gcnt,
                       max_groups);
    if (extra)   // the extra strides some heads have
      hipLaunchKernelGGL(k_group_eval, dim3(nheads, max_groups), dim3(256), 0, st, heads, R, cand, gcnt, max_groups, 4);
  } else {
    hipLaunchKernelGGL(k_group_eval, dim3(nheads, max_groups), dim3(256), 0, st, heads, R, cand, gcnt, max_groups, 0);
  }
  hipLaunchKernelGGL(k_group_pick, dim3((nheads + 63) / 64), dim3(64), 0, st, heads, nheads, R, cand);
  return hipGetLastError();
}

// The chosen stride's union sizes (counted by k_group_eval).
__global__ __launch_bounds__(256) void k_group_count(const HeadDev* heads, const int32_t* gcnt, int max_groups) {
  const HeadDev hd = heads[blockIdx.x];
  const int gr = blockIdx.y * 256 + threadIdx.x;
  if (gr >= hd.gp[1]) return;
  hd.gcount[gr] = gcnt[((int64_t)blockIdx.x * NRHO + hd.gp[2]) * max_groups + gr];
}

hipError_t launch_group_count(const HeadDev* heads, int nheads, const int32_t* gcnt, int max_groups,
                              hipStream_t st) {
  if (nheads <= 0 || max_groups <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_group_count, dim3(nheads, (max_groups + 255) / 256), dim3(256), 0, st, heads, gcnt,
                     max_groups);
  return hipGetLastError();
}

// ---------------------------------------------------------------- scans
constexpr int SCAN_T = 1024;

// exclusive block scan of one int per thread; returns the block total
__device__ int block_exscan(int v, int* buf, int& excl) {
  const int tid = threadIdx.x;
  buf[tid] = v;
  __syncthreads();
  for (int off = 1; off < SCAN_T; off <<= 1) {
    const int t = tid >= off ? buf[tid - off] : 0;
    __syncthreads();
    buf[tid] += t;
    __syncthreads();
  }
  excl = buf[tid] - v;
  const int tot = buf[SCAN_T - 1];
  __syncthreads();
  return tot;
}

__global__ __launch_bounds__(SCAN_T) void k_blocks_scan(const HeadDev* heads, int min_chunk, int items_per_head,
                                                        int avg_factor, int64_t* totals) {
  const HeadDev hd = heads[blockIdx.x];
  __shared__ int buf[SCAN_T];
  int c_nnz = 0;
  for (int start = 0; start < hd.nbq; start += SCAN_T) {
    const int i = start + threadIdx.x;
    const int cnt = i < hd.nbq ? hd.counts[i] : 0;
    int e0;
    const int t0 = block_exscan(cnt, buf, e0);
    if (i < hd.nbq) hd.rowptr[i] = c_nnz + e0;
    c_nnz += t0;
  }
  const int ngroups = hd.gp[1];
  int c_g = 0;
  for (int start = 0; start < ngroups; start += SCAN_T) {
    const int i = start + threadIdx.x;
    const int cnt = i < ngroups ? hd.gcount[i] : 0;
    int e0;
    const int t0 = block_exscan(cnt, buf, e0);
    if (i < ngroups) hd.growptr[i] = c_g + e0;
    c_g += t0;
  }
  // long unions are split so that no work item holds much more than a
  // 1/items_per_head share of the head's work
  int chunk = max(min_chunk, (int)(((int64_t)c_g + items_per_head - 1) / items_per_head));
  if (avg_factor > 0 && ngroups > 0)
    chunk = max(chunk, (int)min<int64_t>(INT_BIG, (int64_t)avg_factor * (((int64_t)c_g + ngroups - 1) / ngroups)));
  int c_items = 0, c_split = 0, c_parts = 0;
  for (int start = 0; start < ngroups; start += SCAN_T) {
    const int i = start + threadIdx.x;
    const int ch = i < ngroups ? (hd.gcount[i] + chunk - 1) / chunk : 0;
    const int sp = ch > 1 ? 1 : 0;
    const int pt = ch > 1 ? ch : 0;
    int e1, e2, e3;
    const int t1 = block_exscan(ch, buf, e1);
    const int t2 = block_exscan(sp, buf, e2);
    const int t3 = block_exscan(pt, buf, e3);
    if (i < ngroups) {
      hd.chunks[i] = ch;
      hd.itembase[i] = c_items + e1;
      hd.splitoff[i] = c_split + e2;
      hd.partoff[i] = c_parts + e3;
    }
    c_items += t1; c_split += t2; c_parts += t3;
  }
  if (threadIdx.x == 0) {
    hd.rowptr[hd.nbq] = c_nnz;
    hd.growptr[ngroups] = c_g;
    hd.chunklen[0] = chunk;
    int64_t* t = totals + (int64_t)blockIdx.x * NTOT;
    t[0] = c_nnz; t[1] = c_g; t[2] = c_items; t[3] = c_split; t[4] = c_parts;
  }
}

hipError_t launch_blocks_scan(const HeadDev* heads, int nheads, int min_chunk, int items_per_head,
                              int avg_factor, int64_t* totals, hipStream_t st) {
  if (nheads <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_blocks_scan, dim3(nheads), dim3(SCAN_T), 0, st, heads, min_chunk, items_per_head, avg_factor,
                     totals);
  return hipGetLastError();
}

// Words per thread: a bitmap row has at most MMI_MAX_SEQ / 64 / 32 + 8
// words (one padding block per modality group), so 256 threads need 5.
constexpr int GF_WORDS = 5;

// Exclusive prefix sum of one count per thread over a 256-thread workgroup,
// in thread order (wave shuffles, then the wave totals through LDS);
// *total receives the sum of all.
__device__ __forceinline__ int block_exclusive_scan(int cnt, int* wtot, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int s = cnt;
  for (int off = 1; off < 64; off <<= 1) {
    const int t = __shfl_up(s, off, 64);
    if (lane >= off) s += t;
  }
  if (lane == 63) wtot[wave] = s;
  __syncthreads();
  int pre = 0, tot = 0;
  for (int v = 0; v < 4; ++v) {
    if (v < wave) pre += wtot[v];
    tot += wtot[v];
  }
  *total = tot;
  return pre + s - cnt;
}

// Ascending column list of one query block from its bitmap (each thread's
// words read once, kept in registers for the write).
__global__ __launch_bounds__(256) void k_blocks_fill(const HeadDev* heads) {
  const HeadDev hd = heads[blockIdx.x];
  const int qb = blockIdx.y;
  if (qb >= hd.nbq) return;
  __shared__ int wtot[4];
  const uint32_t* gbm = hd.bitmap + (int64_t)qb * hd.nwords;
  const int per = (hd.nwords + 255) / 256;
  const int w0 = threadIdx.x * per;
  uint32_t x[GF_WORDS];
  int cnt = 0;
#pragma unroll
  for (int k = 0; k < GF_WORDS; ++k) {
    x[k] = k < per && w0 + k < hd.nwords ? gbm[w0 + k] : 0u;
    cnt += __popc(x[k]);
  }
  int total;
  int pos = hd.rowptr[qb] + block_exclusive_scan(cnt, wtot, &total);
#pragma unroll
  for (int k = 0; k < GF_WORDS; ++k) {
    uint32_t v = x[k];
    while (v) {
      const int b = __ffs(v) - 1;
      hd.col[pos++] = (w0 + k) * 32 + b;
      v &= v - 1;
    }
  }
}

// Union entries of a row group: first the key blocks every member selects,
// then the others, each part ascending (row groups running side by side then
// start on the blocks they most likely share, which measured ~2% faster than
// one ascending list at 1M tokens). Key block in
// bits 0-15, bit 16+r set if query block r of the group selects it, bit 24+r
// set if it does and the key block holds a position above the smallest
// query position of query block r (or padding), i.e. needs the causal mask
// (for a bidirectional head: only if the key block holds padding).
__global__ __launch_bounds__(256) void k_group_fill(const HeadDev* heads, int R) {
  const HeadDev hd = heads[blockIdx.x];
  const int gr = blockIdx.y;
  if (gr >= hd.gp[1]) return;
  const int rho = hd.gp[0];
  __shared__ int wtot[2][4];
  __shared__ int qmin[4];
  int rows[4];
  for (int r = 0; r < 4; ++r) rows[r] = r < R ? group_row(gr, r, R, rho) : hd.nbq;
  // smallest query position of each member (for the mask flags)
  if (threadIdx.x < 4) qmin[threadIdx.x] = INT_BIG;
  __syncthreads();
  for (int x = threadIdx.x; x < R * B; x += blockDim.x) {
    const int r = x / B, slot = rows[r] * B + x % B;
    if (rows[r] >= hd.nbq) continue;
    const int p = hd.qperm ? hd.qperm[slot] : (slot < hd.S ? slot : -1);
    if (p >= 0) atomicMin(&qmin[r], hd.causal ? p : INT_BIG - 1);   // bidirectional: only padding masks
  }
  // this thread's words of the members' bitmaps, read once for both passes
  const int per = (hd.nwords + 255) / 256;
  const int w0 = threadIdx.x * per;
  uint32_t bits[GF_WORDS][4];
  int cntA = 0, cntB = 0;        // entries every member selects / the others
#pragma unroll
  for (int k = 0; k < GF_WORDS; ++k) {
    const int w = w0 + k;
    const bool in = k < per && w < hd.nwords;
    uint32_t u = 0, a = 0xffffffffu;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      bits[k][r] = in && rows[r] < hd.nbq ? hd.bitmap[(int64_t)rows[r] * hd.nwords + w] : 0u;
      if (rows[r] < hd.nbq) a &= bits[k][r];
      u |= bits[k][r];
    }
    a &= u;
    cntA += __popc(a);
    cntB += __popc(u & ~a);
  }
  // exclusive prefix sums of both counts over the workgroup in thread order
  int totA, totB;
  const int preA = block_exclusive_scan(cntA, wtot[0], &totA);
  const int preB = block_exclusive_scan(cntB, wtot[1], &totB);
  int posA = hd.growptr[gr] + preA;
  int posB = hd.growptr[gr] + totA + preB;
#pragma unroll
  for (int k = 0; k < GF_WORDS; ++k) {
    const int w = w0 + k;
    uint32_t u = 0, a = 0xffffffffu;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      if (rows[r] < hd.nbq) a &= bits[k][r];
      u |= bits[k][r];
    }
    a &= u;
    while (u) {
      const int b = __ffs(u) - 1;
      const int j = w * 32 + b;
      int kmax;                      // largest key position of block j, INT_BIG with padding
      if (hd.kmaxpos) kmax = hd.kmaxpos[j];
      else kmax = j * B + B - 1 < hd.S ? j * B + B - 1 : INT_BIG;
      uint32_t flags = 0;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const uint32_t sel = (bits[k][r] >> b) & 1u;
        flags |= sel << (16 + r);
        if (sel && kmax > qmin[r]) flags |= 1u << (24 + r);
      }
      const int32_t e = (int32_t)((uint32_t)j | flags);
      if ((a >> b) & 1u) hd.gcol[posA++] = e; else hd.gcol[posB++] = e;
      u &= u - 1;
    }
  }
}

hipError_t launch_blocks_fill(const HeadDev* heads, int nheads, int max_nbq, int R, int max_groups,
                              hipStream_t st) {
  if (nheads <= 0 || max_nbq <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_blocks_fill, dim3(nheads, max_nbq), dim3(256), 0, st, heads);
  hipLaunchKernelGGL(k_group_fill, dim3(nheads, max_groups), dim3(256), 0, st, heads, R);
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void k_work_fill(const HeadDev* heads, const int64_t* item_base,
                                                   const int64_t* part_base, const int64_t* split_base,
                                                   WorkItem* items, SplitRow* splits) {
  const int h = blockIdx.x;
  const HeadDev hd = heads[h];
  const int gr = blockIdx.y * 256 + threadIdx.x;
  if (gr >= hd.gp[1]) return;
  const int chunk = hd.chunklen[0];
  const int nch = hd.chunks[gr];
  const int r0 = hd.growptr[gr], r1 = hd.growptr[gr + 1];
  const int64_t ib = item_base[h] + hd.itembase[gr];
  const bool split = nch > 1;
  const int64_t pb = part_base[h] + hd.partoff[gr];
  for (int c = 0; c < nch; ++c) {
    WorkItem w;
    w.head = h;
    w.group = gr;
    w.e0 = r0 + c * chunk;
    w.e1 = min(r0 + (c + 1) * chunk, r1);
    w.part = split ? (int)(pb + c) : -1;
    w.pad[0] = w.pad[1] = w.pad[2] = 0;
    items[ib + c] = w;
  }
  if (split) {
    SplitRow s;
    s.head = h;
    s.group = gr;
    s.part0 = (int)pb;
    s.nparts = nch;
    splits[split_base[h] + hd.splitoff[gr]] = s;
  }
}

// Cost weights: a staged K/V block costs about 1.5 computed blocks (the
// attention kernel's time fitted over the 1M workloads: 2.6 ms per million
// staged blocks, 1.75 ms per million computed blocks).
constexpr float COST_STAGE = 1.5f, COST_COMPUTE = 1.0f;

// One wave per item: sum over its union entries of the staged block and the
// computed blocks (select flags, bits 16-23).
__global__ __launch_bounds__(256) void k_item_cost(const HeadDev* heads, const WorkItem* items, int64_t nitems,
                                                   float* cost) {
  const int64_t it = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (it >= nitems) return;
  const int lane = threadIdx.x & 63;
  const WorkItem w = items[it];
  const int32_t* g = heads[w.head].gcol;
  float acc = 0.0f;
  for (int e = w.e0 + lane; e < w.e1; e += 64)
    acc += COST_STAGE + COST_COMPUTE * (float)__popc(((uint32_t)g[e] >> 16) & 0xffu);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if (lane == 0) cost[it] = acc;
}

hipError_t launch_item_cost(const HeadDev* heads, const WorkItem* items, int64_t nitems, float* cost,
                            hipStream_t st) {
  if (nitems <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_item_cost, dim3((unsigned)((nitems + 3) / 4)), dim3(256), 0, st, heads, items, nitems,
                     cost);
  return hipGetLastError();
}

hipError_t launch_work_fill(const HeadDev* heads, int nheads, const int64_t* item_base,
                            const int64_t* part_base, const int64_t* split_base, int max_groups,
                            WorkItem* items, SplitRow* splits, hipStream_t st) {
  if (nheads <= 0 || max_groups <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_work_fill, dim3(nheads, (max_groups + 255) / 256), dim3(256), 0, st, heads, item_base,
                     part_base, split_base, items, splits);
  return hipGetLastError();
}

}  // namespace mmi
