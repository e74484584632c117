// Modality layout and permutations.
//
// k_positions: the ascending position list T_m of every modality, all lists
//   packed into one pool (the modality type index i_m of Algorithms 2-3).
// k_perms: slot -> position maps of every head (Section 3.1, Algorithm 1
//   "permute Q, K, V"; Section 3.2, Algorithms 2-3 "permute by modality";
//   Appendix C.4): Grid heads group tokens by phase with the chosen phase
//   last; boundary heads concatenate the modality groups (each padded to a
//   multiple of 64 with -1), a 2D-Boundary group in Grid order when its
//   modality op is Grid. A Q-Boundary head with Grid modalities reads its
//   keys through key layouts (position order, then the Grid order of all
//   positions per Grid modality, each ceil(S/64) blocks). The kernels never
//   move Q/K/V for this: attention gathers rows through these maps.
// k_qb_order_*: the queries of a Q-Boundary Grid modality in phase order
//   (the Grid order of all positions restricted to that modality): a
//   stream compaction of the Grid order by modality, in three passes
//   (counts per chunk, offsets, stable fill).
#include "device.hpp"
#include "internal.hpp"

namespace mmi {

__global__ void k_positions(const Segment* segs, int nseg, const int32_t* toff_by_mod, int32_t* tpos,
                            uint8_t* modpos, int S) {
  const int p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= S) return;
  int lo = 0, hi = nseg - 1;     // last segment with pos <= p
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (segs[mid].pos <= p) lo = mid; else hi = mid - 1;
  }
  const Segment sg = segs[lo];
  tpos[toff_by_mod[sg.mod] + sg.loc + (p - sg.pos)] = p;
  if (modpos) modpos[p] = (uint8_t)sg.mod;
}

hipError_t launch_positions(const Segment* segs, int nseg, const int32_t* toff_by_mod, int32_t* tpos,
                            uint8_t* modpos, int S, hipStream_t st) {
  hipLaunchKernelGGL(k_positions, dim3((S + 255) / 256), dim3(256), 0, st, segs, nseg, toff_by_mod, tpos,
                     modpos, S);
  return hipGetLastError();
}

__device__ __forceinline__ int group_of_slot(const Groups& g, int x) {
  for (int i = 0; i < g.n; ++i) {
    const int padded = (g.len[i] + B - 1) / B * B;
    if (x >= g.off[i] && x < g.off[i] + padded) return i;
  }
  return -1;
}

// Position held by key slot x of a Q-Boundary head with key layouts: the
// layout of key block x / 64 is the Grid order of the Grid op whose layout
// starts there, else the position order.
__device__ int qb_key_pos(const HeadDev& hd, const OpDev* ops, const Groups& g, int x) {
  const int nb = (hd.S + B - 1) / B, jb = x / B;
  const int base = jb / nb * nb, xi = x - base * B;
  if (xi >= hd.S) return -1;
  for (int i = 0; i < g.n; ++i) {
    const OpDev& op = ops[hd.op0 + i];
    if (op.kind == MMI_OP_GRID && op.kbase == base && op.params[0] > 0)
      return grid_coord(grid_geo(hd.S, op.params[0], op.params[1]), xi);
  }
  return xi;
}

// Position held by slot x of the neighborhood-attention tile order (-1 for
// the padding of tiles cut by the grid border).
__device__ int natten_pos(const OpDev& op, int x) {
  const int nt1 = (op.grid[1] + op.tile[1] - 1) / op.tile[1], nt2 = (op.grid[2] + op.tile[2] - 1) / op.tile[2];
  const int tile = x / B, in = x % B;
  const int t = tile / (nt1 * nt2) * op.tile[0] + in / (op.tile[1] * op.tile[2]);
  const int h = tile / nt2 % nt1 * op.tile[1] + in / op.tile[2] % op.tile[1];
  const int w = tile % nt2 * op.tile[2] + in % op.tile[2];
  if (t >= op.grid[0] || h >= op.grid[1] || w >= op.grid[2]) return -1;
  return (t * op.grid[1] + h) * op.grid[2] + w;
}

__global__ __launch_bounds__(256) void k_perms(const HeadDev* heads, const OpDev* ops, Groups g,
                                               const int32_t* tpos) {
  const HeadDev hd = heads[blockIdx.x];
  const int x = blockIdx.y * 256 + threadIdx.x;
  if (hd.kind == MMI_HEAD_QBOUNDARY && hd.kperm && x < hd.nbk * B) hd.kperm[x] = qb_key_pos(hd, ops, g, x);
  if (!hd.qperm || x >= hd.nbq * B) return;
  int pos = -1;
  if (hd.kind == MMI_HEAD_GLOBAL && ops[hd.op0].kind == MMI_OP_NATTEN) {
    pos = natten_pos(ops[hd.op0], x);
  } else if (hd.kind == MMI_HEAD_GLOBAL) {
    const OpDev op = ops[hd.op0];
    const int sig = op.params ? op.params[0] : 0;
    if (x < hd.S) pos = sig > 0 ? grid_coord(grid_geo(hd.S, sig, op.params[1]), x) : x;
  } else {
    const int gi = group_of_slot(g, x);
    const int li = gi >= 0 ? x - g.off[gi] : 0x7fffffff;
    if (gi >= 0 && li < g.len[gi]) {
      int coord = li;
      if (hd.kind == MMI_HEAD_2D) {
        const OpDev op = ops[hd.op0 + gi * g.n + gi];
        if (op.kind == MMI_OP_GRID && op.params[0] > 0)
          coord = grid_coord(grid_geo(g.len[gi], op.params[0], op.params[1]), li);
      }
      pos = tpos[g.toff[gi] + coord];
    }
  }
  hd.qperm[x] = pos;
}

hipError_t launch_perms(const HeadDev* heads, int nheads, const OpDev* ops, Groups g, const int32_t* tpos,
                        int S, int max_slots, hipStream_t st) {
  (void)S;
  if (nheads <= 0 || max_slots <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_perms, dim3(nheads, (max_slots + 255) / 256), dim3(256), 0, st, heads, ops, g, tpos);
  return hipGetLastError();
}

// ------------------------------------------------ Q-Boundary Grid query order
constexpr int QO_PER = 16;                 // Grid slots per thread
constexpr int QO_CHUNK = 256 * QO_PER;     // Grid slots per workgroup

// Flags of this thread's QO_PER Grid slots (bit i: slot holds a position of
// the job's modality) and the positions themselves.
__device__ __forceinline__ uint32_t qo_flags(const QbOrderJob& j, const uint8_t* modpos, int S, int chunk,
                                             int (&pos)[QO_PER]) {
  const GridGeo geo = grid_geo(S, j.params[0], j.params[1]);
  const int x0 = chunk * QO_CHUNK + (int)threadIdx.x * QO_PER;
  uint32_t f = 0;
#pragma unroll
  for (int i = 0; i < QO_PER; ++i) {
    pos[i] = -1;
    if (x0 + i < S) {
      pos[i] = grid_coord(geo, x0 + i);
      if (modpos[pos[i]] == j.mod) f |= 1u << i;
    }
  }
  return f;
}

// exclusive prefix over the workgroup of v (256 threads); *total = sum
__device__ __forceinline__ int qo_scan(int v, int* sh, int* total) {
  const int t = threadIdx.x;
  sh[t] = v;
  __syncthreads();
  for (int d = 1; d < 256; d <<= 1) {
    const int a = t >= d ? sh[t - d] : 0;
    __syncthreads();
    sh[t] += a;
    __syncthreads();
  }
  const int inc = sh[t];
  *total = sh[255];
  __syncthreads();
  return inc - v;
}

__global__ __launch_bounds__(256) void k_qb_order_count(const QbOrderJob* jobs, const uint8_t* modpos, int S) {
  const QbOrderJob j = jobs[blockIdx.x];
  if (j.params[0] <= 1) return;            // dense fallback or stride 1: position order already written
  __shared__ int sh[256];
  int pos[QO_PER], total;
  const int n = __popc(qo_flags(j, modpos, S, blockIdx.y, pos));
  qo_scan(n, sh, &total);
  if (threadIdx.x == 0) j.cnt[blockIdx.y] = total;
}

__global__ void k_qb_order_offsets(const QbOrderJob* jobs, int nchunks) {
  const QbOrderJob j = jobs[blockIdx.x];
  if (j.params[0] <= 1 || threadIdx.x != 0) return;
  int run = 0;
  for (int c = 0; c < nchunks; ++c) {
    const int n = j.cnt[c];
    j.cnt[c] = run;
    run += n;
  }
}

__global__ __launch_bounds__(256) void k_qb_order_fill(const QbOrderJob* jobs, const uint8_t* modpos, int S) {
  const QbOrderJob j = jobs[blockIdx.x];
  if (j.params[0] <= 1) return;
  __shared__ int sh[256];
  int pos[QO_PER], total;
  const uint32_t f = qo_flags(j, modpos, S, blockIdx.y, pos);
  int at = j.cnt[blockIdx.y] + qo_scan(__popc(f), sh, &total);
#pragma unroll
  for (int i = 0; i < QO_PER; ++i)
    if (f >> i & 1u) j.qperm[at++] = pos[i];
}

hipError_t launch_qb_order(const QbOrderJob* jobs, int njobs, const uint8_t* modpos, int S, hipStream_t st) {
  if (njobs <= 0) return hipSuccess;
  const int nch = (S + QO_CHUNK - 1) / QO_CHUNK;
  hipLaunchKernelGGL(k_qb_order_count, dim3(njobs, nch), dim3(256), 0, st, jobs, modpos, S);
  hipLaunchKernelGGL(k_qb_order_offsets, dim3(njobs), dim3(64), 0, st, jobs, nch);
  hipLaunchKernelGGL(k_qb_order_fill, dim3(njobs, nch), dim3(256), 0, st, jobs, modpos, S);
  return hipGetLastError();
}

int qb_order_chunks(int S) { return (S + QO_CHUNK - 1) / QO_CHUNK; }

}  // namespace mmi
