// Modality layout and permutations.
//
// k_positions: the ascending position list T_m of every modality, all lists
//   packed into one pool (the modality type index i_m of Algorithms 2-3).
// k_perms: slot -> position maps of every head (Section 3.1, Algorithm 1
//   "permute Q, K, V"; Section 3.2, Algorithms 2-3 "permute by modality";
//   Appendix C.4): Grid heads group tokens by phase with the chosen phase
//   last; boundary heads concatenate the modality groups (each padded to a
//   multiple of 64 with -1), a 2D-Boundary group in Grid order when its
//   modality op is Grid. The kernels never move Q/K/V for this: attention
//   gathers rows through these maps.
#include "device.hpp"
#include "internal.hpp"

namespace mmi {

__global__ void k_positions(const Segment* segs, int nseg, const int32_t* toff_by_mod, int32_t* tpos,
                            int S) {
  const int p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= S) return;
  int lo = 0, hi = nseg - 1;     // last segment with pos <= p
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (segs[mid].pos <= p) lo = mid; else hi = mid - 1;
  }
  const Segment sg = segs[lo];
  tpos[toff_by_mod[sg.mod] + sg.loc + (p - sg.pos)] = p;
}

hipError_t launch_positions(const Segment* segs, int nseg, const int32_t* toff_by_mod, int32_t* tpos,
                              int S, hipStream_t st) {
  hipLaunchKernelGGL(k_positions, dim3((S + 255) / 256), dim3(256), 0, st, segs, nseg, toff_by_mod, tpos, S);
  return hipGetLastError();
}

__device__ __forceinline__ int group_of_slot(const Groups& g, int x) {
  for (int i = 0; i < g.n; ++i) {
    const int padded = (g.len[i] + B - 1) / B * B;
    if (x >= g.off[i] && x < g.off[i] + padded) return i;
  }
  return -1;
}

__global__ __launch_bounds__(256) void k_perms(const HeadDev* heads, const OpDev* ops, Groups g,
                                               const int32_t* tpos) {
  const HeadDev hd = heads[blockIdx.x];
  const int x = blockIdx.y * 256 + threadIdx.x;
  if (!hd.qperm || x >= hd.nbq * B) return;
  int pos = -1;
  if (hd.kind == MMI_HEAD_GLOBAL) {
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
  if (hd.kperm && hd.kperm != hd.qperm && x < hd.nbk * B) hd.kperm[x] = pos;
}

hipError_t launch_perms(const HeadDev* heads, int nheads, const OpDev* ops, Groups g, const int32_t* tpos,
                        int S, int max_slots, hipStream_t st) {
  (void)S;
  if (nheads <= 0 || max_slots <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_perms, dim3(nheads, (max_slots + 255) / 256), dim3(256), 0, st, heads, ops, g, tpos);
  return hipGetLastError();
}

}  // namespace mmi
