// Work statistics of a plan (not on the prefill path): the query-key pairs
// inside one head's selected blocks that the attention uses. Every pair of a
// selected block is computed (block semantics, "sparse loading, dense
// computation"); live query rows times live key rows with k <= q in original
// positions (all live pairs for a bidirectional head) are the useful part.
#include "device.hpp"
#include "internal.hpp"

namespace mmi {

// One workgroup per row group, one wave per member (lane = query row). A
// union entry without the member's mask bit holds 64 live keys at or below
// every query of the member; with it, the key positions are compared.
__global__ __launch_bounds__(256) void k_pair_count(const HeadDev* heads, int head, int R,
                                                    unsigned long long* out) {
  const HeadDev hd = heads[head];
  const int g = blockIdx.x;
  if (g >= hd.gp[1]) return;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  if (wave >= R) return;
  const int qb = group_row(g, wave, R, hd.gp[0]);
  if (qb >= hd.nbq) return;
  const int qslot = qb * B + lane;
  const int qpos = hd.qperm ? hd.qperm[qslot] : (qslot < hd.S ? qslot : -1);
  unsigned long long acc = 0;
  for (int e = hd.growptr[g]; e < hd.growptr[g + 1]; ++e) {
    const uint32_t en = (uint32_t)hd.gcol[e];
    if (!((en >> (16 + wave)) & 1u)) continue;
    const int kslot = (int)(en & 0xffffu) * B + lane;
    const int kpos = hd.kperm ? hd.kperm[kslot] : (kslot < hd.S ? kslot : -1);
    if (!((en >> (24 + wave)) & 1u)) {
      acc += qpos >= 0 ? B : 0;
      continue;
    }
    int c = 0;
    for (int x = 0; x < B; ++x) {
      const int k = __shfl(kpos, x, 64);
      c += (qpos >= 0 && k >= 0 && (!hd.causal || k <= qpos)) ? 1 : 0;
    }
    acc += c;
  }
  for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 64);
  if (lane == 0 && acc) atomicAdd(out, acc);
}

hipError_t launch_pair_count(const HeadDev* heads, int head, int R, int ngroups, unsigned long long* out,
                             hipStream_t st) {
  if (ngroups <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_pair_count, dim3(ngroups), dim3(256), 0, st, heads, head, R, out);
  return hipGetLastError();
}

}  // namespace mmi
