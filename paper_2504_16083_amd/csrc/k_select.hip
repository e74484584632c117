// Discrete choices taken from the estimate.
//
// Grid stride/phase search (Algorithm 1, "Online search grid stride and
// phase"): for each candidate stride s the column scores v are folded with
// period s, c_s[p] = mean_{t: t s + p < L_c} v[t s + p]; score_s = max_p c_s[p]
// with the smallest maximising phase. k_grid_fold computes one stride per
// workgroup (each thread sums its phases in ascending t: fixed order);
// k_grid_pick scans the strides in ascending order and keeps a later stride
// only if its score exceeds best * 1.02 (fp32 product), then publishes
// {sigma, phase} (sigma 0 = no stride with two visible periods: dense).
//
// Vertical-Slash top-k (Appendix C.3): the n largest scores of [0, L),
// ties to the smaller index, as an ascending index list. Radix select on the
// fp32 bit patterns (scores are non-negative, so bits order like values):
// four 8-bit digit passes with per-wave LDS histograms find the n-th largest
// value T; then one ordered pass (wave prefix sums, eight elements per
// thread) keeps every score > T and the first (n - #greater) indices equal
// to T. All counts are integers, so the result does not depend on thread
// timing.
#include "device.hpp"
#include "internal.hpp"

namespace mmi {

__global__ __launch_bounds__(256) void k_grid_fold(const GridJob* jobs) {
  const GridJob jb = jobs[blockIdx.x];
  const int y = blockIdx.y;
  const int s = jb.lo + y;
  if (jb.hi < jb.lo || s > jb.hi) return;
  __shared__ float bv[256];
  __shared__ int bp[256];
  float best = -1.0f;
  int bestp = 0x7fffffff;
  constexpr int U = 16;   // loads in flight per thread; the sum keeps ascending t order
  for (int p = threadIdx.x; p < s; p += 256) {
    float acc = 0.0f;
    int n = 0;
    int x = p;
    for (; x + (U - 1) * s < jb.L_c; x += U * s) {
      float t[U];
#pragma unroll
      for (int u = 0; u < U; ++u) t[u] = jb.v[x + u * s];
#pragma unroll
      for (int u = 0; u < U; ++u) acc += t[u];
      n += U;
    }
    for (; x < jb.L_c; x += s) {
      acc += jb.v[x];
      ++n;
    }
    const float c = acc / (float)n;
    jb.fold[(int64_t)y * FOLD_W + p] = c;
    if (c > best) { best = c; bestp = p; }     // p ascending per thread: keeps the smallest
  }
  bv[threadIdx.x] = best;
  bp[threadIdx.x] = bestp;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) {
      const float ov = bv[threadIdx.x + w];
      const int op = bp[threadIdx.x + w];
      if (ov > bv[threadIdx.x] || (ov == bv[threadIdx.x] && op < bp[threadIdx.x])) {
        bv[threadIdx.x] = ov;
        bp[threadIdx.x] = op;
      }
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    jb.score[y] = bv[0];
    jb.pick[y] = bp[0];
  }
}

__global__ void k_grid_pick(const GridJob* jobs, int njobs) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= njobs) return;
  const GridJob jb = jobs[j];
  float b = 0.0f;
  int sig = 0, ph = 0;
  const float one_eps = 1.02f;
  for (int s = jb.lo; s <= jb.hi; ++s) {
    const float sc = jb.score[s - jb.lo];
    const float thr = b * one_eps;
    if (sc > thr) {
      b = sc;
      sig = s;
      ph = jb.pick[s - jb.lo];
    }
  }
  jb.params[0] = sig;
  jb.params[1] = ph;
  jb.params[2] = jb.L_c;
  jb.params[3] = jb.nrows;
}

constexpr int TK_THREADS = 1024;
constexpr int TK_WAVES = TK_THREADS / 64;
constexpr int TK_PER = 8;          // consecutive elements per thread in the selection pass

// Radix select of the n-th largest fp32 bit pattern (scores are >= 0, so the
// bit patterns order like the values), then an order-preserving selection:
// every element above it, and the first `remaining` copies of it by index.
__global__ __launch_bounds__(TK_THREADS) void k_topk(const TopkJob* jobs) {
  const TopkJob jb = jobs[blockIdx.x];
  __shared__ int hist[TK_WAVES][256];
  __shared__ int sh_digit, sh_rem;
  __shared__ int wgt[TK_WAVES], weq[TK_WAVES];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (jb.n <= 0) return;
  if (jb.n >= jb.L) {
    for (int i = tid; i < jb.L; i += TK_THREADS) jb.out[i] = i;
    return;
  }
  const uint32_t* bits = reinterpret_cast<const uint32_t*>(jb.x);
  uint32_t prefix = 0, mask = 0;
  int remaining = jb.n;
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int b = tid; b < TK_WAVES * 256; b += TK_THREADS) (&hist[0][0])[b] = 0;
    __syncthreads();
    // one histogram per wave (fewer collisions); eight loads in flight per
    // thread (the counts do not depend on the order they are added in)
    constexpr int HU = 8;
    for (int i0 = tid; i0 < jb.L; i0 += TK_THREADS * HU) {
      uint32_t xs[HU];
#pragma unroll
      for (int u = 0; u < HU; ++u) xs[u] = i0 + u * TK_THREADS < jb.L ? bits[i0 + u * TK_THREADS] : 0u;
#pragma unroll
      for (int u = 0; u < HU; ++u)
        if (i0 + u * TK_THREADS < jb.L && (xs[u] & mask) == prefix) atomicAdd(&hist[wave][(xs[u] >> shift) & 255], 1);
    }
    __syncthreads();
    for (int b = tid; b < 256; b += TK_THREADS) {
      int c = 0;
      for (int w = 0; w < TK_WAVES; ++w) c += hist[w][b];
      hist[0][b] = c;
    }
    __syncthreads();
    if (tid == 0) {
      int cum = 0, d = 255;
      for (; d > 0; --d) {
        if (cum + hist[0][d] >= remaining) break;
        cum += hist[0][d];
      }
      sh_digit = d;
      sh_rem = remaining - cum;
    }
    __syncthreads();
    prefix |= (uint32_t)sh_digit << shift;
    mask |= 255u << shift;
    remaining = sh_rem;
    __syncthreads();
  }
  // prefix = bit pattern T of the n-th largest value; `remaining` of its copies
  // are taken. Output slot of a selected element i = (elements above T before
  // i) + min(copies of T before i, remaining): ascending indices.
  const uint32_t T = prefix;
  int gt_base = 0, eq_base = 0;          // counts before the current chunk
  uint32_t nx[TK_PER];                   // the next chunk, loading while this one is scanned
#pragma unroll
  for (int e = 0; e < TK_PER; ++e) nx[e] = tid * TK_PER + e < jb.L ? bits[tid * TK_PER + e] : 0u;
  for (int start = 0; start < jb.L; start += TK_THREADS * TK_PER) {
    const int i0 = start + tid * TK_PER;
    uint32_t xs[TK_PER];
    int cg = 0, ce = 0;
#pragma unroll
    for (int e = 0; e < TK_PER; ++e) {
      xs[e] = nx[e];
      cg += (i0 + e < jb.L && xs[e] > T) ? 1 : 0;
      ce += (i0 + e < jb.L && xs[e] == T) ? 1 : 0;
    }
    const int n0 = i0 + TK_THREADS * TK_PER;
#pragma unroll
    for (int e = 0; e < TK_PER; ++e) nx[e] = n0 + e < jb.L ? bits[n0 + e] : 0u;
    int sg = cg, se = ce;                // inclusive scan over the wave's lanes
    for (int off = 1; off < 64; off <<= 1) {
      const int a = __shfl_up(sg, off, 64), b2 = __shfl_up(se, off, 64);
      if (lane >= off) { sg += a; se += b2; }
    }
    if (lane == 63) { wgt[wave] = sg; weq[wave] = se; }
    __syncthreads();
    int pg = 0, pe = 0, tg = 0, te = 0;
    for (int w = 0; w < TK_WAVES; ++w) {
      if (w < wave) { pg += wgt[w]; pe += weq[w]; }
      tg += wgt[w];
      te += weq[w];
    }
    __syncthreads();                     // wgt/weq are rewritten by the next chunk
    int g_before = gt_base + pg + sg - cg, e_before = eq_base + pe + se - ce;
#pragma unroll
    for (int e = 0; e < TK_PER; ++e) {
      if (i0 + e < jb.L) {
        const bool gt = xs[e] > T, eq = xs[e] == T;
        if (gt || (eq && e_before < remaining)) {
          const int pos = g_before + min(e_before, remaining);
          if (pos < jb.n) jb.out[pos] = i0 + e;
        }
        g_before += gt ? 1 : 0;
        e_before += eq ? 1 : 0;
      }
    }
    gt_base += tg;
    eq_base += te;
  }
}

hipError_t launch_grid_search(const GridJob* jobs, int njobs, int max_cands, hipStream_t st) {
  if (njobs <= 0) return hipSuccess;
  if (max_cands > 0) hipLaunchKernelGGL(k_grid_fold, dim3(njobs, max_cands), dim3(256), 0, st, jobs);
  hipLaunchKernelGGL(k_grid_pick, dim3((njobs + 63) / 64), dim3(64), 0, st, jobs, njobs);
  return hipGetLastError();
}

hipError_t launch_topk(const TopkJob* jobs, int njobs, hipStream_t st) {
  if (njobs <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_topk, dim3(njobs), dim3(TK_THREADS), 0, st, jobs);
  return hipGetLastError();
}

}  // namespace mmi
