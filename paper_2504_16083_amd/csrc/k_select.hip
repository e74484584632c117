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
// four 8-bit digit passes with an LDS histogram find the n-th largest value
// T; then one ordered pass keeps every score > T and the first
// (n - #greater) indices equal to T. All counts are integers, so the result
// does not depend on thread timing.
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
  for (int p = threadIdx.x; p < s; p += 256) {
    float acc = 0.0f;
    int n = 0;
    for (int x = p; x < jb.L_c; x += s) {
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

__global__ __launch_bounds__(TK_THREADS) void k_topk(const TopkJob* jobs) {
  const TopkJob jb = jobs[blockIdx.x];
  __shared__ int hist[256];
  __shared__ int sh_digit, sh_rem;
  __shared__ int scan[TK_THREADS];
  const int tid = threadIdx.x;
  if (jb.n <= 0) return;
  if (jb.n >= jb.L) {
    for (int i = tid; i < jb.L; i += TK_THREADS) jb.out[i] = i;
    return;
  }
  const uint32_t* bits = reinterpret_cast<const uint32_t*>(jb.x);
  uint32_t prefix = 0, mask = 0;
  int remaining = jb.n;
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int b = tid; b < 256; b += TK_THREADS) hist[b] = 0;
    __syncthreads();
    for (int i = tid; i < jb.L; i += TK_THREADS) {
      const uint32_t x = bits[i];
      if ((x & mask) == prefix) atomicAdd(&hist[(x >> shift) & 255], 1);
    }
    __syncthreads();
    if (tid == 0) {
      int cum = 0, d = 255;
      for (; d > 0; --d) {
        if (cum + hist[d] >= remaining) break;
        cum += hist[d];
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
  // prefix = bit pattern of the n-th largest value; `remaining` of its copies are taken
  const uint32_t T = prefix;
  int out_base = 0, eq_base = 0;
  for (int start = 0; start < jb.L; start += TK_THREADS) {
    const int i = start + tid;
    const uint32_t x = i < jb.L ? bits[i] : 0u;
    const int gt = (i < jb.L && x > T) ? 1 : 0;
    const int eq = (i < jb.L && x == T) ? 1 : 0;
    // inclusive scan of eq (bits 0-15) and gt (bits 16-31) packed
    scan[tid] = eq | (gt << 16);
    __syncthreads();
    for (int off = 1; off < TK_THREADS; off <<= 1) {
      const int v = tid >= off ? scan[tid - off] : 0;
      __syncthreads();
      scan[tid] += v;
      __syncthreads();
    }
    const int inc = scan[tid];
    const int eq_before = eq_base + (inc & 0xffff) - eq;
    const int take_eq = eq && eq_before < remaining;
    const int sel = gt | take_eq;
    // selected before i in this chunk: greater ones + equal ones taken since the chunk start
    const int gt_before = (inc >> 16) - gt;
    const int pos = out_base + gt_before + min(eq_before, remaining) - min(eq_base, remaining);
    if (sel && pos < jb.n) jb.out[pos] = i;
    const int tot = scan[TK_THREADS - 1];
    __syncthreads();
    out_base += (tot >> 16) + max(0, min(eq_base + (tot & 0xffff), remaining) - min(eq_base, remaining));
    eq_base += tot & 0xffff;
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
