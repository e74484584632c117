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
#include <algorithm>

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

// Top-n of a score array: a radix select of the n-th largest fp32 bit
// pattern T (scores are >= 0, so the bit patterns order like the values),
// 8 bits per pass from the top, then an order-preserving selection: every
// element above T and the first `remaining` copies of T by index, written in
// ascending index order. Each pass spreads a job over TK_CHUNKS workgroups:
// they add their chunk's digit histogram into the job's global one, and the
// last workgroup to finish (a counter) picks the digit for the next pass.
// Counts are integers, so the result does not depend on the order of the
// additions. Per-job scratch (int32, TK_SCR): prefix, mask, remaining, then
// a 256-bin histogram and a finish counter per pass, then the chunks' counts
// of elements above T and equal to T.
constexpr int TK_WG = 256;
constexpr int TK_WAVES = TK_WG / 64;
constexpr int TK_CHUNKS = 16;
constexpr int TK_PER = 8;          // consecutive elements per thread in the selection pass
constexpr int TK_HIST = 4;
constexpr int TK_DONE = TK_HIST + 4 * 256;
constexpr int TK_CNT = TK_DONE + 4;
constexpr int TK_SCR = TK_CNT + 2 * TK_CHUNKS;

__device__ __forceinline__ bool topk_trivial(const TopkJob& jb) { return jb.n <= 0 || jb.n >= jb.L; }

__device__ __forceinline__ void chunk_range(const TopkJob& jb, int c, int& lo, int& hi) {
  const int ch = (jb.L + TK_CHUNKS - 1) / TK_CHUNKS;
  lo = min(jb.L, c * ch);
  hi = min(jb.L, lo + ch);
}

__global__ __launch_bounds__(256) void k_topk_init(const TopkJob* jobs, int njobs, int32_t* scr) {
  const int j = blockIdx.x;
  if (j >= njobs) return;
  int32_t* sj = scr + (int64_t)j * TK_SCR;
  for (int x = threadIdx.x; x < TK_SCR; x += blockDim.x) sj[x] = x == 2 ? jobs[j].n : 0;
}

__global__ __launch_bounds__(TK_WG) void k_topk_hist(const TopkJob* jobs, int32_t* scr, int pass) {
  const TopkJob jb = jobs[blockIdx.x];
  if (topk_trivial(jb)) return;
  int32_t* sj = scr + (int64_t)blockIdx.x * TK_SCR;
  __shared__ int hist[TK_WAVES][256];
  __shared__ int sh_last;
  const int tid = threadIdx.x, wave = tid >> 6;
  const int shift = 24 - 8 * pass;
  const uint32_t prefix = (uint32_t)sj[0], mask = (uint32_t)sj[1];
  for (int b = tid; b < TK_WAVES * 256; b += TK_WG) (&hist[0][0])[b] = 0;
  __syncthreads();
  int lo, hi;
  chunk_range(jb, blockIdx.y, lo, hi);
  const uint32_t* bits = reinterpret_cast<const uint32_t*>(jb.x);
  constexpr int HU = 8;            // loads in flight per thread
  for (int i0 = lo + tid; i0 < hi; i0 += TK_WG * HU) {
    uint32_t xs[HU];
#pragma unroll
    for (int u = 0; u < HU; ++u) xs[u] = i0 + u * TK_WG < hi ? bits[i0 + u * TK_WG] : 0u;
#pragma unroll
    for (int u = 0; u < HU; ++u)
      if (i0 + u * TK_WG < hi && (xs[u] & mask) == prefix) atomicAdd(&hist[wave][(xs[u] >> shift) & 255], 1);
  }
  __syncthreads();
  int32_t* gh = sj + TK_HIST + pass * 256;
  for (int b = tid; b < 256; b += TK_WG) {
    int c = 0;
    for (int w = 0; w < TK_WAVES; ++w) c += hist[w][b];
    if (c) atomicAdd(&gh[b], c);
  }
  __threadfence();
  __syncthreads();
  if (tid == 0) sh_last = atomicAdd(&sj[TK_DONE + pass], 1) == TK_CHUNKS - 1;
  __syncthreads();
  if (!sh_last) return;
  __threadfence();
  if (tid == 0) {                  // the digit of the n-th largest among the candidates
    const int remaining = sj[2];
    int cum = 0, d = 255;
    for (; d > 0; --d) {
      const int h = __atomic_load_n(&gh[d], __ATOMIC_RELAXED);
      if (cum + h >= remaining) break;
      cum += h;
    }
    sj[0] = (int32_t)(prefix | ((uint32_t)d << shift));
    sj[1] = (int32_t)(mask | (255u << shift));
    sj[2] = remaining - cum;
  }
}

// Elements above T and equal to T in each chunk.
__global__ __launch_bounds__(TK_WG) void k_topk_count(const TopkJob* jobs, int32_t* scr) {
  const TopkJob jb = jobs[blockIdx.x];
  if (topk_trivial(jb)) return;
  int32_t* sj = scr + (int64_t)blockIdx.x * TK_SCR;
  __shared__ int wg[TK_WAVES], we[TK_WAVES];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint32_t T = (uint32_t)sj[0];
  int lo, hi;
  chunk_range(jb, blockIdx.y, lo, hi);
  const uint32_t* bits = reinterpret_cast<const uint32_t*>(jb.x);
  int g = 0, e = 0;
  for (int i = lo + tid; i < hi; i += TK_WG) {
    const uint32_t x = bits[i];
    g += x > T ? 1 : 0;
    e += x == T ? 1 : 0;
  }
  for (int off = 32; off > 0; off >>= 1) { g += __shfl_xor(g, off, 64); e += __shfl_xor(e, off, 64); }
  if (lane == 0) { wg[wave] = g; we[wave] = e; }
  __syncthreads();
  if (tid == 0) {
    int tg = 0, te = 0;
    for (int w = 0; w < TK_WAVES; ++w) { tg += wg[w]; te += we[w]; }
    sj[TK_CNT + blockIdx.y] = tg;
    sj[TK_CNT + TK_CHUNKS + blockIdx.y] = te;
  }
}

// Output slot of a selected element i = (elements above T before i) +
// min(copies of T before i, remaining): ascending indices.
__global__ __launch_bounds__(TK_WG) void k_topk_write(const TopkJob* jobs, const int32_t* scr) {
  const TopkJob jb = jobs[blockIdx.x];
  int lo, hi;
  chunk_range(jb, blockIdx.y, lo, hi);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (jb.n <= 0) return;
  if (jb.n >= jb.L) {
    for (int i = lo + tid; i < hi; i += TK_WG) jb.out[i] = i;
    return;
  }
  const int32_t* sj = scr + (int64_t)blockIdx.x * TK_SCR;
  __shared__ int wgt[TK_WAVES], weq[TK_WAVES];
  const uint32_t T = (uint32_t)sj[0];
  const int remaining = sj[2];
  int gt_base = 0, eq_base = 0;    // counts of the chunks before this one
  for (int c = 0; c < (int)blockIdx.y; ++c) {
    gt_base += sj[TK_CNT + c];
    eq_base += sj[TK_CNT + TK_CHUNKS + c];
  }
  const uint32_t* bits = reinterpret_cast<const uint32_t*>(jb.x);
  for (int start = lo; start < hi; start += TK_WG * TK_PER) {
    const int i0 = start + tid * TK_PER;
    uint32_t xs[TK_PER];
    int cg = 0, ce = 0;
#pragma unroll
    for (int e = 0; e < TK_PER; ++e) {
      xs[e] = i0 + e < hi ? bits[i0 + e] : 0u;
      cg += (i0 + e < hi && xs[e] > T) ? 1 : 0;
      ce += (i0 + e < hi && xs[e] == T) ? 1 : 0;
    }
    int sg = cg, se = ce;          // inclusive scan over the wave's lanes
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
    __syncthreads();               // wgt/weq are rewritten by the next stretch
    int g_before = gt_base + pg + sg - cg, e_before = eq_base + pe + se - ce;
#pragma unroll
    for (int e = 0; e < TK_PER; ++e) {
      if (i0 + e < hi) {
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

size_t topk_scratch_ints(int njobs) { return (size_t)std::max(njobs, 1) * TK_SCR; }

hipError_t launch_topk(const TopkJob* jobs, int njobs, int32_t* scr, hipStream_t st) {
  if (njobs <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_topk_init, dim3(njobs), dim3(256), 0, st, jobs, njobs, scr);
  for (int pass = 0; pass < 4; ++pass)
    hipLaunchKernelGGL(k_topk_hist, dim3(njobs, TK_CHUNKS), dim3(TK_WG), 0, st, jobs, scr, pass);
  hipLaunchKernelGGL(k_topk_count, dim3(njobs, TK_CHUNKS), dim3(TK_WG), 0, st, jobs, scr);
  hipLaunchKernelGGL(k_topk_write, dim3(njobs, TK_CHUNKS), dim3(TK_WG), 0, st, jobs, scr);
  return hipGetLastError();
}

}  // namespace mmi
