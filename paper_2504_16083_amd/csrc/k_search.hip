// Objective of the pattern search (Appendix A, Algorithm 4): per head and
// token class, the sum of squared differences between two attention
// outputs. One workgroup per head; each thread accumulates whole rows in
// fp64, then a fixed-order reduction (lane shuffles, then waves in order), so
// the result is bitwise reproducible.
#include "device.hpp"
#include "internal.hpp"

namespace mmi {

constexpr int SQ_THREADS = 1024;

__global__ __launch_bounds__(SQ_THREADS) void k_sqerr(const uint16_t* a, const uint16_t* b, int64_t ss, int64_t sh,
                                                      const uint8_t* cls, int n_class, int S, double* out) {
  const int h = blockIdx.x;
  double acc[MMI_MAX_MODALITIES];
#pragma unroll
  for (int c = 0; c < MMI_MAX_MODALITIES; ++c) acc[c] = 0.0;
  for (int x = threadIdx.x; x < S; x += SQ_THREADS) {
    const int c = cls[x];
    if (c >= n_class) continue;
    const uint16_t* ra = a + (int64_t)x * ss + (int64_t)h * sh;
    const uint16_t* rb = b + (int64_t)x * ss + (int64_t)h * sh;
    double rowd = 0.0;
    for (int d = 0; d < D; d += 8) {
      const bf16x8 va = load16(ra + d), vb = load16(rb + d);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float diff = (float)va[e] - (float)vb[e];
        rowd += (double)diff * (double)diff;
      }
    }
#pragma unroll
    for (int k = 0; k < MMI_MAX_MODALITIES; ++k)
      if (k == c) acc[k] += rowd;
  }
  __shared__ double part[SQ_THREADS / 64][MMI_MAX_MODALITIES];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int k = 0; k < MMI_MAX_MODALITIES; ++k) {
    double v = acc[k];
    for (int off = 32; off > 0; off >>= 1) v += __shfl_down(v, off, 64);
    if (lane == 0) part[wave][k] = v;
  }
  __syncthreads();
  if ((int)threadIdx.x < n_class) {
    double s = 0.0;
    for (int w = 0; w < SQ_THREADS / 64; ++w) s += part[w][threadIdx.x];
    out[(int64_t)h * n_class + threadIdx.x] = s;
  }
}

hipError_t launch_sqerr(const void* a, const void* b, int64_t ss, int64_t sh, const uint8_t* cls, int n_class,
                        int S, int H, double* out, hipStream_t st) {
  if (H <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_sqerr, dim3(H), dim3(SQ_THREADS), 0, st, reinterpret_cast<const uint16_t*>(a),
                     reinterpret_cast<const uint16_t*>(b), ss, sh, cls, n_class, S, out);
  return hipGetLastError();
}

}  // namespace mmi
