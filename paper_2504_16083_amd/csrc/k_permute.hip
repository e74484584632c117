// Explicit row permutation: the permute(Q), permute(K), permute(V) steps of
// Algorithms 1-3 done as a separate HBM pass (the attention kernel performs
// the same gathers inline; this pass exists for the identity tests and to
// measure what an explicit permutation costs). 16-byte vector copies, one
// wavefront per row segment of up to 1 KiB; perm = -1 writes a zero row.
#include "device.hpp"
#include "internal.hpp"

namespace mmi {

__global__ __launch_bounds__(256) void k_permute(const uint8_t* src, int64_t ss, uint8_t* dst, int64_t ds,
                                                 const int32_t* perm, int64_t n, int64_t row_bytes,
                                                 int inverse) {
  const int64_t vec_per_row = row_bytes / 16;
  const int64_t total = n * vec_per_row;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int64_t x = idx / vec_per_row, c = idx % vec_per_row;
    const int p = perm[x];
    if (!inverse) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (p >= 0) v = *reinterpret_cast<const uint4*>(src + p * ss + c * 16);
      *reinterpret_cast<uint4*>(dst + x * ds + c * 16) = v;
    } else if (p >= 0) {
      *reinterpret_cast<uint4*>(dst + p * ds + c * 16) = *reinterpret_cast<const uint4*>(src + x * ss + c * 16);
    }
  }
}

hipError_t launch_permute(const void* src, int64_t ss, void* dst, int64_t ds, const int32_t* perm, int64_t n,
                          int64_t row_bytes, int inverse, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const int64_t total = n * (row_bytes / 16);
  const int64_t blocks = (total + 255) / 256;
  const unsigned grid = (unsigned)(blocks < 65536 * 4 ? blocks : 65536 * 4);
  hipLaunchKernelGGL(k_permute, dim3(grid), dim3(256), 0, st, reinterpret_cast<const uint8_t*>(src), ss,
                     reinterpret_cast<uint8_t*>(dst), ds, perm, n, row_bytes, inverse);
  return hipGetLastError();
}

}  // namespace mmi
