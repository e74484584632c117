// Device helpers shared by the gfx950 kernels: vector types, MFMA wrappers,
// bf16 packing and the closed-form Grid permutation geometry.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mmi {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;

constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;
constexpr float NEG_BIG = -1.0e30f;   // finite "minus infinity" for running maxima

// C += A * B with A: 32x16 (lane r = l%32 holds row r, k-half l/32),
// B: 16x32 (lane c = l%32 holds column c), C: 32x32 fp32 where lane
// (c = l%32, h = l/32) holds C[8i + 4h + j][c] in element 4i + j.
__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 load16(const void* p) {
  return *reinterpret_cast<const bf16x8*>(p);
}

__device__ __forceinline__ bf16x8 zero8() {
  bf16x8 z;
#pragma unroll
  for (int e = 0; e < 8; ++e) z[e] = (__bf16)0.0f;
  return z;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

// Query block held by member r of row group g (R members, row stride rho).
__host__ __device__ inline int group_row(int g, int r, int R, int rho) {
  return (g / rho) * (R * rho) + (g % rho) + r * rho;
}

__host__ __device__ inline int groups_for(int nbq, int R, int rho) {
  return (nbq + R * rho - 1) / (R * rho) * rho;
}

// ------------------------------------------------------------------ Grid geometry
// Tokens with coordinates [0, L) are grouped by phase (coordinate mod s); the
// groups are ordered p+1, p+2, ..., p (mod s) and packed without padding.
// A phase f holds A + (f < R) tokens where L = A*s + R.
struct GridGeo {
  int L, s, p, A, R;
};

__host__ __device__ inline GridGeo grid_geo(int L, int s, int p) {
  GridGeo g;
  g.L = L; g.s = s; g.p = p; g.A = L / s; g.R = L % s;
  return g;
}

// number of y in [0, x) with (y mod s) < R
__host__ __device__ inline int grid_f(int x, int s, int R) { return (x / s) * R + min(x % s, R); }

// first slot of the group of rank rho (rho in [0, s])
__host__ __device__ inline int grid_g0_rank(const GridGeo& g, int rho) {
  return rho * g.A + grid_f(g.p + 1 + rho, g.s, g.R) - grid_f(g.p + 1, g.s, g.R);
}

__host__ __device__ inline int grid_rank(const GridGeo& g, int phase) {
  int r = (phase - g.p - 1) % g.s;
  return r < 0 ? r + g.s : r;
}

__host__ __device__ inline int grid_g0(const GridGeo& g, int phase) {
  return grid_g0_rank(g, grid_rank(g, phase));
}

// coordinate held by slot x in [0, L)
__host__ __device__ inline int grid_coord(const GridGeo& g, int x) {
  int lo = 0, hi = g.s - 1;      // largest rank with g0_rank(rank) <= x
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (grid_g0_rank(g, mid) <= x) lo = mid; else hi = mid - 1;
  }
  int phase = (g.p + 1 + lo) % g.s;
  return (x - grid_g0_rank(g, lo)) * g.s + phase;
}

// slot holding coordinate c
__host__ __device__ inline int grid_slot(const GridGeo& g, int c) {
  return grid_g0(g, c % g.s) + c / g.s;
}

}  // namespace mmi
