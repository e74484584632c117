// Block-sparse causal attention over permuted 64x64 blocks (Algorithms 5-7:
// the Grid, Q-Boundary and 2D-Boundary FlashAttention kernels are one
// kernel here, because the permutation and the selected key blocks are data:
// qperm / kperm say which token each slot holds, the block index says which
// key blocks each query block visits).
//
// One work item = a row group of R consecutive permuted query blocks and a
// contiguous range of the union of their key-block lists; each union entry
// carries one flag per query block. The workgroup has 2R waves; waves 2r and
// 2r+1 own the 64 rows of query block r (32 rows each). Every key block of
// the range is loaded from HBM/L2 once into LDS and used by all query blocks
// that selected it, so each byte of K/V feeds up to 64R rows. Per key block
// and active wave:
//   S^T (64 keys x 32 queries) = K Q^T         16 MFMA 32x32x16 bf16
//   mask by original positions (k <= q) where the block reaches past the
//   wave's first query, online softmax in fp32 (log2 domain)
//   O^T (128 x 32) += V^T P^T                  16 MFMA 32x32x16 bf16
// Computing S^T rather than S puts one query per lane, so the row max/sum
// needs one cross-lane exchange and the accumulator doubles as the P operand
// of the PV product (the key order inside the contraction is permuted the
// same way in V^T). K is staged row-major and V transposed in LDS; the next
// block's K/V are fetched into registers while the current one is computed.
// Gathered rows are 256-byte contiguous loads, 16 lanes per row.
#include "device.hpp"
#include "internal.hpp"

namespace mmi {

constexpr int KPITCH = 136;   // bf16 per K row in LDS: 128 + 8 pad (272 B)
constexpr int VPITCH = 68;    // bf16 per V^T row in LDS: 64 + 4 pad (136 B)

// V^T rows hold 16 groups of 4 keys; the group index is XOR-swizzled with
// bits of the row so both the transposing writes and the operand reads
// spread over the 64 LDS banks.
__device__ __forceinline__ int vt_off(int d, int kgroup) { return d * VPITCH + ((kgroup ^ ((d >> 3) & 7)) << 2); }

struct __align__(16) AttnSmem {
  uint16_t k[B * KPITCH];
  uint16_t vt[D * VPITCH];
  int32_t kpos[B];
};

__device__ __forceinline__ int slot_pos(const int32_t* perm, int slot, int S) {
  return perm ? perm[slot] : (slot < S ? slot : -1);
}

template <int R>
struct Tile {
  static constexpr int NT = 128 * R;           // threads
  static constexpr int KL = 1024 / NT;         // 16-byte K chunks loaded per thread
  static constexpr int VG = KL >= 4 ? 4 : KL;  // keys per V unit (same 16-byte chunk of VG rows)
  static constexpr int VU = KL / VG;           // V units per thread
};

template <int R>
struct BlockRegs {
  bf16x8 k[Tile<R>::KL];
  bf16x8 v[Tile<R>::VU * Tile<R>::VG];
};

template <int R>
__device__ __forceinline__ void fetch_block(BlockRegs<R>& r, const AttnArgs& a, const HeadDev& hd, int jblk,
                                            int tid) {
  using T = Tile<R>;
  const uint16_t* kb = reinterpret_cast<const uint16_t*>(a.k.p) + (int64_t)hd.kvh * a.k.sh;
  const uint16_t* vb = reinterpret_cast<const uint16_t*>(a.v.p) + (int64_t)hd.kvh * a.v.sh;
  const int base = jblk * B;
#pragma unroll
  for (int it = 0; it < T::KL; ++it) {
    const int u = tid + it * T::NT;
    const int key = u >> 4, chunk = u & 15;
    const int kp = slot_pos(hd.kperm, base + key, a.S);
    r.k[it] = kp >= 0 ? load16(kb + (int64_t)kp * a.k.ss + chunk * 8) : zero8();
  }
#pragma unroll
  for (int it = 0; it < T::VU; ++it) {
    const int u = tid + it * T::NT;
    const int kg = u >> 4, chunk = u & 15;
#pragma unroll
    for (int rr = 0; rr < T::VG; ++rr) {
      const int kp = slot_pos(hd.kperm, base + kg * T::VG + rr, a.S);
      r.v[it * T::VG + rr] = kp >= 0 ? load16(vb + (int64_t)kp * a.v.ss + chunk * 8) : zero8();
    }
  }
}

template <int R>
__device__ __forceinline__ void stage_block(AttnSmem& sm, const BlockRegs<R>& r, const HeadDev& hd, int jblk,
                                            int S, int tid) {
  using T = Tile<R>;
#pragma unroll
  for (int it = 0; it < T::KL; ++it) {
    const int u = tid + it * T::NT;
    *reinterpret_cast<bf16x8*>(&sm.k[(u >> 4) * KPITCH + (u & 15) * 8]) = r.k[it];
  }
#pragma unroll
  for (int it = 0; it < T::VU; ++it) {
    const int u = tid + it * T::NT;
    const int kg = u >> 4, chunk = u & 15;
    const int key0 = kg * T::VG;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      uint16_t* dst = &sm.vt[vt_off(chunk * 8 + e, key0 >> 2) + (key0 & 3)];
      if constexpr (T::VG == 4) {
        bf16x4 t;
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) t[rr] = r.v[it * 4 + rr][e];
        *reinterpret_cast<bf16x4*>(dst) = t;
      } else {
        typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2;
        bf16x2 t;
        t[0] = r.v[it * 2][e];
        t[1] = r.v[it * 2 + 1][e];
        *reinterpret_cast<bf16x2*>(dst) = t;
      }
    }
  }
  if (tid < B) sm.kpos[tid] = slot_pos(hd.kperm, jblk * B + tid, S);
}

// Largest key position of key block j, or INT_BIG if the block holds padding.
__device__ __forceinline__ int block_kmax(const HeadDev& hd, int j, int S) {
  if (hd.kmaxpos) return hd.kmaxpos[j];
  const int last = j * B + B - 1;
  return last < S ? last : INT_BIG;
}

// Work-item order: hardware hands consecutive workgroups to the 8 XCDs in
// turn. Runs of XCD_RUN consecutive items go to one XCD, and the runs are
// interleaved across XCDs, so neighbouring row groups (which share key
// blocks) meet in one L2 while heavy and light heads stay spread out.
constexpr int XCD_RUN = 16;

__device__ __forceinline__ int64_t item_of_block(int64_t b) {
  const int64_t xcd = b & 7, k = b >> 3;
  return (k / XCD_RUN) * (8 * XCD_RUN) + xcd * XCD_RUN + (k % XCD_RUN);
}

template <int R>
__global__ __launch_bounds__(128 * R) __attribute__((amdgpu_waves_per_eu(2))) void k_attention(AttnArgs a) {
  __shared__ AttnSmem sm;
  const int64_t it = item_of_block(blockIdx.x);
  if (it >= a.nitems) return;
  const WorkItem w = a.items[it];
  const HeadDev hd = a.heads[w.head];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int c = lane & 31, h = lane >> 5;
  const int rb = wave >> 1;                        // member of the group owned by this wave
  const int qblk = group_row(w.group, rb, R, hd.gp[0]);
  const int qpos = qblk < hd.nbq ? slot_pos(hd.qperm, qblk * B + (wave & 1) * 32 + c, a.S) : -1;
  int qmin = qpos >= 0 ? qpos : INT_BIG;      // smallest valid query position of the wave
#pragma unroll
  for (int off = 1; off < 32; off <<= 1) qmin = min(qmin, __shfl_xor(qmin, off));
  bf16x8 qr[8];
  {
    const uint16_t* qb = reinterpret_cast<const uint16_t*>(a.q.p) + (int64_t)w.head * a.q.sh;
    const uint16_t* row = qb + (int64_t)max(qpos, 0) * a.q.ss + h * 64;
#pragma unroll
    for (int s = 0; s < 8; ++s) qr[s] = qpos >= 0 ? load16(row + 8 * s) : zero8();
  }

  f32x16 o[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[dt][e] = 0.0f;
  float m = NEG_BIG, l = 0.0f;
  const float sc = 0.08838834764831845f * LOG2E;   // sqrt(1/128) * log2(e)

  BlockRegs<R> regs;
  fetch_block<R>(regs, a, hd, hd.gcol[w.e0] & 0xffff, tid);
  for (int e = w.e0; e < w.e1; ++e) {
    const int ent = hd.gcol[e];
    const int jcur = ent & 0xffff;
    stage_block<R>(sm, regs, hd, jcur, a.S, tid);
    __syncthreads();
    if (e + 1 < w.e1) fetch_block<R>(regs, a, hd, hd.gcol[e + 1] & 0xffff, tid);
    if ((ent >> (16 + rb)) & 1) {          // this wave's query block selected key block jcur
      const bool need_mask = block_kmax(hd, jcur, a.S) > qmin;   // wave-uniform
      f32x16 s[2];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int x = 0; x < 16; ++x) s[kt][x] = 0.0f;
#pragma unroll
      for (int st = 0; st < 8; ++st) {
        const bf16x8 k0 = *reinterpret_cast<const bf16x8*>(&sm.k[c * KPITCH + h * 64 + st * 8]);
        const bf16x8 k1 = *reinterpret_cast<const bf16x8*>(&sm.k[(32 + c) * KPITCH + h * 64 + st * 8]);
        s[0] = mfma32(k0, qr[st], s[0]);
        s[1] = mfma32(k1, qr[st], s[1]);
      }
      if (need_mask) {
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int4 kp = *reinterpret_cast<const int4*>(&sm.kpos[kt * 32 + 8 * i + 4 * h]);
            if (kp.x < 0 || kp.x > qpos) s[kt][4 * i + 0] = -INFINITY;
            if (kp.y < 0 || kp.y > qpos) s[kt][4 * i + 1] = -INFINITY;
            if (kp.z < 0 || kp.z > qpos) s[kt][4 * i + 2] = -INFINITY;
            if (kp.w < 0 || kp.w > qpos) s[kt][4 * i + 3] = -INFINITY;
          }
      }
      float mx = NEG_BIG;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int x = 0; x < 16; ++x) mx = fmaxf(mx, s[kt][x]);
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m, mx * sc);     // scale > 0: max commutes with it
      float rs = 0.0f;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int x = 0; x < 16; ++x) {
          const float p = fast_exp2(fmaf(s[kt][x], sc, -m_new));
          s[kt][x] = p;
          rs += p;
        }
      rs += __shfl_xor(rs, 32);
      if (__any(m_new != m)) {   // rescale only when some row's running max moved
        const float alpha = fast_exp2(m - m_new);
        l *= alpha;
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
#pragma unroll
          for (int x = 0; x < 16; ++x) o[dt][x] *= alpha;
      }
      l += rs;
      m = m_new;
#pragma unroll
      for (int st = 0; st < 4; ++st) {
        const int kt = st >> 1, half = st & 1;
        bf16x8 pb;
#pragma unroll
        for (int x = 0; x < 8; ++x) pb[x] = (__bf16)s[kt][4 * (2 * half + (x >> 2)) + (x & 3)];
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) {
          const int d = 32 * dt + c, g = 8 * kt + 4 * half + h;
          const bf16x4 lo = *reinterpret_cast<const bf16x4*>(&sm.vt[vt_off(d, g)]);
          const bf16x4 hi = *reinterpret_cast<const bf16x4*>(&sm.vt[vt_off(d, g + 2)]);
          bf16x8 va;
#pragma unroll
          for (int x = 0; x < 4; ++x) { va[x] = lo[x]; va[4 + x] = hi[x]; }
          o[dt] = mfma32(va, pb, o[dt]);
        }
      }
    }
    __syncthreads();
  }

  if (w.part < 0) {
    if (qpos >= 0) {
      const float inv = 1.0f / l;
      uint16_t* orow = reinterpret_cast<uint16_t*>(a.o) + (int64_t)qpos * a.o_ss + (int64_t)w.head * a.o_sh;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          bf16x4 t;
#pragma unroll
          for (int j = 0; j < 4; ++j) t[j] = (__bf16)(o[dt][4 * i + j] * inv);
          *reinterpret_cast<bf16x4*>(orow + 32 * dt + 8 * i + 4 * h) = t;
        }
      if (h == 0 && a.lse) a.lse[(int64_t)w.head * a.S + qpos] = (m + fast_log2(l)) * LN2;
    }
  } else {
    const int row = wave * 32 + c;             // row of the group, 0 .. 64R-1
    float* po = a.part_o + ((int64_t)w.part * (B * R) + row) * D;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float4 t = make_float4(o[dt][4 * i], o[dt][4 * i + 1], o[dt][4 * i + 2], o[dt][4 * i + 3]);
        *reinterpret_cast<float4*>(po + 32 * dt + 8 * i + 4 * h) = t;
      }
    if (h == 0) {
      float* ml = a.part_ml + ((int64_t)w.part * (B * R) + row) * 2;
      ml[0] = m;
      ml[1] = l;
    }
  }
}

// Merge the (O, m, l) partials of a split row group in a fixed order:
// M = max m_p, L = sum l_p 2^(m_p - M), O = sum O_p 2^(m_p - M) / L.
// Workgroup = the 64 rows of query block blockIdx.y of the group, 4 threads per row.
__global__ __launch_bounds__(256) void k_combine(AttnArgs a, const SplitRow* splits) {
  const SplitRow sr = splits[blockIdx.x];
  const HeadDev hd = a.heads[sr.head];
  const int rb = blockIdx.y;
  const int qblk = group_row(sr.group, rb, a.R, hd.gp[0]);
  if (qblk >= hd.nbq) return;
  const int row = rb * B + (threadIdx.x >> 2), quarter = threadIdx.x & 3;
  const int qpos = slot_pos(hd.qperm, qblk * B + (threadIdx.x >> 2), a.S);
  if (qpos < 0) return;
  const int64_t stride = (int64_t)B * a.R;
  float M = NEG_BIG;
  for (int p = 0; p < sr.nparts; ++p) M = fmaxf(M, a.part_ml[((int64_t)(sr.part0 + p) * stride + row) * 2]);
  float acc[32];
#pragma unroll
  for (int x = 0; x < 32; ++x) acc[x] = 0.0f;
  float L = 0.0f;
  for (int p = 0; p < sr.nparts; ++p) {
    const int64_t pr = (int64_t)(sr.part0 + p) * stride + row;
    const float wgt = fast_exp2(a.part_ml[pr * 2] - M);
    L += a.part_ml[pr * 2 + 1] * wgt;
    const float4* src = reinterpret_cast<const float4*>(a.part_o + pr * D + quarter * 32);
#pragma unroll
    for (int x = 0; x < 8; ++x) {
      const float4 t = src[x];
      acc[4 * x] += t.x * wgt; acc[4 * x + 1] += t.y * wgt;
      acc[4 * x + 2] += t.z * wgt; acc[4 * x + 3] += t.w * wgt;
    }
  }
  const float inv = 1.0f / L;
  uint16_t* orow = reinterpret_cast<uint16_t*>(a.o) + (int64_t)qpos * a.o_ss + (int64_t)sr.head * a.o_sh + quarter * 32;
#pragma unroll
  for (int x = 0; x < 4; ++x) {
    bf16x8 t;
#pragma unroll
    for (int e = 0; e < 8; ++e) t[e] = (__bf16)(acc[8 * x + e] * inv);
    *reinterpret_cast<bf16x8*>(orow + 8 * x) = t;
  }
  if (quarter == 0 && a.lse) a.lse[(int64_t)sr.head * a.S + qpos] = (M + fast_log2(L)) * LN2;
}

hipError_t launch_attention(const AttnArgs& a, hipStream_t st) {
  if (a.nitems <= 0) return hipSuccess;
  const int64_t run = 8 * XCD_RUN;
  const int64_t grid = (a.nitems + run - 1) / run * run;
  switch (a.R) {
    case 1: hipLaunchKernelGGL(k_attention<1>, dim3((unsigned)grid), dim3(128), 0, st, a); break;
    case 2: hipLaunchKernelGGL(k_attention<2>, dim3((unsigned)grid), dim3(256), 0, st, a); break;
    case 4: hipLaunchKernelGGL(k_attention<4>, dim3((unsigned)grid), dim3(512), 0, st, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_combine(const AttnArgs& a, const SplitRow* splits, int64_t nsplit, hipStream_t st) {
  if (nsplit <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_combine, dim3((unsigned)nsplit, a.R), dim3(256), 0, st, a, splits);
  return hipGetLastError();
}

}  // namespace mmi
