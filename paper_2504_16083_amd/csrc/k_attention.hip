// Block-sparse causal attention over permuted 64x64 blocks (Algorithms 5-7:
// the Grid, Q-Boundary and 2D-Boundary FlashAttention kernels are one
// kernel here, because the permutation and the selected key blocks are data:
// qperm / kperm say which token each slot holds, the CSR says which key
// blocks each query block visits).
//
// One work item = one permuted query block (64 rows) and a contiguous range
// of its selected key blocks. Workgroup = 2 waves; wave w owns query rows
// 32w..32w+31. Per key block:
//   S^T (64 keys x 32 queries) = K Q^T         16 MFMA 32x32x16 bf16
//   mask by original positions (k <= q), online softmax in fp32 (log2 domain)
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
constexpr int VPITCH = 72;    // bf16 per V^T row in LDS: 64 + 8 pad (144 B)

struct __align__(16) AttnSmem {
  uint16_t k[B * KPITCH];
  uint16_t vt[D * VPITCH];
  int32_t kpos[B];
};

__device__ __forceinline__ int slot_pos(const int32_t* perm, int slot, int S) {
  return perm ? perm[slot] : (slot < S ? slot : -1);
}

struct BlockRegs {
  bf16x8 k[8];
  bf16x8 v[8];
  int32_t kp;      // key position for LDS (threads < 64)
};

__device__ __forceinline__ void fetch_block(BlockRegs& r, const AttnArgs& a, const HeadDev& hd,
                                            int jblk, int tid) {
  const uint16_t* kb = reinterpret_cast<const uint16_t*>(a.k.p) + (int64_t)hd.kvh * a.k.sh;
  const uint16_t* vb = reinterpret_cast<const uint16_t*>(a.v.p) + (int64_t)hd.kvh * a.v.sh;
  const int base = jblk * B;
  const int chunk = tid & 15;
#pragma unroll
  for (int it = 0; it < 8; ++it) {
    const int key = (tid >> 4) + 8 * it;
    const int kp = slot_pos(hd.kperm, base + key, a.S);
    r.k[it] = kp >= 0 ? load16(kb + (int64_t)kp * a.k.ss + chunk * 8) : zero8();
  }
  const int kg = tid >> 4;
#pragma unroll
  for (int g2 = 0; g2 < 2; ++g2) {
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const int key = 32 * g2 + 4 * kg + rr;
      const int kp = slot_pos(hd.kperm, base + key, a.S);
      r.v[g2 * 4 + rr] = kp >= 0 ? load16(vb + (int64_t)kp * a.v.ss + chunk * 8) : zero8();
    }
  }
  r.kp = tid < B ? slot_pos(hd.kperm, base + tid, a.S) : 0;
}

__device__ __forceinline__ void stage_block(AttnSmem& sm, const BlockRegs& r, int tid) {
  const int chunk = tid & 15;
#pragma unroll
  for (int it = 0; it < 8; ++it) {
    const int key = (tid >> 4) + 8 * it;
    *reinterpret_cast<bf16x8*>(&sm.k[key * KPITCH + chunk * 8]) = r.k[it];
  }
  const int kg = tid >> 4;
#pragma unroll
  for (int g2 = 0; g2 < 2; ++g2) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      bf16x4 t;
      t[0] = r.v[g2 * 4 + 0][e];
      t[1] = r.v[g2 * 4 + 1][e];
      t[2] = r.v[g2 * 4 + 2][e];
      t[3] = r.v[g2 * 4 + 3][e];
      *reinterpret_cast<bf16x4*>(&sm.vt[(chunk * 8 + e) * VPITCH + 32 * g2 + 4 * kg]) = t;
    }
  }
  if (tid < B) sm.kpos[tid] = r.kp;
}

__global__ __launch_bounds__(128, 2) void k_attention(AttnArgs a) {
  __shared__ AttnSmem sm;
  const WorkItem w = a.items[blockIdx.x];
  const HeadDev hd = a.heads[w.head];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int c = lane & 31, h = lane >> 5;

  const int qslot = w.qblk * B + wave * 32 + c;
  const int qpos = slot_pos(hd.qperm, qslot, a.S);
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

  BlockRegs regs;
  fetch_block(regs, a, hd, hd.col[w.e0], tid);
  for (int e = w.e0; e < w.e1; ++e) {
    stage_block(sm, regs, tid);
    __syncthreads();
    if (e + 1 < w.e1) fetch_block(regs, a, hd, hd.col[e + 1], tid);

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

    float mx = NEG_BIG;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int kp = sm.kpos[kt * 32 + 8 * i + 4 * h + j];
          float x = s[kt][4 * i + j] * sc;
          x = (kp < 0 || kp > qpos) ? -INFINITY : x;
          s[kt][4 * i + j] = x;
          mx = fmaxf(mx, x);
        }
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m, mx);
    const float alpha = fast_exp2(m - m_new);
    float rs = 0.0f;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int x = 0; x < 16; ++x) {
        const float p = fast_exp2(s[kt][x] - m_new);
        s[kt][x] = p;
        rs += p;
      }
    rs += __shfl_xor(rs, 32);
    l = l * alpha + rs;
    m = m_new;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int x = 0; x < 16; ++x) o[dt][x] *= alpha;

#pragma unroll
    for (int st = 0; st < 4; ++st) {
      const int kt = st >> 1, half = st & 1;
      bf16x8 pb;
#pragma unroll
      for (int x = 0; x < 8; ++x) pb[x] = (__bf16)s[kt][4 * (2 * half + (x >> 2)) + (x & 3)];
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        const uint16_t* vr = &sm.vt[(32 * dt + c) * VPITCH + kt * 32 + 16 * half + 4 * h];
        const bf16x4 lo = *reinterpret_cast<const bf16x4*>(vr);
        const bf16x4 hi = *reinterpret_cast<const bf16x4*>(vr + 8);
        bf16x8 va;
#pragma unroll
        for (int x = 0; x < 4; ++x) { va[x] = lo[x]; va[4 + x] = hi[x]; }
        o[dt] = mfma32(va, pb, o[dt]);
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
    const int row = wave * 32 + c;
    float* po = a.part_o + ((int64_t)w.part * B + row) * D;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float4 t = make_float4(o[dt][4 * i], o[dt][4 * i + 1], o[dt][4 * i + 2], o[dt][4 * i + 3]);
        *reinterpret_cast<float4*>(po + 32 * dt + 8 * i + 4 * h) = t;
      }
    if (h == 0) {
      float* ml = a.part_ml + ((int64_t)w.part * B + row) * 2;
      ml[0] = m;
      ml[1] = l;
    }
  }
}

// Merge the (O, m, l) partials of a split query block in a fixed order:
// M = max m_p, L = sum l_p 2^(m_p - M), O = sum O_p 2^(m_p - M) / L.
__global__ __launch_bounds__(256) void k_combine(AttnArgs a, const SplitRow* splits) {
  const SplitRow sr = splits[blockIdx.x];
  const HeadDev hd = a.heads[sr.head];
  const int row = threadIdx.x >> 2, quarter = threadIdx.x & 3;
  const int qslot = sr.qblk * B + row;
  const int qpos = slot_pos(hd.qperm, qslot, a.S);
  if (qpos < 0) return;
  float M = NEG_BIG;
  for (int p = 0; p < sr.nparts; ++p) M = fmaxf(M, a.part_ml[((int64_t)(sr.part0 + p) * B + row) * 2]);
  float acc[32];
#pragma unroll
  for (int x = 0; x < 32; ++x) acc[x] = 0.0f;
  float L = 0.0f;
  for (int p = 0; p < sr.nparts; ++p) {
    const int64_t pr = (int64_t)(sr.part0 + p) * B + row;
    const float w = fast_exp2(a.part_ml[pr * 2] - M);
    L += a.part_ml[pr * 2 + 1] * w;
    const float4* src = reinterpret_cast<const float4*>(a.part_o + pr * D + quarter * 32);
#pragma unroll
    for (int x = 0; x < 8; ++x) {
      const float4 t = src[x];
      acc[4 * x] += t.x * w; acc[4 * x + 1] += t.y * w;
      acc[4 * x + 2] += t.z * w; acc[4 * x + 3] += t.w * w;
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
  hipLaunchKernelGGL(k_attention, dim3((unsigned)a.nitems), dim3(128), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_combine(const AttnArgs& a, const SplitRow* splits, int64_t nsplit, hipStream_t st) {
  if (nsplit <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_combine, dim3((unsigned)nsplit), dim3(256), 0, st, a, splits);
  return hipGetLastError();
}

}  // namespace mmi
