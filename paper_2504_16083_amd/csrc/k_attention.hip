// Block-sparse causal attention over permuted 64x64 blocks (Algorithms 5-7:
// the Grid, Q-Boundary and 2D-Boundary FlashAttention kernels are one
// kernel here, because the permutation and the selected key blocks are data:
// qperm / kperm say which token each slot holds, the block index says which
// key blocks each query block visits).
//
// One work item = a row group of R permuted query blocks and a contiguous
// range of the union of their key-block lists; each union entry carries one
// flag per query block. The workgroup has 2R waves; waves 2r and 2r+1 own
// the 64 rows of member r (32 rows each). Every key block of the range is
// loaded once into LDS and used by all members that selected it. Per key
// block and active wave:
//   S^T (64 keys x 32 queries) = K Q^T         16 MFMA 32x32x16 bf16
//   mask by original positions (k <= q) where the block reaches past the
//   wave's first query, online softmax in fp32 (log2 domain)
//   O^T (128 x 32) += V^T P^T                  16 MFMA 32x32x16 bf16
// S^T puts one query per lane: row max/sum need one cross-lane exchange and
// the accumulator is already the P operand of the PV product.
//
// Pipeline: K/V blocks rotate through three LDS stages, one barrier per
// block. While the softmax of block t runs on the VALU, the same wave issues
// the QK MFMAs of block t+1 (independent, so the matrix core and the VALU
// overlap); the global loads of block t+3 are in flight meanwhile. V stays
// row-major in LDS and is read into the PV operand with the gfx950
// transpose read (ds_read_b64_tr_b16): in each 16-lane group, output lane i,
// element e is element i%4 of the 8-byte row addressed by lane 4e + i/4.
#include "device.hpp"
#include "internal.hpp"

namespace mmi {

constexpr int KPITCH = 136;   // bf16 per K row in LDS (272 B): conflict-free 16-byte operand reads
constexpr int VPITCH = 160;   // bf16 per V row in LDS (320 B): transpose reads of 4 rows hit distinct banks
constexpr int NSTAGE = 3;

struct __align__(16) Stage {
  uint16_t k[B * KPITCH];
  uint16_t v[B * VPITCH];
  int32_t kpos[B];
};

__device__ __forceinline__ int slot_pos(const int32_t* perm, int slot, int S) {
  return perm ? perm[slot] : (slot < S ? slot : -1);
}

template <int R>
struct Tile {
  static constexpr int NT = 128 * R;           // threads
  static constexpr int L = 1024 / NT;          // 16-byte chunks of K (and of V) per thread and block
};

template <int R>
struct BlockRegs {
  bf16x8 k[Tile<R>::L];
  bf16x8 v[Tile<R>::L];
};

template <int R>
__device__ __forceinline__ void fetch_block(BlockRegs<R>& r, const AttnArgs& a, const HeadDev& hd, int jblk,
                                            int tid) {
  const uint16_t* kb = reinterpret_cast<const uint16_t*>(a.k.p) + (int64_t)hd.kvh * a.k.sh;
  const uint16_t* vb = reinterpret_cast<const uint16_t*>(a.v.p) + (int64_t)hd.kvh * a.v.sh;
#pragma unroll
  for (int it = 0; it < Tile<R>::L; ++it) {
    const int u = tid + it * Tile<R>::NT;
    const int key = u >> 4, chunk = u & 15;
    const int kp = slot_pos(hd.kperm, jblk * B + key, a.S);
    r.k[it] = kp >= 0 ? load16(kb + (int64_t)kp * a.k.ss + chunk * 8) : zero8();
    r.v[it] = kp >= 0 ? load16(vb + (int64_t)kp * a.v.ss + chunk * 8) : zero8();
  }
}

template <int R>
__device__ __forceinline__ void stage_block(Stage& st, const BlockRegs<R>& r, const HeadDev& hd, int jblk, int S,
                                            int tid) {
#pragma unroll
  for (int it = 0; it < Tile<R>::L; ++it) {
    const int u = tid + it * Tile<R>::NT;
    const int key = u >> 4, chunk = u & 15;
    *reinterpret_cast<bf16x8*>(&st.k[key * KPITCH + chunk * 8]) = r.k[it];
    *reinterpret_cast<bf16x8*>(&st.v[key * VPITCH + chunk * 8]) = r.v[it];
  }
  if (tid < B) st.kpos[tid] = slot_pos(hd.kperm, jblk * B + tid, S);
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

typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

__device__ __forceinline__ bf16x4 tr_read(const uint16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p));
}

// S^T tile pair (keys 0-31 and 32-63 of the block) for this wave's 32 queries.
__device__ __forceinline__ void qk_block(const Stage& st, const bf16x8 (&qr)[8], int c, int h, f32x16 (&s)[2]) {
#pragma unroll
  for (int kt = 0; kt < 2; ++kt)
#pragma unroll
    for (int x = 0; x < 16; ++x) s[kt][x] = 0.0f;
#pragma unroll
  for (int st8 = 0; st8 < 8; ++st8) {
    const bf16x8 k0 = *reinterpret_cast<const bf16x8*>(&st.k[c * KPITCH + h * 64 + st8 * 8]);
    const bf16x8 k1 = *reinterpret_cast<const bf16x8*>(&st.k[(32 + c) * KPITCH + h * 64 + st8 * 8]);
    s[0] = mfma32(k0, qr[st8], s[0]);
    s[1] = mfma32(k1, qr[st8], s[1]);
  }
}

__device__ __forceinline__ void mask_block(const Stage& st, int qpos, int h, f32x16 (&s)[2]) {
#pragma unroll
  for (int kt = 0; kt < 2; ++kt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int4 kp = *reinterpret_cast<const int4*>(&st.kpos[kt * 32 + 8 * i + 4 * h]);
      if (kp.x < 0 || kp.x > qpos) s[kt][4 * i + 0] = -INFINITY;
      if (kp.y < 0 || kp.y > qpos) s[kt][4 * i + 1] = -INFINITY;
      if (kp.z < 0 || kp.z > qpos) s[kt][4 * i + 2] = -INFINITY;
      if (kp.w < 0 || kp.w > qpos) s[kt][4 * i + 3] = -INFINITY;
    }
}

// Online-softmax step: new running max, P = 2^(s*sc - m) packed to bf16
// B operands, row sum. Returns the rescale factor (1 when the max held).
__device__ __forceinline__ void softmax_block(f32x16 (&s)[2], float sc, float& m, float& l, bf16x8 (&pb)[4],
                                              float& alpha) {
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
#pragma unroll
  for (int stp = 0; stp < 4; ++stp) {
    const int kt = stp >> 1, half = stp & 1;
#pragma unroll
    for (int x = 0; x < 8; ++x) pb[stp][x] = (__bf16)s[kt][4 * (2 * half + (x >> 2)) + (x & 3)];
  }
  rs += __shfl_xor(rs, 32);
  alpha = fast_exp2(m - m_new);
  l = l * alpha + rs;
  m = m_new;
}

// O^T += V^T P^T; the V^T operand comes from row-major V by transpose reads.
__device__ __forceinline__ void pv_block(const Stage& st, const bf16x8 (&pb)[4], int vlane, f32x16 (&o)[4]) {
#pragma unroll
  for (int stp = 0; stp < 4; ++stp) {
    const int kt = stp >> 1, half = stp & 1;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      const uint16_t* p0 = &st.v[vlane + (32 * kt + 16 * half) * VPITCH + 32 * dt];
      const bf16x4 lo = tr_read(p0);
      const bf16x4 hi = tr_read(p0 + 8 * VPITCH);
      const bf16x8 va = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
      o[dt] = mfma32(va, pb[stp], o[dt]);
    }
  }
}

template <int R>
__global__ __launch_bounds__(128 * R) __attribute__((amdgpu_waves_per_eu(R == 4 ? 2 : 1))) void k_attention(AttnArgs a) {
  __shared__ Stage stg[NSTAGE];
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
  // transpose-read source row/column of this lane inside a V stage
  const int grp = lane >> 4, li = lane & 15;
  const int vlane = (4 * (grp >> 1) + (li >> 2)) * VPITCH + 16 * (grp & 1) + 4 * (li & 3);

  f32x16 o[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[dt][e] = 0.0f;
  float m = NEG_BIG, l = 0.0f;
  const float sc = 0.08838834764831845f * LOG2E;   // sqrt(1/128) * log2(e)

  const int n = w.e1 - w.e0;
  const int32_t* ent = hd.gcol + w.e0;
  BlockRegs<R> regs;
  int e_cur = ent[0];
  fetch_block<R>(regs, a, hd, e_cur & 0xffff, tid);
  stage_block<R>(stg[0], regs, hd, e_cur & 0xffff, a.S, tid);
  int e_nxt = n > 1 ? ent[1] : 0;
  if (n > 1) {
    fetch_block<R>(regs, a, hd, e_nxt & 0xffff, tid);
    stage_block<R>(stg[1], regs, hd, e_nxt & 0xffff, a.S, tid);
  }
  int e_far = n > 2 ? ent[2] : 0;
  if (n > 2) fetch_block<R>(regs, a, hd, e_far & 0xffff, tid);
  __syncthreads();

  f32x16 s_cur[2], s_nxt[2];
  bool act_cur = (e_cur >> (16 + rb)) & 1;
  if (act_cur) qk_block(stg[0], qr, c, h, s_cur);
  int cs = 0;                                   // stage of block t
  for (int t = 0; t < n; ++t) {
    const int ns = cs == NSTAGE - 1 ? 0 : cs + 1;
    const bool act_nxt = t + 1 < n && ((e_nxt >> (16 + rb)) & 1);
    if (act_cur && block_kmax(hd, e_cur & 0xffff, a.S) > qmin) mask_block(stg[cs], qpos, h, s_cur);
    bf16x8 pb[4];
    float alpha = 1.0f;
    if (act_cur && act_nxt) {
      // QK MFMAs of block t+1 are independent of the softmax of block t
      qk_block(stg[ns], qr, c, h, s_nxt);
      softmax_block(s_cur, sc, m, l, pb, alpha);
    } else {
      if (act_nxt) qk_block(stg[ns], qr, c, h, s_nxt);
      if (act_cur) softmax_block(s_cur, sc, m, l, pb, alpha);
    }
    if (act_cur) {
      if (__any(alpha != 1.0f)) {
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
#pragma unroll
          for (int x = 0; x < 16; ++x) o[dt][x] *= alpha;
      }
      pv_block(stg[cs], pb, vlane, o);
    }
    if (t + 2 < n) {
      const int fs = ns == NSTAGE - 1 ? 0 : ns + 1;
      stage_block<R>(stg[fs], regs, hd, e_far & 0xffff, a.S, tid);
      if (t + 3 < n) {
        const int e3 = ent[t + 3];
        fetch_block<R>(regs, a, hd, e3 & 0xffff, tid);
        e_cur = e_nxt; e_nxt = e_far; e_far = e3;
      } else {
        e_cur = e_nxt; e_nxt = e_far; e_far = 0;
      }
    } else {
      e_cur = e_nxt; e_nxt = e_far; e_far = 0;
    }
    __syncthreads();
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) s_cur[kt] = s_nxt[kt];
    act_cur = act_nxt;
    cs = ns;
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
