// Block-sparse causal attention over permuted 64x64 blocks (Algorithms 5-7:
// the Grid, Q-Boundary and 2D-Boundary FlashAttention kernels are one
// kernel here, because the permutation and the selected key blocks are data:
// qperm / kperm say which token each slot holds, the block index says which
// key blocks each query block visits).
//
// One work item = a row group of R permuted query blocks and a contiguous
// range of the union of their key-block lists; each union entry carries one
// flag per query block. The workgroup has 2R waves, each owning 32 rows of
// one member. Every key block of the range is loaded once into LDS and used
// by all members that selected it. Per key block and active wave:
//   S^T (64 keys x 32 queries) = K Q^T         16 MFMA 32x32x16 bf16
//   mask by original positions (k <= q) where the block reaches past the
//   wave's first query, online softmax in fp32 (log2 domain)
//   O^T (128 x 32) += V^T P^T                  16 MFMA 32x32x16 bf16
// S^T puts one query per lane: row max/sum need one cross-lane exchange and
// the accumulator is already the P operand of the PV product.
//
// Pipeline: K/V blocks rotate through four LDS stages with one barrier per
// block. Step t multiplies P(t)V(t), turns the scores of block t+1 into
// P(t+1) and computes the scores of block t+2; the three share no data and
// are issued interleaved within each wave (MFMA, then a share of the
// softmax), because the vector ALU overlaps only MFMAs of the same wave.
// Meanwhile block t+3 is written to its stage from registers, the global
// loads of block t+4 are in flight and the key positions of block t+5 are
// loading. The two waves of a SIMD stage at opposite ends of the step (one
// before its products, one after), so that the SIMD's matrix core is fed by
// one wave while the other waits on its loads.
// V stays row-major in LDS and is read into the PV operand with the gfx950
// transpose read (ds_read_b64_tr_b16): in each 16-lane group, output lane i,
// element e is element i%4 of the 8-byte row addressed by lane 4e + i/4.
//
// The running maximum is only moved when a row's block maximum exceeds it by
// more than RESCALE_SLACK (log2 units): P entries then stay below 2^8, which
// neither bf16 nor the fp32 sums mind, and the O rescale becomes rare.
// Each row keeps the sum lo of the bf16-rounded P that the PV product
// actually uses (O = PV / lo): O is then a convex combination of V rows
// whatever the rounding of P, so a row dominated by one key is not scaled by
// that key's rounding error (up to 2^-8 relative, which for |V| of several
// units exceeds the output bound). Only when the caller asks for the LSE
// (kernel variant WL) does a row also sum the fp32 P into l, for LSE = m +
// log l; split rows merge their O by lo in either variant.
#include "device.hpp"
#include "internal.hpp"

namespace mmi {

constexpr int KPITCH = 136;   // bf16 per K row in LDS (272 B): conflict-free 16-byte operand reads
constexpr int VPITCH = 160;   // bf16 per V row in LDS (320 B): transpose reads of 4 rows hit distinct banks
constexpr int NSTAGE = 4;
constexpr float RESCALE_SLACK = 8.0f;

struct __align__(16) Stage {
  uint16_t k[B * KPITCH];
  uint16_t v[B * VPITCH];
  int32_t kpos[B];            // original key position, INT_BIG for padding
};

// Load of plan data through a global-address-space pointer (a generic one
// would become a flat load, which also counts against the LDS wait counter).
__device__ __forceinline__ int ld_global(const int32_t* p) {
  return *(const __attribute__((address_space(1))) int32_t*)(p);
}

__device__ __forceinline__ int slot_pos(const int32_t* perm, int slot, int S) {
  return perm ? ld_global(perm + slot) : (slot < S ? slot : -1);
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
  int kp[Tile<R>::L];          // original positions of the thread's keys (-1 = padding)
};

// Per-thread view of the K/V rows it loads. A thread always loads the same
// 16-byte chunk (tid % 16) of keys key0, key0 + NT/16, ...; K and V of the
// KV head are buffer resources (base and size in scalar registers), and a
// row's byte offset is one 24-bit multiply-add: positions are below 2^21
// and S times the token stride in bytes stays below 2^32 (checked on the
// host). Loads past the resource size would read zeros.
template <int R>
struct KeySrc {
  __amdgpu_buffer_rsrc_t kr, vr;
  uint32_t kss, vss;          // token strides in bytes
  uint32_t cb;                // this thread's chunk offset in bytes
  const int32_t* perm;
  int S, key0;
  __device__ __forceinline__ void init(const AttnArgs& a, const HeadDev& hd, int tid) {
    const uint16_t* kb = reinterpret_cast<const uint16_t*>(a.k.p) + (int64_t)hd.kvh * a.k.sh;
    const uint16_t* vb = reinterpret_cast<const uint16_t*>(a.v.p) + (int64_t)hd.kvh * a.v.sh;
    kss = (uint32_t)a.k.ss * 2u;
    vss = (uint32_t)a.v.ss * 2u;
    kr = __builtin_amdgcn_make_buffer_rsrc((void*)kb, (short)0, (int)((uint32_t)(a.S - 1) * kss + 2u * D), 0x00020000);
    vr = __builtin_amdgcn_make_buffer_rsrc((void*)vb, (short)0, (int)((uint32_t)(a.S - 1) * vss + 2u * D), 0x00020000);
    cb = (uint32_t)(tid & 15) * 16u;
    perm = hd.kperm;
    S = a.S;
    key0 = tid >> 4;
  }
};

__device__ __forceinline__ bf16x8 buffer_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0));
}

// Original positions of the keys this thread loads from key block jblk.
template <int R, bool PERM>
__device__ __forceinline__ void fetch_pos(int (&kp)[Tile<R>::L], const KeySrc<R>& ks, int jblk) {
#pragma unroll
  for (int it = 0; it < Tile<R>::L; ++it) {
    const int slot = jblk * B + ks.key0 + it * (Tile<R>::NT / 16);
    kp[it] = PERM ? ld_global(ks.perm + slot) : (slot < ks.S ? slot : -1);
  }
}

// Global loads of one K/V block (positions from fetch_pos). Padding slots
// read key row 0 (always present); their V is zeroed when staged and their
// scores are masked, so the values never reach the output. Nothing here
// touches the loaded data: the loads stay in flight until stage_block.
template <int R>
__device__ __forceinline__ void fetch_block(BlockRegs<R>& r, const KeySrc<R>& ks, const int (&kp)[Tile<R>::L]) {
#pragma unroll
  for (int it = 0; it < Tile<R>::L; ++it) {
    const uint32_t row = kp[it] >= 0 ? (uint32_t)kp[it] : 0u;
    r.k[it] = buffer_load16(ks.kr, __umul24(row, ks.kss) + ks.cb);
    r.v[it] = buffer_load16(ks.vr, __umul24(row, ks.vss) + ks.cb);
    r.kp[it] = kp[it];
  }
}

template <int R>
__device__ __forceinline__ void stage_block(Stage& st, const BlockRegs<R>& r, int tid) {
#pragma unroll
  for (int it = 0; it < Tile<R>::L; ++it) {
    const int u = tid + it * Tile<R>::NT;
    const int key = u >> 4, chunk = u & 15;
    const bool pad = r.kp[it] < 0;
    *reinterpret_cast<bf16x8*>(&st.k[key * KPITCH + chunk * 8]) = r.k[it];
    *reinterpret_cast<bf16x8*>(&st.v[key * VPITCH + chunk * 8]) = pad ? zero8() : r.v[it];
    if (chunk == 0) st.kpos[key] = pad ? INT_BIG : r.kp[it];
  }
}

// Union entries of a work item, read 64 at a time into one VGPR per lane and
// taken out with readlane (wave-uniform results, no scalar-load waits on the
// LDS counter inside the block loop).
struct EntryStream {
  const int32_t* ent;
  int n, lane;
  int cur, nxt;                // entries [base, base+64) and [base+64, base+128)
  __device__ __forceinline__ void init(const int32_t* e, int count, int ln) {
    ent = e; n = count; lane = ln;
    cur = lane < n ? ld_global(ent + lane) : 0;
    nxt = 64 + lane < n ? ld_global(ent + 64 + lane) : 0;
  }
  // entry i; calls come with i = 0, 1, 2, ... in order
  __device__ __forceinline__ int get(int i) {
    if (i >= n) return 0;
    if (i >= 64 && (i & 63) == 0) {
      cur = nxt;
      nxt = i + 64 + lane < n ? ld_global(ent + i + 64 + lane) : 0;
    }
    return __builtin_amdgcn_readlane(cur, i & 63);
  }
};

// Work-item order: hardware hands consecutive workgroups to the 8 XCDs in
// turn, so workgroup b runs on XCD b mod 8 as that XCD's (b / 8)-th. The
// plan's item map lists each XCD's items in order (runs of neighbouring row
// groups, which share key blocks in that XCD's L2, balanced over the XCDs by
// modelled cost).
__device__ __forceinline__ int64_t item_of_block(const AttnArgs& a, int64_t b) {
  const int64_t k = b >> 3;
  return k < a.map_len ? a.item_map[(b & 7) * a.map_len + k] : -1;
}

typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

__device__ __forceinline__ bf16x4 tr_read(const uint16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p));
}

// S^T tile pair (keys 0-31 and 32-63 of the block) for this wave's 32 queries.
__device__ __forceinline__ void qk_block(const Stage& st, const bf16x8 (&qr)[8], int c, int h, f32x16 (&s)[2]) {
  const f32x16 zero = {};
#pragma unroll
  for (int st8 = 0; st8 < 8; ++st8) {
    const bf16x8 k0 = *reinterpret_cast<const bf16x8*>(&st.k[c * KPITCH + h * 64 + st8 * 8]);
    const bf16x8 k1 = *reinterpret_cast<const bf16x8*>(&st.k[(32 + c) * KPITCH + h * 64 + st8 * 8]);
    s[0] = mfma32(k0, qr[st8], st8 == 0 ? zero : s[0]);
    s[1] = mfma32(k1, qr[st8], st8 == 0 ? zero : s[1]);
  }
}

__device__ __forceinline__ void mask_block(const Stage& st, int qpos, int h, f32x16 (&s)[2]) {
#pragma unroll
  for (int kt = 0; kt < 2; ++kt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int4 kp = *reinterpret_cast<const int4*>(&st.kpos[kt * 32 + 8 * i + 4 * h]);
      if (kp.x > qpos) s[kt][4 * i + 0] = -INFINITY;
      if (kp.y > qpos) s[kt][4 * i + 1] = -INFINITY;
      if (kp.z > qpos) s[kt][4 * i + 2] = -INFINITY;
      if (kp.w > qpos) s[kt][4 * i + 3] = -INFINITY;
    }
}

// Combination of the two 32-lane halves (lanes l and l ^ 32 hold the two
// halves of a query's scores) by a lane swap instead of an LDS permute.
__device__ __forceinline__ float xhalf_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float xhalf_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;

// Sum of the 8 bf16 values of a packed P operand, added to acc (v_dot2 with ones).
__device__ __forceinline__ float sum8(const bf16x8& p, float acc) {
  const bf16x2 one = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
  for (int x = 0; x < 4; ++x) acc = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{p[2 * x], p[2 * x + 1]}, one, acc, false);
  return acc;
}

// Online-softmax step on the scores of one block: P = 2^(s*sc - m) packed to
// bf16 B operands, row sums into l (fp32 P) and lo (bf16 P). m moves (alpha < 1) only when some row's
// block maximum passes it by more than RESCALE_SLACK. Branch-free, so that
// the compiler can interleave it with independent MFMAs.
template <bool WL>
__device__ __forceinline__ void softmax_block(f32x16 (&s)[2], float sc, float& m, float& l, float& lo,
                                              bf16x8 (&pb)[4], float& alpha) {
  float mx = NEG_BIG;
#pragma unroll
  for (int kt = 0; kt < 2; ++kt)
#pragma unroll
    for (int x = 0; x < 16; ++x) mx = fmaxf(mx, s[kt][x]);
  mx = xhalf_max(mx) * sc;                       // scale > 0: max commutes with it
  const bool move = __any(mx > m + RESCALE_SLACK);
  const float m_new = move ? fmaxf(m, mx) : m;
  alpha = fast_exp2(m - m_new);
  m = m_new;
  float rs = 0.0f;
#pragma unroll
  for (int kt = 0; kt < 2; ++kt)
#pragma unroll
    for (int x = 0; x < 16; ++x) {
      const float p = fast_exp2(fmaf(s[kt][x], sc, -m_new));
      s[kt][x] = p;
      if constexpr (WL) rs += p;
    }
  float ro = 0.0f;
#pragma unroll
  for (int stp = 0; stp < 4; ++stp) {
    const int kt = stp >> 1, half = stp & 1;
#pragma unroll
    for (int x = 0; x < 8; ++x) pb[stp][x] = (__bf16)s[kt][4 * (2 * half + (x >> 2)) + (x & 3)];
    ro = sum8(pb[stp], ro);
  }
  if constexpr (WL) l = l * alpha + xhalf_sum(rs);
  lo = lo * alpha + xhalf_sum(ro);
}

// Per-wave state of the block loop.
struct WaveState {
  f32x16 o[4];
  bf16x8 qr[8];
  float m, l, lo;
  int qpos, rb, c, h, vlane;
  bool late;                  // stages before the products (second wave of a SIMD)
};

// Mask threshold of a wave's rows: keys above it are masked. A bidirectional
// head masks only padding keys (position INT_BIG).
__device__ __forceinline__ int mask_limit(const WaveState& ws, bool causal) {
  return causal || ws.qpos < 0 ? ws.qpos : INT_BIG - 1;
}

__device__ __forceinline__ bool sel(int e, int rb) { return (e >> (16 + rb)) & 1; }
__device__ __forceinline__ bool needs_mask(int e, int rb) { return (e >> (24 + rb)) & 1; }

// Softmax of one block cut into pieces that can be spread between MFMAs:
// 0-3 running maximum over 8 scores each, 4 new maximum, 5-36 one
// exponential each, 37-40 bf16 packing and the bf16 row sum, 41 row sums.
constexpr int SM_PIECES = 42;

struct SoftmaxState {
  float mx, m_new, rs, ro;
};

template <bool WL>
__device__ __forceinline__ void softmax_piece(int pc, f32x16 (&s)[2], float sc, float& m, float& l, float& lo,
                                              bf16x8 (&pb)[4], float& alpha, SoftmaxState& st) {
  if (pc < 4) {
    const int kt = pc >> 1, x0 = (pc & 1) * 8;
    float v = pc == 0 ? NEG_BIG : st.mx;
#pragma unroll
    for (int x = 0; x < 8; ++x) v = fmaxf(v, s[kt][x0 + x]);
    st.mx = v;
  } else if (pc == 4) {
    const float mx = xhalf_max(st.mx) * sc;      // scale > 0: max commutes with it
    const bool move = __any(mx > m + RESCALE_SLACK);
    st.m_new = move ? fmaxf(m, mx) : m;
    alpha = fast_exp2(m - st.m_new);
    m = st.m_new;
    st.rs = 0.0f;
    st.ro = 0.0f;
  } else if (pc < 37) {
    const int e = pc - 5, kt = e >> 4, x = e & 15;
    const float p = fast_exp2(fmaf(s[kt][x], sc, -st.m_new));
    s[kt][x] = p;
    if constexpr (WL) st.rs += p;
  } else if (pc < 41) {
    const int stp = pc - 37, kt = stp >> 1, half = stp & 1;
#pragma unroll
    for (int x = 0; x < 8; ++x) pb[stp][x] = (__bf16)s[kt][4 * (2 * half + (x >> 2)) + (x & 3)];
    st.ro = sum8(pb[stp], st.ro);
  } else {
    if constexpr (WL) l = l * alpha + xhalf_sum(st.rs);
    lo = lo * alpha + xhalf_sum(st.ro);
  }
}

// The three pieces of step t that share no data: QK(t+2) and PV(t) on the
// matrix cores, softmax(t+1) on the vector ALU (SM). They are written out
// interleaved (MFMA, then a share of the softmax), because the hardware
// overlaps vector instructions only with MFMAs of the same wave, and a
// scheduling barrier after each slot keeps that order. MFMA A operands are
// read from LDS three slots ahead, also in steps without a softmax (a wave
// whose member skips block t+1), where an operand read right before each
// MFMA would leave every MFMA waiting for LDS; those steps keep the operands
// in the P buffer of block t+1, which the member does not use.
template <bool QK, bool PV, bool SM, bool WL>
__device__ __forceinline__ void fused_step(WaveState& ws, const Stage& kst, const Stage& vst, f32x16 (&s_qk)[2],
                                           const bf16x8 (&p_cur)[4], f32x16 (&s_sm)[2], bf16x8 (&p_new)[4],
                                           float sc, float& alpha) {
  constexpr int NQ = QK ? 16 : 0;
  constexpr int NM = NQ + (PV ? 16 : 0);
  constexpr int AHEAD = 3;
  SoftmaxState st;
  const f32x16 zero = {};
  // A operand of MFMA slot i: K rows for QK slots, transposed V for PV slots
  auto operand = [&](int i) -> bf16x8 {
    if (i < NQ) {
      const int st8 = i >> 1, kt = i & 1;
      return *reinterpret_cast<const bf16x8*>(&kst.k[(kt * 32 + ws.c) * KPITCH + ws.h * 64 + st8 * 8]);
    }
    const int j = i - NQ, stp = j >> 2, dt = j & 3, kt = stp >> 1, half = stp & 1;
    const uint16_t* p0 = &vst.v[ws.vlane + (32 * kt + 16 * half) * VPITCH + 32 * dt];
    const bf16x4 lo = tr_read(p0);
    const bf16x4 hi = tr_read(p0 + 8 * VPITCH);
    return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  };
  // without a softmax the P buffer of block t+1 is free (the member skips
  // that block) and holds the operands in flight
  bf16x8 opa_own[AHEAD + 1];
  bf16x8* opa = SM ? opa_own : p_new;
#pragma unroll
  for (int i = 0; i < AHEAD && i < NM; ++i) opa[i] = operand(i);
  int pc = 0;
#pragma unroll
  for (int i = 0; i < NM; ++i) {
    if (i + AHEAD < NM) opa[(i + AHEAD) % (AHEAD + 1)] = operand(i + AHEAD);
    const bf16x8 av = opa[i % (AHEAD + 1)];
    if (i < NQ) {
      const int st8 = i >> 1, kt = i & 1;
      s_qk[kt] = mfma32(av, ws.qr[st8], st8 == 0 ? zero : s_qk[kt]);
    } else {
      const int j = i - NQ, stp = j >> 2, dt = j & 3;
      ws.o[dt] = mfma32(av, p_cur[stp], ws.o[dt]);
    }
    if constexpr (SM) {
      const int pe = (i + 1) * SM_PIECES / (NM > 0 ? NM : 1);
#pragma unroll
      for (; pc < pe; ++pc) softmax_piece<WL>(pc, s_sm, sc, ws.m, ws.l, ws.lo, p_new, alpha, st);
    }
    // keep each slot's softmax share next to its MFMA: left to itself the
    // scheduler bunches the vector work and leaves runs of MFMAs without any
    __builtin_amdgcn_sched_barrier(0);
  }
  if constexpr (SM) {
#pragma unroll
    for (; pc < SM_PIECES; ++pc) softmax_piece<WL>(pc, s_sm, sc, ws.m, ws.l, ws.lo, p_new, alpha, st);
  }
}

// Step t. Entries e0..e2 are the union entries t..t+2 (0 past the end): key
// block in bits 0-15, per-member select flags from bit 16, per-member mask
// flags from bit 24. On entry: P(t) in p_cur, the scores of block t+1 in
// s_sm, `regs` loading block t+3, kpn the key positions of block t+4. The
// step multiplies P(t)V(t), turns the scores of t+1 into P(t+1) (p_new),
// computes the scores of t+2 into s_qk, stages t+3 and starts loading t+4.
template <int R, bool PERM, bool CAUSAL, bool WL>
__device__ __forceinline__ void block_step(WaveState& ws, Stage* stg, const KeySrc<R>& ks,
                                           BlockRegs<R>& regs, int (&kpn)[Tile<R>::L], int tid, int t, int n,
                                           int e0, int e1, int e2, int e5, f32x16 (&s_qk)[2],
                                           const bf16x8 (&p_cur)[4], f32x16 (&s_sm)[2], bf16x8 (&p_new)[4],
                                           float sc) {
  const bool a0 = sel(e0, ws.rb);
  const bool a1 = t + 1 < n && sel(e1, ws.rb);
  const bool a2 = t + 2 < n && sel(e2, ws.rb);
  const Stage& vst = stg[t & (NSTAGE - 1)];
  const Stage& kst = stg[(t + 2) & (NSTAGE - 1)];
  float alpha = 1.0f;
  // the second wave of each SIMD stages before its products, the first after
  // them: the SIMD's MFMAs then overlap one wave's staging
  auto side = [&]() {
    if (t + 3 < n) stage_block<R>(stg[(t + 3) & (NSTAGE - 1)], regs, tid);
    if (t + 4 < n) fetch_block<R>(regs, ks, kpn);
    if (t + 5 < n) fetch_pos<R, PERM>(kpn, ks, e5 & 0xffff);
  };
  if (ws.late) side();
  if (a1) {
    if (needs_mask(e1, ws.rb)) mask_block(stg[(t + 1) & (NSTAGE - 1)], mask_limit(ws, CAUSAL), ws.h, s_sm);
    if (a2 && a0) fused_step<true, true, true, WL>(ws, kst, vst, s_qk, p_cur, s_sm, p_new, sc, alpha);
    else if (a2) fused_step<true, false, true, WL>(ws, kst, vst, s_qk, p_cur, s_sm, p_new, sc, alpha);
    else if (a0) fused_step<false, true, true, WL>(ws, kst, vst, s_qk, p_cur, s_sm, p_new, sc, alpha);
    else fused_step<false, false, true, WL>(ws, kst, vst, s_qk, p_cur, s_sm, p_new, sc, alpha);
  } else {
    if (a2 && a0) fused_step<true, true, false, WL>(ws, kst, vst, s_qk, p_cur, s_sm, p_new, sc, alpha);
    else if (a2) fused_step<true, false, false, WL>(ws, kst, vst, s_qk, p_cur, s_sm, p_new, sc, alpha);
    else if (a0) fused_step<false, true, false, WL>(ws, kst, vst, s_qk, p_cur, s_sm, p_new, sc, alpha);
  }
  // stage t+3 (its stage was last read in step t-1), load t+4, positions of t+5
  if (!ws.late) side();
  // O holds P(t)V(t) relative to the old maximum: move it to the new one
  if (a1 && __any(alpha != 1.0f)) {
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int x = 0; x < 16; ++x) ws.o[dt][x] *= alpha;
  }
  __syncthreads();
}

template <int R, bool PERM, bool CAUSAL, bool WL>
__device__ __forceinline__ void block_loop(WaveState& ws, Stage* stg, const AttnArgs& a, const HeadDev& hd,
                                           const WorkItem& w, int tid) {
  KeySrc<R> ks;
  ks.init(a, hd, tid);
  const float sc = 0.08838834764831845f * LOG2E;   // sqrt(1/128) * log2(e)
  const int n = w.e1 - w.e0;
  EntryStream es;
  es.init(hd.gcol + w.e0, n, tid & 63);
  int e0 = es.get(0), e1 = es.get(1), e2 = es.get(2), e3 = es.get(3), e4 = es.get(4);

  // prologue: blocks 0-2 staged, block 3 loading, positions of block 4
  BlockRegs<R> regs;
  int kpn[Tile<R>::L];
  const int ep[3] = {e0, e1, e2};
#pragma unroll
  for (int j = 0; j < 3; ++j) {
    if (j < n) {
      fetch_pos<R, PERM>(kpn, ks, ep[j] & 0xffff);
      fetch_block<R>(regs, ks, kpn);
      stage_block<R>(stg[j], regs, tid);
    }
  }
  if (n > 3) {
    fetch_pos<R, PERM>(kpn, ks, e3 & 0xffff);
    fetch_block<R>(regs, ks, kpn);
  }
  if (n > 4) fetch_pos<R, PERM>(kpn, ks, e4 & 0xffff);
  __syncthreads();

  f32x16 sa[2], sb[2];
  bf16x8 pa[4], pb[4];
  if (sel(e0, ws.rb)) {
    qk_block(stg[0], ws.qr, ws.c, ws.h, sa);
    if (needs_mask(e0, ws.rb)) mask_block(stg[0], mask_limit(ws, CAUSAL), ws.h, sa);
    float alpha;
    softmax_block<WL>(sa, sc, ws.m, ws.l, ws.lo, pa, alpha);
  }
  if (n > 1 && sel(e1, ws.rb)) qk_block(stg[1], ws.qr, ws.c, ws.h, sb);
  // two steps per trip so that the buffers swap roles without copies
  for (int t = 0; t < n; t += 2) {
    int e5 = es.get(t + 5);
    block_step<R, PERM, CAUSAL, WL>(ws, stg, ks, regs, kpn, tid, t, n, e0, e1, e2, e5, sa, pa, sb, pb, sc);
    e0 = e1; e1 = e2; e2 = e3; e3 = e4; e4 = e5;
    if (t + 1 >= n) break;
    e5 = es.get(t + 6);
    block_step<R, PERM, CAUSAL, WL>(ws, stg, ks, regs, kpn, tid, t + 1, n, e0, e1, e2, e5, sb, pb, sa, pa, sc);
    e0 = e1; e1 = e2; e2 = e3; e3 = e4; e4 = e5;
  }
}

template <int R, bool WL>
__global__ __launch_bounds__(128 * R) __attribute__((amdgpu_waves_per_eu(R == 4 ? 2 : 1))) void k_attention(AttnArgs a) {
  __shared__ Stage stg[NSTAGE];
  const int64_t it = item_of_block(a, blockIdx.x);
  if (it < 0 || it >= a.nitems) return;
  const WorkItem w = a.items[it];
  const HeadDev hd = a.heads[w.head];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  // Waves 0..R-1 own rows 0-31 of member `wave`; waves R..2R-1 own rows
  // 32-63 of member (wave - R + R/2) mod R, so that the two waves sharing a
  // SIMD (wave and wave + 4 for R = 4) serve different members.
  const bool upper = wave >= R;
  WaveState ws;
  ws.rb = upper ? (wave - R + R / 2) % R : wave;
  ws.late = upper;
  const int half = upper ? 1 : 0;
  ws.c = lane & 31;
  ws.h = lane >> 5;
  const int qblk = group_row(w.group, ws.rb, R, hd.gp[0]);
  ws.qpos = qblk < hd.nbq ? slot_pos(hd.qperm, qblk * B + half * 32 + ws.c, a.S) : -1;
  {
    const uint16_t* qb = reinterpret_cast<const uint16_t*>(a.q.p) + (int64_t)w.head * a.q.sh;
    const uint16_t* row = qb + (int64_t)max(ws.qpos, 0) * a.q.ss + ws.h * 64;
#pragma unroll
    for (int s = 0; s < 8; ++s) ws.qr[s] = ws.qpos >= 0 ? load16(row + 8 * s) : zero8();
  }
  // transpose-read source row/column of this lane inside a V stage
  const int grp = lane >> 4, li = lane & 15;
  ws.vlane = (4 * (grp >> 1) + (li >> 2)) * VPITCH + 16 * (grp & 1) + 4 * (li & 3);
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int e = 0; e < 16; ++e) ws.o[dt][e] = 0.0f;
  ws.m = NEG_BIG;
  ws.l = 0.0f;
  ws.lo = 0.0f;
  if (!hd.causal) block_loop<R, true, false, WL>(ws, stg, a, hd, w, tid);
  else if (hd.kperm) block_loop<R, true, true, WL>(ws, stg, a, hd, w, tid);
  else block_loop<R, false, true, WL>(ws, stg, a, hd, w, tid);

  const float m = ws.m, l = ws.l;
  const int qpos = ws.qpos, h = ws.h;
  // every live row has its own key, so lo > 0 unless this part of a split
  // row selected nothing (then O, lo are 0 and the part weighs nothing)
  const float inv = ws.lo > 0.0f ? 1.0f / ws.lo : 0.0f;
  if (w.part < 0) {
    if (qpos >= 0) {
      uint16_t* orow = reinterpret_cast<uint16_t*>(a.o) + (int64_t)qpos * a.o_ss + (int64_t)w.head * a.o_sh;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          bf16x4 t;
#pragma unroll
          for (int j = 0; j < 4; ++j) t[j] = (__bf16)(ws.o[dt][4 * i + j] * inv);
          *reinterpret_cast<bf16x4*>(orow + 32 * dt + 8 * i + 4 * h) = t;
        }
      if (WL && h == 0) a.lse[(int64_t)w.head * a.S + qpos] = (m + fast_log2(l)) * LN2;
    }
  } else {
    const int row = ws.rb * B + half * 32 + ws.c;    // row of the group, 0 .. 64R-1
    float* po = a.part_o + ((int64_t)w.part * (B * R) + row) * D;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float4 t = make_float4(ws.o[dt][4 * i] * inv, ws.o[dt][4 * i + 1] * inv, ws.o[dt][4 * i + 2] * inv,
                               ws.o[dt][4 * i + 3] * inv);
        *reinterpret_cast<float4*>(po + 32 * dt + 8 * i + 4 * h) = t;
      }
    if (h == 0) {
      float* ml = a.part_ml + ((int64_t)w.part * (B * R) + row) * 4;
      ml[0] = m;
      ml[1] = ws.lo;
      ml[2] = WL ? l : 0.0f;
    }
  }
}

// Merge the partials of a split row group in a fixed order; each partial
// O_p is already normalised by its own bf16-P sum lo_p and weighs
// w_p = lo_p 2^(m_p - M): M = max m_p, O = sum w_p O_p / sum w_p (the O of
// the unsplit row), LSE = M + log2 sum l_p 2^(m_p - M) in natural-log units.
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
  for (int p = 0; p < sr.nparts; ++p) M = fmaxf(M, a.part_ml[((int64_t)(sr.part0 + p) * stride + row) * 4]);
  float acc[32];
#pragma unroll
  for (int x = 0; x < 32; ++x) acc[x] = 0.0f;
  float L = 0.0f, Ll = 0.0f;
  for (int p = 0; p < sr.nparts; ++p) {
    const int64_t pr = (int64_t)(sr.part0 + p) * stride + row;
    const float e = fast_exp2(a.part_ml[pr * 4] - M);
    const float wgt = a.part_ml[pr * 4 + 1] * e;
    L += wgt;
    Ll += a.part_ml[pr * 4 + 2] * e;
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
  if (quarter == 0 && a.lse) a.lse[(int64_t)sr.head * a.S + qpos] = (M + fast_log2(Ll)) * LN2;
}

hipError_t launch_attention(const AttnArgs& a, hipStream_t st) {
  if (a.nitems <= 0) return hipSuccess;
  const int64_t grid = 8 * a.map_len;
  const bool wl = a.lse != nullptr;      // the fp32-P row sums only when the LSE is asked for
  switch (a.R * 2 + (wl ? 1 : 0)) {
    case 2: hipLaunchKernelGGL((k_attention<1, false>), dim3((unsigned)grid), dim3(128), 0, st, a); break;
    case 3: hipLaunchKernelGGL((k_attention<1, true>), dim3((unsigned)grid), dim3(128), 0, st, a); break;
    case 4: hipLaunchKernelGGL((k_attention<2, false>), dim3((unsigned)grid), dim3(256), 0, st, a); break;
    case 5: hipLaunchKernelGGL((k_attention<2, true>), dim3((unsigned)grid), dim3(256), 0, st, a); break;
    case 8: hipLaunchKernelGGL((k_attention<4, false>), dim3((unsigned)grid), dim3(512), 0, st, a); break;
    case 9: hipLaunchKernelGGL((k_attention<4, true>), dim3((unsigned)grid), dim3(512), 0, st, a); break;
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
