// Block-sparse causal attention over permuted 64x64 blocks (Algorithms 5-7:
// the Grid, Q-Boundary and 2D-Boundary FlashAttention kernels are one
// kernel here, because the permutation and the selected key blocks are data:
// qperm / kperm say which token each slot holds, the block index says which
// key blocks each query block visits).
//
// One work item = a row group of R permuted query blocks and a contiguous
// range of the union of their key-block lists; each union entry carries one
// select flag and one mask flag per query block. Every key block of the
// range is loaded once into LDS and used by all members that selected it.
// A wave owns QT x 32 query rows of one member (QT = 2: one wave per
// member, one wave per SIMD; QT = 1: two waves per member). Per key block
// and 32-query tile of an active wave:
//   S^T (64 keys x 32 queries) = K Q^T         16 MFMA 32x32x16 bf16
//   mask by original positions (k <= q) where the block reaches past the
//   member's first query, online softmax in fp32 (log2 domain)
//   O^T (128 x 32) += V^T P^T                  16 MFMA 32x32x16 bf16
// S^T puts one query per lane: row max/sum need one cross-lane exchange and
// the accumulator is already the P operand of the PV product. With QT = 2
// each K and V operand read from LDS feeds two MFMAs.
//
// Pipeline: K/V blocks rotate through four LDS stages with one barrier per
// block. Step t multiplies P(t)V(t), turns the scores of block t+1 into
// P(t+1) and computes the scores of block t+2; these three pieces share no
// data, and they are written out interleaved (an MFMA, then a share of the
// softmax) because the vector ALU only overlaps MFMAs of its own wave. The
// global loads of block t+4 are in flight meanwhile.
// V stays row-major in LDS and is read into the PV operand with the gfx950
// transpose read (ds_read_b64_tr_b16): in each 16-lane group, output lane i,
// element e is element i%4 of the 8-byte row addressed by lane 4e + i/4.
//
// The running maximum is only moved when a row's block maximum exceeds it by
// more than RESCALE_SLACK (log2 units): P entries then stay below 2^8, which
// neither bf16 nor the fp32 sums mind, and the O rescale becomes rare.
#include "device.hpp"
#include "internal.hpp"

namespace mmi {

constexpr int NSTAGE = 4;
constexpr float RESCALE_SLACK = 8.0f;
constexpr uint32_t REGION = B * 256;          // bytes of K (or V) per stage: 64 rows x 256 B

// LDS: K of the four stages, then V of the four stages (so that every
// operand read reaches its stage with an immediate offset below 64 KB),
// then the original key positions (INT_BIG for padding). K/V rows are 256
// bytes; their 16-byte chunks are XOR-swizzled, chunk c of row r at
// c ^ swz(r), so that the 16-byte K operand reads (one chunk of 16
// consecutive rows) and the transpose V reads (4 chunks of 4 consecutive
// rows) hit all 64 banks once.
struct Smem {
  uint8_t k[NSTAGE][REGION];
  uint8_t v[NSTAGE][REGION];
  int32_t kpos[NSTAGE][B];
};

__device__ __forceinline__ uint32_t swz(uint32_t r) { return ((r & 3u) << 2) | ((r >> 2) & 3u); }

// Load of plan data through a global-address-space pointer (a generic one
// would become a flat load, which also counts against the LDS wait counter).
__device__ __forceinline__ int ld_global(const int32_t* p) {
  return *(const __attribute__((address_space(1))) int32_t*)(p);
}

__device__ __forceinline__ int slot_pos(const int32_t* perm, int slot, int S) {
  return perm ? ld_global(perm + slot) : (slot < S ? slot : -1);
}

template <int R, int QT>
struct Tile {
  static constexpr int NW = 2 * R / QT;        // waves
  static constexpr int J = 16 / NW;            // 4-row groups of a block each wave loads
};

// K/V of one block go from global memory straight to LDS (buffer loads
// with the LDS flag): a wave instruction fills 1 KB = 4 rows, lane l
// writing physical chunk l % 16 of row l / 16, so it fetches logical chunk
// (l % 16) ^ swz(row). Wave w loads rows 4(wJ + j) + l/16, j < J. K and V
// of the KV head are buffer resources; a row's byte offset is one 24-bit
// multiply-add (positions below 2^21, S x token stride in bytes below 2^32,
// checked on the host). Padding rows use an offset past the resource size,
// for which the hardware returns zeros.
template <int J>
struct KeySrc {
  __amdgpu_buffer_rsrc_t kr, vr;
  uint32_t kss, vss;          // token strides in bytes
  uint32_t lcb[J];            // logical chunk offset (bytes) this lane fetches for group j
  const int32_t* perm;
  int S, row0;                // row of group 0 for this lane
  __device__ __forceinline__ void init(const AttnArgs& a, const HeadDev& hd, int wave, int lane) {
    const uint16_t* kb = reinterpret_cast<const uint16_t*>(a.k.p) + (int64_t)hd.kvh * a.k.sh;
    const uint16_t* vb = reinterpret_cast<const uint16_t*>(a.v.p) + (int64_t)hd.kvh * a.v.sh;
    kss = (uint32_t)a.k.ss * 2u;
    vss = (uint32_t)a.v.ss * 2u;
    kr = __builtin_amdgcn_make_buffer_rsrc((void*)kb, (short)0, (int)((uint32_t)(a.S - 1) * kss + 2u * D), 0x00020000);
    vr = __builtin_amdgcn_make_buffer_rsrc((void*)vb, (short)0, (int)((uint32_t)(a.S - 1) * vss + 2u * D), 0x00020000);
    perm = hd.kperm;
    S = a.S;
    row0 = 4 * (wave * J) + (lane >> 4);
#pragma unroll
    for (int j = 0; j < J; ++j) lcb[j] = (((uint32_t)lane & 15u) ^ swz((uint32_t)(row0 + 4 * j))) << 4;
  }
};

// Original positions of this lane's rows of key block jblk (-1 = padding).
template <int J, bool PERM>
__device__ __forceinline__ void fetch_pos(int (&kp)[J], const KeySrc<J>& ks, int jblk) {
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int slot = jblk * B + ks.row0 + 4 * j;
    kp[j] = PERM ? ld_global(ks.perm + slot) : (slot < ks.S ? slot : -1);
  }
}

typedef __attribute__((address_space(3))) void lds_void;

// Start the loads of one key block into stage st (positions from fetch_pos).
template <int J>
__device__ __forceinline__ void load_block(Smem& sm, int st, const KeySrc<J>& ks, const int (&kp)[J], int wave,
                                           int lane) {
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const uint32_t g = 4u * (uint32_t)(wave * J + j);           // first row of the instruction
    const bool pad = kp[j] < 0;
    const uint32_t row = pad ? 0u : (uint32_t)kp[j];
    const uint32_t ko = pad ? 0xFFFFFFF0u : __umul24(row, ks.kss) + ks.lcb[j];
    const uint32_t vo = pad ? 0xFFFFFFF0u : __umul24(row, ks.vss) + ks.lcb[j];
    __builtin_amdgcn_raw_ptr_buffer_load_lds(ks.kr, (lds_void*)&sm.k[st][g * 256u], 16, (int)ko, 0, 0, 0);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(ks.vr, (lds_void*)&sm.v[st][g * 256u], 16, (int)vo, 0, 0, 0);
    if ((lane & 15) == 0) sm.kpos[st][ks.row0 + 4 * j] = pad ? INT_BIG : kp[j];
  }
}

// Wait until this wave's LDS loads have landed (vmcnt 0; the other counters
// left alone).
__device__ __forceinline__ void wait_loads() { __builtin_amdgcn_s_waitcnt(0x0F70); }

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
// turn. Runs of XCD_RUN consecutive items go to one XCD, and the runs are
// interleaved across XCDs, so neighbouring row groups (which share key
// blocks) meet in one L2 while heavy and light heads stay spread out.
constexpr int XCD_RUN = 16;

__device__ __forceinline__ int64_t item_of_block(int64_t b) {
  const int64_t xcd = b & 7, k = b >> 3;
  return (k / XCD_RUN) * (8 * XCD_RUN) + xcd * XCD_RUN + (k % XCD_RUN);
}

typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

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

// Per-wave state: QT tiles of 32 queries, and this lane's operand read
// offsets in stage 0 (K: one per 16-dim step st8; V: one per 32-row tile dt
// of O^T and per 8-row half of the transpose read).
template <int QT>
struct WaveState {
  f32x16 o[QT][4];
  bf16x8 qr[QT][8];
  float m[QT], l[QT];
  int qpos[QT];
  int rb, h;
  uint32_t koff[8];
  uint32_t voff[4][2];
};

// Operand read offsets. K: lane (c, h) needs dims 64h + 8 st8 .. +7 of key
// row c (+32 for the second key tile), logical chunk 8h + st8. V (transpose
// read): in 16-lane group grp, lane li addresses row 4(grp/2) + li/4 (+8 for
// the upper half, +16 / +32 per key step), bytes 32(grp%2) + 8(li%4) + 64dt.
template <int QT>
__device__ __forceinline__ void operand_offsets(WaveState<QT>& ws, int lane) {
  const uint32_t c = lane & 31, h = lane >> 5;
#pragma unroll
  for (int st8 = 0; st8 < 8; ++st8) ws.koff[st8] = c * 256u + (((h * 8u + st8) ^ swz(c)) << 4);
  const uint32_t grp = lane >> 4, li = lane & 15;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int hi = 0; hi < 2; ++hi) {
      const uint32_t row = (li >> 2) + 4 * (grp >> 1) + 8 * hi;
      const uint32_t byte = 32 * (grp & 1) + 8 * (li & 3) + 64 * dt;
      ws.voff[dt][hi] = row * 256u + (((byte >> 4) ^ swz(row)) << 4) + (byte & 15);
    }
}

// A operands of a block in stage st: K rows (QK, unit u = 2*st8 + kt) and
// transposed V (PV, unit u = 4*stp + dt), each used by the QT tiles.
template <int QT>
__device__ __forceinline__ bf16x8 k_operand(const Smem& sm, int st, const WaveState<QT>& ws, int u) {
  const int st8 = u >> 1, kt = u & 1;
  return *reinterpret_cast<const bf16x8*>(&sm.k[st][ws.koff[st8] + kt * 32 * 256]);
}

template <int QT>
__device__ __forceinline__ bf16x8 v_operand(const Smem& sm, int st, const WaveState<QT>& ws, int u) {
  const int stp = u >> 2, dt = u & 3, kt = stp >> 1, half = stp & 1;
  const uint32_t rows = (32 * kt + 16 * half) * 256;
  const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)&sm.v[st][ws.voff[dt][0] + rows]);
  const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)&sm.v[st][ws.voff[dt][1] + rows]);
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

// S^T tiles (keys 0-31 and 32-63 of the block, each query tile) of a block.
template <int QT>
__device__ __forceinline__ void qk_block(const Smem& sm, int st, const WaveState<QT>& ws, f32x16 (&s)[QT][2]) {
  const f32x16 zero = {};
#pragma unroll
  for (int u = 0; u < 16; ++u) {
    const bf16x8 ka = k_operand(sm, st, ws, u);
    const int st8 = u >> 1, kt = u & 1;
#pragma unroll
    for (int q = 0; q < QT; ++q) s[q][kt] = mfma32(ka, ws.qr[q][st8], st8 == 0 ? zero : s[q][kt]);
  }
}

// O^T += V^T P^T for each query tile.
template <int QT>
__device__ __forceinline__ void pv_block(const Smem& sm, int st, WaveState<QT>& ws, const bf16x8 (&p)[QT][4]) {
#pragma unroll
  for (int u = 0; u < 16; ++u) {
    const bf16x8 va = v_operand(sm, st, ws, u);
    const int stp = u >> 2, dt = u & 3;
#pragma unroll
    for (int q = 0; q < QT; ++q) ws.o[q][dt] = mfma32(va, p[q][stp], ws.o[q][dt]);
  }
}

__device__ __forceinline__ void mask_tile(const Smem& sm, int st, int qpos, int h, f32x16 (&s)[2]) {
#pragma unroll
  for (int kt = 0; kt < 2; ++kt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int4 kp = *reinterpret_cast<const int4*>(&sm.kpos[st][kt * 32 + 8 * i + 4 * h]);
      if (kp.x > qpos) s[kt][4 * i + 0] = -INFINITY;
      if (kp.y > qpos) s[kt][4 * i + 1] = -INFINITY;
      if (kp.z > qpos) s[kt][4 * i + 2] = -INFINITY;
      if (kp.w > qpos) s[kt][4 * i + 3] = -INFINITY;
    }
}

// Softmax of one tile cut into pieces that can be spread between MFMAs:
// 0-3 running maximum over 8 scores each, 4 new maximum, 5-36 one
// exponential each, 37-40 bf16 packing, 41 row sum. Branch-free.
constexpr int SM_PIECES = 42;

struct SoftmaxState {
  float mx, m_new, rs;
};

__device__ __forceinline__ void softmax_piece(int pc, f32x16 (&s)[2], float sc, float& m, float& l,
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
  } else if (pc < 37) {
    const int e = pc - 5, kt = e >> 4, x = e & 15;
    const float p = fast_exp2(fmaf(s[kt][x], sc, -st.m_new));
    s[kt][x] = p;
    st.rs += p;
  } else if (pc < 41) {
    const int stp = pc - 37, kt = stp >> 1, half = stp & 1;
#pragma unroll
    for (int x = 0; x < 8; ++x) pb[stp][x] = (__bf16)s[kt][4 * (2 * half + (x >> 2)) + (x & 3)];
  } else {
    l = l * alpha + xhalf_sum(st.rs);
  }
}

// The three pieces of step t that share no data: QK(t+2) and PV(t) on the
// matrix cores, softmax(t+1) on the vector ALU, written out interleaved
// (MFMA slot I, then its share of the softmax pieces). Operands are read
// from LDS three units ahead. Slots are unrolled by template recursion so
// that every register-array index is a compile-time constant.
template <int QT, bool QK, bool PV>
struct Fused {
  static constexpr int NQU = QK ? 16 : 0;          // operand units
  static constexpr int NU = NQU + (PV ? 16 : 0);
  static constexpr int NM = NU * QT;               // MFMA slots
  static constexpr int NP = SM_PIECES * QT;        // softmax pieces
  static constexpr int AHEAD = 3;

  WaveState<QT>& ws;
  const Smem& sm;
  int kst, vst;
  f32x16 (&s_qk)[QT][2];
  const bf16x8 (&p_cur)[QT][4];
  f32x16 (&s_sm)[QT][2];
  bf16x8 (&p_new)[QT][4];
  float sc;
  float (&alpha)[QT];
  SoftmaxState st[QT];
  bf16x8 opa[AHEAD + 1];

  __device__ __forceinline__ bf16x8 operand(int u) {
    return u < NQU ? k_operand(sm, kst, ws, u) : v_operand(sm, vst, ws, u - NQU);
  }

  template <int P>
  __device__ __forceinline__ void piece() {
    constexpr int sq = P / SM_PIECES;
    softmax_piece(P % SM_PIECES, s_sm[sq], sc, ws.m[sq], ws.l[sq], p_new[sq], alpha[sq], st[sq]);
  }

  template <int P, int PE>
  __device__ __forceinline__ void pieces() {
    if constexpr (P < PE) {
      piece<P>();
      pieces<P + 1, PE>();
    }
  }

  template <int I>
  __device__ __forceinline__ void slot() {
    if constexpr (I < NM) {
      constexpr int u = I / QT, q = I % QT;
      if constexpr (q == 0 && u + AHEAD < NU) opa[(u + AHEAD) % (AHEAD + 1)] = operand(u + AHEAD);
      const bf16x8 av = opa[u % (AHEAD + 1)];
      if constexpr (u < NQU) {
        constexpr int st8 = u >> 1, kt = u & 1;
        if constexpr (st8 == 0) s_qk[q][kt] = mfma32(av, ws.qr[q][st8], f32x16{});
        else s_qk[q][kt] = mfma32(av, ws.qr[q][st8], s_qk[q][kt]);
      } else {
        constexpr int w = u - NQU, stp = w >> 2, dt = w & 3;
        ws.o[q][dt] = mfma32(av, p_cur[q][stp], ws.o[q][dt]);
      }
      pieces<I * NP / NM, (I + 1) * NP / NM>();
      // keep the slot boundaries: unconstrained, the scheduler hoists all
      // operand reads and runs out of registers
      __builtin_amdgcn_sched_barrier(0);
      slot<I + 1>();
    }
  }

  __device__ __forceinline__ void run() {
#pragma unroll
    for (int u = 0; u < AHEAD && u < NU; ++u) opa[u] = operand(u);
    if constexpr (NM > 0) slot<0>();
    else pieces<0, NP>();
  }
};

template <int QT, bool QK, bool PV>
__device__ __forceinline__ void fused_step(WaveState<QT>& ws, const Smem& sm, int kst, int vst,
                                           f32x16 (&s_qk)[QT][2], const bf16x8 (&p_cur)[QT][4],
                                           f32x16 (&s_sm)[QT][2], bf16x8 (&p_new)[QT][4], float sc,
                                           float (&alpha)[QT]) {
  Fused<QT, QK, PV> f{ws, sm, kst, vst, s_qk, p_cur, s_sm, p_new, sc, alpha, {}, {}};
  f.run();
}

__device__ __forceinline__ bool sel(int e, int rb) { return (e >> (16 + rb)) & 1; }
__device__ __forceinline__ bool needs_mask(int e, int rb) { return (e >> (24 + rb)) & 1; }

// Step t. Entries e0..e2 are the union entries t..t+2 (0 past the end): key
// block in bits 0-15, per-member select flags from bit 16, per-member mask
// flags from bit 24. On entry: P(t) in p_cur, the scores of block t+1 in
// s_sm, blocks t..t+2 in their stages, kp3 / kp4 the key positions of
// blocks t+3 / t+4. The step starts loading block t+3 into its stage (last
// read in step t-1), multiplies P(t)V(t), turns the scores of t+1 into
// P(t+1) (p_new), computes the scores of t+2 into s_qk, waits for its loads
// and fetches the positions of block t+5 into kp3.
template <int R, int QT, bool PERM>
__device__ __forceinline__ void block_step(WaveState<QT>& ws, Smem& sm, const KeySrc<Tile<R, QT>::J>& ks,
                                           int (&kp3)[Tile<R, QT>::J], int wave, int lane, int t, int n, int e0,
                                           int e1, int e2, int e5, f32x16 (&s_qk)[QT][2],
                                           const bf16x8 (&p_cur)[QT][4], f32x16 (&s_sm)[QT][2],
                                           bf16x8 (&p_new)[QT][4], float sc) {
  constexpr int J = Tile<R, QT>::J;
  if (t + 3 < n) load_block<J>(sm, (t + 3) & (NSTAGE - 1), ks, kp3, wave, lane);
  const bool a0 = sel(e0, ws.rb);
  const bool a1 = t + 1 < n && sel(e1, ws.rb);
  const bool a2 = t + 2 < n && sel(e2, ws.rb);
  const int vst = t & (NSTAGE - 1), kst = (t + 2) & (NSTAGE - 1);
  float alpha[QT];
#pragma unroll
  for (int q = 0; q < QT; ++q) alpha[q] = 1.0f;
  if (a1) {
    if (needs_mask(e1, ws.rb)) {
#pragma unroll
      for (int q = 0; q < QT; ++q) mask_tile(sm, (t + 1) & (NSTAGE - 1), ws.qpos[q], ws.h, s_sm[q]);
    }
    if (a2 && a0) fused_step<QT, true, true>(ws, sm, kst, vst, s_qk, p_cur, s_sm, p_new, sc, alpha);
    else if (a2) fused_step<QT, true, false>(ws, sm, kst, vst, s_qk, p_cur, s_sm, p_new, sc, alpha);
    else if (a0) fused_step<QT, false, true>(ws, sm, kst, vst, s_qk, p_cur, s_sm, p_new, sc, alpha);
    else fused_step<QT, false, false>(ws, sm, kst, vst, s_qk, p_cur, s_sm, p_new, sc, alpha);
  } else {
    if (a2) qk_block(sm, kst, ws, s_qk);
    if (a0) pv_block(sm, vst, ws, p_cur);
  }
  // O holds P(t)V(t) relative to the old maximum: move it to the new one
  if (a1) {
#pragma unroll
    for (int q = 0; q < QT; ++q)
      if (__any(alpha[q] != 1.0f)) {
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
#pragma unroll
          for (int x = 0; x < 16; ++x) ws.o[q][dt][x] *= alpha[q];
      }
  }
  wait_loads();
  if (t + 5 < n) fetch_pos<J, PERM>(kp3, ks, e5 & 0xffff);
  __syncthreads();
}

template <int R, int QT, bool PERM>
__device__ __forceinline__ void block_loop(WaveState<QT>& ws, Smem& sm, const AttnArgs& a, const HeadDev& hd,
                                           const WorkItem& w, int wave, int lane) {
  constexpr int J = Tile<R, QT>::J;
  KeySrc<J> ks;
  ks.init(a, hd, wave, lane);
  const float sc = 0.08838834764831845f * LOG2E;   // sqrt(1/128) * log2(e)
  const int n = w.e1 - w.e0;
  EntryStream es;
  es.init(hd.gcol + w.e0, n, lane);
  int e0 = es.get(0), e1 = es.get(1), e2 = es.get(2), e3 = es.get(3), e4 = es.get(4);

  // prologue: blocks 0-2 in stages 0-2, positions of blocks 3 and 4
  int ka[J], kb[J];
  const int ep[3] = {e0, e1, e2};
#pragma unroll
  for (int j = 0; j < 3; ++j) {
    if (j < n) {
      fetch_pos<J, PERM>(ka, ks, ep[j] & 0xffff);
      load_block<J>(sm, j, ks, ka, wave, lane);
    }
  }
  if (n > 3) fetch_pos<J, PERM>(ka, ks, e3 & 0xffff);
  if (n > 4) fetch_pos<J, PERM>(kb, ks, e4 & 0xffff);
  wait_loads();
  __syncthreads();

  f32x16 sa[QT][2], sb[QT][2];
  bf16x8 pa[QT][4], pb[QT][4];
  if (sel(e0, ws.rb)) {
    qk_block(sm, 0, ws, sa);
#pragma unroll
    for (int q = 0; q < QT; ++q) {
      if (needs_mask(e0, ws.rb)) mask_tile(sm, 0, ws.qpos[q], ws.h, sa[q]);
      float alpha;
      SoftmaxState st;
#pragma unroll
      for (int pc = 0; pc < SM_PIECES; ++pc) softmax_piece(pc, sa[q], sc, ws.m[q], ws.l[q], pa[q], alpha, st);
    }
  }
  if (n > 1 && sel(e1, ws.rb)) qk_block(sm, 1, ws, sb);
  // two steps per trip so that the buffers swap roles without copies
  for (int t = 0; t < n; t += 2) {
    int e5 = es.get(t + 5);
    block_step<R, QT, PERM>(ws, sm, ks, ka, wave, lane, t, n, e0, e1, e2, e5, sa, pa, sb, pb, sc);
    e0 = e1; e1 = e2; e2 = e3; e3 = e4; e4 = e5;
    if (t + 1 >= n) break;
    e5 = es.get(t + 6);
    block_step<R, QT, PERM>(ws, sm, ks, kb, wave, lane, t + 1, n, e0, e1, e2, e5, sb, pb, sa, pa, sc);
    e0 = e1; e1 = e2; e2 = e3; e3 = e4; e4 = e5;
  }
}

template <int R, int QT>
__global__ __launch_bounds__(128 * R / QT) __attribute__((amdgpu_waves_per_eu(R * 2 / QT >= 8 ? 2 : 1)))
void k_attention(AttnArgs a) {
  __shared__ Smem sm;
  const int64_t it = item_of_block(blockIdx.x);
  if (it >= a.nitems) return;
  const WorkItem w = a.items[it];
  const HeadDev hd = a.heads[w.head];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  WaveState<QT> ws;
  int row0[QT];                    // first row of each tile within the member's query block
  if (QT == 2) {
    // one wave per member
    ws.rb = wave;
    row0[0] = 0;
    row0[QT - 1] = 32;
  } else {
    // waves 0..R-1 own rows 0-31 of member `wave`, waves R..2R-1 rows 32-63 of
    // member (wave - R + R/2) mod R: the two waves sharing a SIMD (wave and
    // wave + 4 for R = 4) serve different members
    const bool upper = wave >= R;
    ws.rb = upper ? (wave - R + R / 2) % R : wave;
    row0[0] = upper ? 32 : 0;
  }
  const int c = lane & 31;
  ws.h = lane >> 5;
  const int qblk = group_row(w.group, ws.rb, R, hd.gp[0]);
  const uint16_t* qb = reinterpret_cast<const uint16_t*>(a.q.p) + (int64_t)w.head * a.q.sh;
#pragma unroll
  for (int q = 0; q < QT; ++q) {
    ws.qpos[q] = qblk < hd.nbq ? slot_pos(hd.qperm, qblk * B + row0[q] + c, a.S) : -1;
    const uint16_t* row = qb + (int64_t)max(ws.qpos[q], 0) * a.q.ss + ws.h * 64;
#pragma unroll
    for (int s = 0; s < 8; ++s) ws.qr[q][s] = ws.qpos[q] >= 0 ? load16(row + 8 * s) : zero8();
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int e = 0; e < 16; ++e) ws.o[q][dt][e] = 0.0f;
    ws.m[q] = NEG_BIG;
    ws.l[q] = 0.0f;
  }
  operand_offsets(ws, lane);
  if (hd.kperm) block_loop<R, QT, true>(ws, sm, a, hd, w, wave, lane);
  else block_loop<R, QT, false>(ws, sm, a, hd, w, wave, lane);

  const int h = ws.h;
#pragma unroll
  for (int q = 0; q < QT; ++q) {
    const float m = ws.m[q], l = ws.l[q];
    const int qpos = ws.qpos[q];
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
            for (int j = 0; j < 4; ++j) t[j] = (__bf16)(ws.o[q][dt][4 * i + j] * inv);
            *reinterpret_cast<bf16x4*>(orow + 32 * dt + 8 * i + 4 * h) = t;
          }
        if (h == 0 && a.lse) a.lse[(int64_t)w.head * a.S + qpos] = (m + fast_log2(l)) * LN2;
      }
    } else {
      const int row = ws.rb * B + row0[q] + c;      // row of the group, 0 .. 64R-1
      float* po = a.part_o + ((int64_t)w.part * (B * R) + row) * D;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float4 t = make_float4(ws.o[q][dt][4 * i], ws.o[q][dt][4 * i + 1], ws.o[q][dt][4 * i + 2],
                                 ws.o[q][dt][4 * i + 3]);
          *reinterpret_cast<float4*>(po + 32 * dt + 8 * i + 4 * h) = t;
        }
      if (h == 0) {
        float* ml = a.part_ml + ((int64_t)w.part * (B * R) + row) * 2;
        ml[0] = m;
        ml[1] = l;
      }
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
  const dim3 g((unsigned)grid);
  if (a.wide) {
    switch (a.R) {
      case 1: hipLaunchKernelGGL((k_attention<1, 2>), g, dim3(64), 0, st, a); break;
      case 2: hipLaunchKernelGGL((k_attention<2, 2>), g, dim3(128), 0, st, a); break;
      case 4: hipLaunchKernelGGL((k_attention<4, 2>), g, dim3(256), 0, st, a); break;
      default: return hipErrorInvalidValue;
    }
  } else {
    switch (a.R) {
      case 1: hipLaunchKernelGGL((k_attention<1, 1>), g, dim3(128), 0, st, a); break;
      case 2: hipLaunchKernelGGL((k_attention<2, 1>), g, dim3(256), 0, st, a); break;
      case 4: hipLaunchKernelGGL((k_attention<4, 1>), g, dim3(512), 0, st, a); break;
      default: return hipErrorInvalidValue;
    }
  }
  return hipGetLastError();
}

hipError_t launch_combine(const AttnArgs& a, const SplitRow* splits, int64_t nsplit, hipStream_t st) {
  if (nsplit <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_combine, dim3((unsigned)nsplit, a.R), dim3(256), 0, st, a, splits);
  return hipGetLastError();
}

}  // namespace mmi
