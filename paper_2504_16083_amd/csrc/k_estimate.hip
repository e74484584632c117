// Online estimate of the attention map from the final queries (Algorithm 1,
// first step; Appendix C.3): A_hat[r, k] = exp(tau q_r.k_k - LSE_r) for
// k <= pos(r), each row normalised over all causal keys of the sequence.
//
// Pass 1 (k_est_lse): per query set and key chunk, running (max, sum) of
//   2^(tau log2e q.k) per row -> partials; k_est_merge folds the chunks in
//   a fixed order into log2-domain LSE.
// Pass 2 (k_est_scores): per query set and run of 64-key tiles of the key
//   coordinate system, A_hat tile through MFMA, then in LDS the column sums
//   (v, written directly: each tile owns its keys) and the 127 diagonal
//   partial sums of the tile; k_est_udiag adds the (at most two) tiles that
//   touch each diagonal offset. Every reduction has a fixed order, so the
//   scores are bitwise reproducible.
// The query rows are contiguous positions [row0, row0+nrows), nrows <= 64,
// and contiguous in the key coordinate system too (coordinate coord0 + r).
// The query sets that read the same keys (pass 1: one KV head; pass 2 also
// one key coordinate system) form a group, and the work of a group over one
// key range runs back to back on one XCD. Pass 1 takes up to four sets of a
// group per workgroup (two waves each, 32 rows per wave, the query rows in
// registers as the MFMA B operand): each 64-key tile is loaded once by all
// 512 threads into LDS (the next tile's rows load while the current one is
// multiplied) and read as the A operand by every set. Pass 2 takes one job
// per workgroup and reads its K rows straight from HBM into MFMA operands,
// each row by one wave (wave w multiplies keys 32 w .. 32 w + 31 of every
// tile by all 64 rows; two tiles of rows in registers: tile t + 2 loads
// while t and t + 1 are multiplied and reduced); the jobs of a group over
// one range find it in that XCD's L2.
#include "device.hpp"
#include "internal.hpp"

namespace mmi {

namespace {

constexpr float SC = 0.08838834764831845f * LOG2E;   // sqrt(1/128) * log2(e)
constexpr int EKP = 136;          // bf16 per staged K row (272 B: conflict-free operand reads)
constexpr int EMEM = 4;           // query sets (LSE pass) or score jobs per workgroup, 2 waves each

// Logical work index of physical workgroup b when runs of `run` consecutive
// logical items go to one XCD (workgroups are dispatched to the 8 XCDs in
// turn) and the runs to XCDs in turn.
__device__ __forceinline__ int64_t run_item(int64_t b, int run) {
  const int64_t xcd = b & 7, k = b >> 3;
  return (k / run) * (8 * (int64_t)run) + xcd * run + (k % run);
}

struct __align__(16) EstStage {
  uint16_t k[B * EKP];
};

__device__ __forceinline__ void load_q_operand(bf16x8 (&qr)[8], const Tensor& q, int head, int pos,
                                               int h) {
  const uint16_t* row = reinterpret_cast<const uint16_t*>(q.p) + (int64_t)head * q.sh +
                        (int64_t)max(pos, 0) * q.ss + h * 64;
#pragma unroll
  for (int s = 0; s < 8; ++s) qr[s] = pos >= 0 ? load16(row + 8 * s) : zero8();
}

// This thread's 32 bytes of key row kpos (zeros for kpos < 0): thread
// (key, part) of the 512 stages dims [16 part, 16 part + 16) of one key.
__device__ __forceinline__ void fetch_key(bf16x8 (&r)[2], const Tensor& k, int kvh, int kpos, int part) {
  const uint16_t* row = reinterpret_cast<const uint16_t*>(k.p) + (int64_t)kvh * k.sh +
                        (int64_t)max(kpos, 0) * k.ss + part * 16;
  r[0] = kpos >= 0 ? load16(row) : zero8();
  r[1] = kpos >= 0 ? load16(row + 8) : zero8();
}

__device__ __forceinline__ void stage_key(EstStage& st, const bf16x8 (&r)[2], int key, int part) {
  *reinterpret_cast<bf16x8*>(&st.k[key * EKP + part * 16]) = r[0];
  *reinterpret_cast<bf16x8*>(&st.k[key * EKP + part * 16 + 8]) = r[1];
}

// S^T of the 64 staged keys x this wave's 32 queries: s[kt] holds keys
// 32 kt + 8i + 4h + j for query c in element 4i + j.
__device__ __forceinline__ void staged_product(const EstStage& st, const bf16x8 (&qr)[8], int c, int h,
                                               f32x16 (&s)[2]) {
  const f32x16 zero = {};
#pragma unroll
  for (int st8 = 0; st8 < 8; ++st8) {
    const bf16x8 k0 = *reinterpret_cast<const bf16x8*>(&st.k[c * EKP + h * 64 + st8 * 8]);
    const bf16x8 k1 = *reinterpret_cast<const bf16x8*>(&st.k[(32 + c) * EKP + h * 64 + st8 * 8]);
    s[0] = mfma32(k0, qr[st8], st8 == 0 ? zero : s[0]);
    s[1] = mfma32(k1, qr[st8], st8 == 0 ? zero : s[1]);
  }
}


// This lane's half of key row kpos (zeros for kpos < 0): the K operand of
// one 32-key S^T tile.
__device__ __forceinline__ void load_key(bf16x8 (&ka)[8], const Tensor& k, int kvh, int kpos, int h) {
  const uint16_t* row = reinterpret_cast<const uint16_t*>(k.p) + (int64_t)kvh * k.sh +
                        (int64_t)max(kpos, 0) * k.ss + h * 64;
#pragma unroll
  for (int s = 0; s < 8; ++s) ka[s] = kpos >= 0 ? load16(row + 8 * s) : zero8();
}

// S^T tile of 32 keys x 32 queries; lane (c, h) holds keys 8i + 4h + j for query c.
__device__ __forceinline__ f32x16 key_product(const bf16x8 (&ka)[8], const bf16x8 (&qr)[8]) {
  f32x16 acc;
#pragma unroll
  for (int x = 0; x < 16; ++x) acc[x] = 0.0f;
#pragma unroll
  for (int s = 0; s < 8; ++s) acc = mfma32(ka[s], qr[s], acc);
  return acc;
}

}  // namespace

// Pass 1. Logical item = (group, key chunk, batch of EMEM members):
// order[group * nr + member] is a row-set index (-1 = none); the row sets
// of a group share one KV head, so every 64-key tile of the chunk is staged
// once in LDS and multiplied by all members' query rows. Waves w and w + 4
// hold rows 0-31 and 32-63 of member w. Per row: running (max, sum) of
// 2^(tau log2e q.k) over its causal keys of the chunk, the fixed order of
// the tiles, then the two key halves of each tile.
__global__ __launch_bounds__(512) void k_est_lse(const RowSet* sets, const int32_t* order, int ngrp, int nr,
                                                 int nbat, int nch, Tensor q, Tensor k, int chunk_keys) {
  __shared__ EstStage stg[2];
  const int64_t lg = run_item(blockIdx.x, nbat);
  const int bat = (int)(lg % nbat);
  const int64_t pair = lg / nbat;
  const int grp = (int)(pair / nch), ch = (int)(pair % nch);
  if (grp >= ngrp) return;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, c = lane & 31, h = lane >> 5;
  int kend = 0;                        // keys [0, kend) are visible to some member
  for (int m = 0; m < EMEM; ++m) {
    const int mi = bat * EMEM + m;
    const int si = mi < nr ? order[grp * nr + mi] : -1;
    if (si >= 0) kend = max(kend, sets[si].row0 + sets[si].nrows);
  }
  const int k0 = ch * chunk_keys;
  if (k0 >= kend) return;
  const int k1 = min(k0 + chunk_keys, kend);
  const int kvh = sets[order[grp * nr]].kvh;
  const int mem = wave & (EMEM - 1), half = wave >> 2;
  const int mi = bat * EMEM + mem;
  const int si = mi < nr ? order[grp * nr + mi] : -1;
  RowSet rs{};
  if (si >= 0) rs = sets[si];
  const bool active = si >= 0 && ch < rs.nchunks;
  const int r = half * 32 + c;
  const int qpos = active && r < rs.nrows ? rs.row0 + r : -1;
  bf16x8 qr[8];
  load_q_operand(qr, q, rs.head, qpos, h);
  const int key = tid >> 3, part = tid & 7;
  const int ntile = (k1 - k0 + B - 1) / B;
  bf16x8 rg[2];
  fetch_key(rg, k, kvh, k0 + key < k1 ? k0 + key : -1, part);
  stage_key(stg[0], rg, key, part);
  if (ntile > 1) fetch_key(rg, k, kvh, k0 + B + key < k1 ? k0 + B + key : -1, part);
  __syncthreads();
  float m = NEG_BIG, l = 0.0f;
  for (int t = 0; t < ntile; ++t) {
    const int kb = k0 + t * B;
    if (active) {
      f32x16 s[2];
      staged_product(stg[t & 1], qr, c, h, s);
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        float mx = NEG_BIG;
        float x[16];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int kk = kb + kt * 32 + 8 * i + 4 * h + j;
            const float v = s[kt][4 * i + j] * SC;
            x[4 * i + j] = (kk < k1 && kk <= qpos) ? v : -INFINITY;
            mx = fmaxf(mx, x[4 * i + j]);
          }
        const float mn = fmaxf(m, mx);
        float acc = 0.0f;
#pragma unroll
        for (int e = 0; e < 16; ++e) acc += fast_exp2(x[e] - mn);
        l = l * fast_exp2(m - mn) + acc;
        m = mn;
      }
    }
    // tile t+1 was loaded during tile t-1; its stage was last read in tile t-1
    if (t + 1 < ntile) {
      stage_key(stg[(t + 1) & 1], rg, key, part);
      const int nk = k0 + (t + 2) * B + key;
      if (t + 2 < ntile) fetch_key(rg, k, kvh, nk < k1 ? nk : -1, part);
    }
    __syncthreads();
  }
  if (!active) return;
  const float m2 = __shfl_xor(m, 32), l2 = __shfl_xor(l, 32);
  const float mt = fmaxf(m, m2);
  const float lt = h == 0 ? l * fast_exp2(m - mt) + l2 * fast_exp2(m2 - mt)
                          : l2 * fast_exp2(m2 - mt) + l * fast_exp2(m - mt);
  if (h == 0 && r < rs.nrows) {
    float* p = rs.part + ((int64_t)ch * LASTQ + r) * 2;
    p[0] = mt;
    p[1] = lt;
  }
}

__global__ __launch_bounds__(64) void k_est_merge(const RowSet* sets) {
  const RowSet rs = sets[blockIdx.x];
  const int r = threadIdx.x;
  if (r >= rs.nrows) return;
  float M = NEG_BIG;
  for (int ch = 0; ch < rs.nchunks; ++ch) M = fmaxf(M, rs.part[((int64_t)ch * LASTQ + r) * 2]);
  float L = 0.0f;
  for (int ch = 0; ch < rs.nchunks; ++ch) {
    const float* p = rs.part + ((int64_t)ch * LASTQ + r) * 2;
    L += p[1] * fast_exp2(p[0] - M);
  }
  rs.lse2[r] = M + fast_log2(L);
}

constexpr int APITCH = 65;   // floats per key row of A_hat in LDS: odd, so that the lanes of the
                             // diagonal sums (one diagonal each) read distinct banks
constexpr int EST_TPW = 8;    // 64-key tiles per workgroup of the score pass

// Each workgroup takes EST_TPW consecutive tiles of one job: the query rows
// are loaded once, and the key positions and K rows of the tile after next
// load while the current tile is reduced. The arithmetic of every tile is the same as
// one tile per workgroup.
// Logical item = (group, run of EST_TPW tiles, member): order[group * nr +
// member] is a job index (-1 = none), nrun runs per group.
__global__ __launch_bounds__(128) __attribute__((amdgpu_waves_per_eu(2))) void k_est_scores(const EstJob* jobs, const int32_t* order, int ngrp, int nr,
                                                    int nrun, const RowSet* sets, Tensor q, Tensor k) {
  __shared__ __align__(16) float ahat[B * APITCH];
  __shared__ int kposl[B];      // key positions of the current tile, INT_BIG past L_c
  const int64_t lg = run_item(blockIdx.x, nr);
  const int64_t pair = lg / nr;
  const int grp = (int)(pair / nrun), tr = (int)(pair % nrun);
  if (grp >= ngrp) return;
  const int ji = order[grp * nr + (int)(lg % nr)];
  if (ji < 0) return;
  const EstJob jb = jobs[ji];
  const int ta = tr * EST_TPW;
  if (ta >= jb.ntiles) return;
  const int tb = min(ta + EST_TPW, jb.ntiles);
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, c = lane & 31, h = lane >> 5;
  // wave w multiplies keys 32 w .. 32 w + 31 of each tile by all 64 rows
  // (each K row is loaded once per workgroup); lane (c, h) holds rows c and
  // 32 + c as B operands
  int qpos[2];
  float lse2[2];
  bf16x8 qr[2][8];
#pragma unroll
  for (int hf = 0; hf < 2; ++hf) {
    const int r = hf * 32 + c;
    qpos[hf] = r < jb.nrows ? jb.row0 + r : -1;
    lse2[hf] = qpos[hf] >= 0 ? sets[jb.rowset].lse2[r] : 0.0f;
    load_q_operand(qr[hf], q, jb.head, qpos[hf], h);
  }
  auto key_pos = [&](int kap) { return kap < jb.L_c ? (jb.keymap ? jb.keymap[kap] : kap) : -1; };
  // two tiles of K rows in registers: tile t + 2 loads while tiles t and t + 1 are used
  int kp[2];
  bf16x8 ka[2][8];
  auto fetch = [&](int buf, int t) {
    kp[buf] = key_pos(t * B + wave * 32 + c);
    load_key(ka[buf], k, jb.kvh, kp[buf], h);
  };
  auto tile = [&](int buf, int t) {
    f32x16 s[2];
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) s[hf] = key_product(ka[buf], qr[hf]);
    if (h == 0) kposl[wave * 32 + c] = kp[buf] >= 0 ? kp[buf] : INT_BIG;
    if (t + 2 < tb) fetch(buf, t + 2);
    __syncthreads();
#pragma unroll
    for (int hf = 0; hf < 2; ++hf)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int kk = wave * 32 + 8 * i + 4 * h + j;   // key index inside the tile
          const int kp2 = kposl[kk];
          const float a = (qpos[hf] >= 0 && kp2 <= qpos[hf]) ? fast_exp2(s[hf][4 * i + j] * SC - lse2[hf]) : 0.0f;
          ahat[kk * APITCH + hf * 32 + c] = a;
        }
    __syncthreads();
    {   // column sums: two threads per key, rows 0-31 and 32-63, then the pair
      const int kk = tid >> 1, half = tid & 1;
      const float* src = &ahat[kk * APITCH + 32 * half];
      float acc = 0.0f;
#pragma unroll
      for (int x = 0; x < 32; ++x) acc += src[x];
      const float other = __shfl_xor(acc, 1);
      const float tot = half == 0 ? acc + other : other + acc;
      const int kap = t * B + kk;
      if (half == 0 && kap < jb.L_c) jb.v[kap] = tot;
    }
    if (jb.dpart) {   // diagonal d = r - kk + 63, d in [0, 127)
      const int d = tid;
      float acc = 0.0f;
      if (d < 127) {
        // rows rr with key rr + 63 - d inside the tile, ascending; the others add 0
#pragma unroll 16
        for (int rr = 0; rr < B; ++rr) {
          const int kk = rr + 63 - d;
          const bool in = kk >= 0 && kk < B;
          const float x = ahat[(in ? kk : 0) * APITCH + rr];
          acc += in ? x : 0.0f;
        }
      }
      jb.dpart[(int64_t)t * 128 + d] = acc;
    }
    __syncthreads();    // ahat and kposl are rewritten by the next tile
  };
  fetch(0, ta);
  if (ta + 1 < tb) fetch(1, ta + 1);
  for (int t = ta; t < tb; t += 2) {
    tile(0, t);
    if (t + 1 < tb) tile(1, t + 1);
  }
}

__device__ __forceinline__ int floordiv(int a, int b) {
  int q = a / b;
  return (a % b != 0 && ((a < 0) != (b < 0))) ? q - 1 : q;
}

// u[o] = sum over tiles t (ascending) of dpart[t][o - coord0 + 64 t + 63].
__global__ __launch_bounds__(256) void k_est_udiag(const EstJob* jobs) {
  const EstJob jb = jobs[blockIdx.x];
  if (!jb.u) return;
  const int o = blockIdx.y * 256 + threadIdx.x;
  if (o >= jb.L_c) return;
  const int base = jb.coord0 - o;
  const int tlo = max(0, -floordiv(-(base - 63), 64));   // ceil((base - 63) / 64)
  const int thi = min(jb.ntiles - 1, floordiv(base + 63, 64));
  float acc = 0.0f;
  for (int t = tlo; t <= thi; ++t) {
    const int d = o - jb.coord0 + 64 * t + 63;
    if (d >= 0 && d < 127) acc += jb.dpart[(int64_t)t * 128 + d];
  }
  jb.u[o] = acc;
}

// Workgroups for ngrp groups x nper items x nr members, rounded up to whole
// runs of nr on each of the 8 XCDs.
static unsigned grouped_grid(int ngrp, int nper, int nr) {
  const int64_t items = (int64_t)ngrp * nper * nr, run = 8 * (int64_t)nr;
  return (unsigned)((items + run - 1) / run * run);
}

hipError_t launch_est_lse(const RowSet* rs, int nrs, const int32_t* order, int ngrp, int nr, int max_chunks,
                          Tensor q, Tensor k, int chunk_keys, hipStream_t st) {
  if (nrs <= 0) return hipSuccess;
  const int nbat = (nr + EMEM - 1) / EMEM;
  hipLaunchKernelGGL(k_est_lse, dim3(grouped_grid(ngrp, max_chunks, nbat)), dim3(512), 0, st, rs, order, ngrp, nr,
                     nbat, max_chunks, q, k, chunk_keys);
  hipLaunchKernelGGL(k_est_merge, dim3(nrs), dim3(64), 0, st, rs);
  return hipGetLastError();
}

hipError_t launch_est_scores(const EstJob* jobs, int njobs, const int32_t* order, int ngrp, int nr, int max_tiles,
                             const RowSet* rs, Tensor q, Tensor k, hipStream_t st) {
  if (njobs <= 0) return hipSuccess;
  const int nrun = (max_tiles + EST_TPW - 1) / EST_TPW;
  hipLaunchKernelGGL(k_est_scores, dim3(grouped_grid(ngrp, nrun, nr)), dim3(128), 0, st, jobs, order, ngrp, nr,
                     nrun, rs, q, k);
  return hipGetLastError();
}

hipError_t launch_est_udiag(const EstJob* jobs, int njobs, int max_L, hipStream_t st) {
  if (njobs <= 0 || max_L <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_est_udiag, dim3(njobs, (max_L + 255) / 256), dim3(256), 0, st, jobs);
  return hipGetLastError();
}

}  // namespace mmi
