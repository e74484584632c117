// Internal device-side descriptors and launch entry points of libmmi.
// Host C++ (runtime.hip) fills these records; the kernels in k_*.hip read
// them. Nothing here is part of the public C-ABI (include/mmi.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <stdexcept>
#include <string>

#include "../../include/mmi.h"

namespace mmi {

// Error of a host call: the C entry points turn it into their status code
// and the thread's last-error text.
struct Error : std::runtime_error {
  int code;
  Error(int c, const std::string& m) : std::runtime_error(m), code(c) {}
};

constexpr int B = 64;            // block size (rows and keys)
constexpr int D = 128;           // head dim
constexpr int LASTQ = 64;        // estimation rows
constexpr int FOLD_W = 1024;     // fold row width (max stride)
constexpr int INT_BIG = 0x7fffffff;

// Tensor view: element strides, head dim contiguous.
struct Tensor {
  const void* p;
  int64_t ss, sh;
};

// ---------------------------------------------------------------- layout
struct Segment {      // maximal run of one modality
  int32_t pos;        // first position
  int32_t len;
  int32_t loc;        // index of `pos` inside its modality's position list
  int32_t mod;
};

// ---------------------------------------------------------------- estimation
struct RowSet {       // estimation query rows: positions [row0, row0 + nrows)
  int32_t head, kvh, row0, nrows;
  int32_t nchunks;    // key chunks of pass 1
  float* part;        // [nchunks][64][2] (max, sum) in log2 domain
  float* lse2;        // [64] log2-domain LSE
};

struct EstJob {       // one query set x one key coordinate system
  int32_t head, kvh, row0, nrows, rowset;
  int32_t coord0;     // coordinate of row0 in the key system (u only)
  const int32_t* keymap;  // coordinate -> position, nullptr = identity
  int32_t L_c, ntiles;
  float* v;           // [L_c]
  float* u;           // [L_c] or nullptr
  float* dpart;       // [ntiles][128] or nullptr
};

struct GridJob {      // stride search over one job's v
  const float* v;
  int32_t L_c, lo, hi;   // candidate strides after the 2*s <= L_c cut (hi < lo: none)
  float* fold;        // [hi-lo+1][1024]
  float* score;       // [hi-lo+1]
  int32_t* pick;      // [hi-lo+1] phase of the max
  int32_t* params;    // [4] out: sigma (0 = dense), phase, L_c, nrows
  int32_t nrows;
};

struct TopkJob {
  const float* x;
  int32_t L, n;       // n <= L
  int32_t* out;       // [n] ascending
};

// ---------------------------------------------------------------- plan
struct OpDev {
  int32_t kind;               // MMI_OP_* (GRID may fall back to dense via params)
  int32_t sink, local;
  int32_t use_h, use_v, use_s;
  int32_t stride, bottom;     // SF_FIXED / SF_STRIDED stride; TRISHAPE final queries
  int32_t L;                  // extent of the op's coordinate system
  int32_t kbase, nkblk;       // first key block / number of key blocks of the key group
  const int32_t* params;      // GRID: {sigma, phase}
  const int32_t* vsel; int32_t nv;
  const int32_t* ssel; int32_t ns;
  int2* selpb;                // [nv] position and key block (from kbase) of each selected vertical
  const int32_t* keymap;      // coordinate -> position for VSLASH/VERT (nullptr = identity)
  int32_t kgrid;              // key group is Grid-ordered (VERT into a Grid group)
  const int32_t* kparams;     // that group's {sigma, phase}
  int32_t koff;               // key group slot offset
  int32_t grid[3], win[3], tile[3];   // NATTEN token grid, window, permutation tile
};

struct HeadDev {
  int32_t kind, kvh;
  int32_t causal;             // 0: bidirectional (NATTEN), only padding keys are masked
  int32_t nbq, nbk;           // permuted query / key blocks
  int32_t S;
  int32_t* qperm;             // [nbq*64] or nullptr (identity)
  int32_t* kperm;             // [nbk*64] or nullptr (identity)
  int32_t* kminpos;           // [nbk] smallest key position per key block
  int32_t* kmaxpos;           // [nbk] largest key position per key block (INT_BIG if it holds padding)
  int32_t* counts;            // [nbq]
  int32_t* rowptr;            // [nbq+1]
  uint32_t* bitmap;           // [nbq][nwords]
  int32_t nwords;
  int32_t* col;               // [nnz]
  int32_t op0;                // first OpDev of this head
  // Row groups: R query blocks processed by one work item over the union of
  // their key lists (entries: key block | flags << 16, bit r of the flags =
  // member r selects that key block). Member r of group g is query block
  // (g / rho) * R * rho + g % rho + r * rho; rho is chosen per head.
  int32_t gcap;               // capacity of the per-group arrays (>= groups for any stride)
  int32_t rho_alt[2];         // extra row-stride candidates besides 1, 2, 4, 8 (0 = none)
  int32_t* gp;                // [3] chosen row stride rho, number of groups, index of rho among the candidates
  int32_t* gcount;            // [groups] union sizes
  int32_t* growptr;           // [ngroups+1]
  int32_t* gcol;              // [gnnz] union entries: key block, select flags << 16, mask flags << 24
  int32_t* chunklen;          // [1] union entries per work item for this head (set by the scan)
  int32_t* chunks;            // [ngroups] work items per group
  int32_t* itembase;          // [ngroups] exclusive prefix of chunks
  int32_t* splitoff;          // [ngroups] exclusive prefix of (chunks > 1)
  int32_t* partoff;           // [ngroups] exclusive prefix of chunks over split groups
};

// group table (modalities present, ascending); identical for every boundary head
struct Groups {
  int32_t n;
  int32_t mod[MMI_MAX_MODALITIES];
  int32_t off[MMI_MAX_MODALITIES];    // slot offset (multiple of 64)
  int32_t len[MMI_MAX_MODALITIES];    // |T_m|
  int32_t toff[MMI_MAX_MODALITIES];   // offset of T_m inside the position pool
};

struct QbOrderJob {   // phase order of one Q-Boundary Grid modality's queries
  const int32_t* params;      // the op's {sigma, phase} (sigma <= 1: position order stays)
  int32_t* qperm;             // the head's qperm at the modality group's slot offset
  int32_t mod;                // modality id
  int32_t* cnt;               // [qb_order_chunks(S)] scratch: counts, then offsets
};

struct WorkItem {
  int32_t head, group, e0, e1;   // union entries [e0, e1) of row group `group`
  int32_t part;       // -1: write O directly; else partial slot
  int32_t pad[3];
};

struct SplitRow {     // a row group whose union list is split over several items
  int32_t head, group, part0, nparts;
};

// ---------------------------------------------------------------- launches
// k_layout.hip
// modpos (nullable): [S] modality id of every position
hipError_t launch_positions(const Segment* segs, int nseg, const int32_t* toff_by_mod, int32_t* tpos,
                            uint8_t* modpos, int S, hipStream_t st);
// max_slots >= every head's nbq*64 and nbk*64
hipError_t launch_perms(const HeadDev* heads, int nheads, const OpDev* ops, Groups g,
                        const int32_t* tpos, int S, int max_slots, hipStream_t st);
// after launch_perms: Q-Boundary Grid modalities' queries in phase order
hipError_t launch_qb_order(const QbOrderJob* jobs, int njobs, const uint8_t* modpos, int S, hipStream_t st);
int qb_order_chunks(int S);
// k_estimate.hip
// order: [ngrp][nr] member indices (-1 = none) of the groups that read the
// same keys (row sets of one KV head; jobs of one KV head and key map).
hipError_t launch_est_lse(const RowSet* rs, int nrs, const int32_t* order, int ngrp, int nr, int max_chunks,
                          Tensor q, Tensor k, int chunk_keys, hipStream_t st);
hipError_t launch_est_scores(const EstJob* jobs, int njobs, const int32_t* order, int ngrp, int nr, int max_tiles,
                             const RowSet* rs, Tensor q, Tensor k, hipStream_t st);
hipError_t launch_est_udiag(const EstJob* jobs, int njobs, int max_L, hipStream_t st);
// k_select.hip
hipError_t launch_grid_search(const GridJob* jobs, int njobs, int max_cands, hipStream_t st);
// scr: int32 scratch of topk_scratch_ints(njobs) entries (initialised by the launch)
size_t topk_scratch_ints(int njobs);
hipError_t launch_topk(const TopkJob* jobs, int njobs, int32_t* scr, hipStream_t st);
// k_blocks.hip
hipError_t launch_key_summaries(const HeadDev* heads, int nheads, OpDev* ops, int nops,
                                Groups g, int max_nbk, int max_sel, hipStream_t st);
hipError_t launch_blocks_count(const HeadDev* heads, int nheads, const OpDev* ops, Groups g, int max_nbq,
                               hipStream_t st);
// Chooses each head's row stride rho among 1, 2, 4, 8 and the head's
// rho_alt (smallest total union, ties to the earlier candidate); cand: int64
// scratch [nheads][NRHO]; extra: some head has rho_alt candidates.
constexpr int NRHO = 6;
hipError_t launch_group_stride(const HeadDev* heads, int nheads, int R, int max_groups, int max_nbq, bool extra,
                               int64_t* cand, int32_t* gcnt, hipStream_t st);
hipError_t launch_group_count(const HeadDev* heads, int nheads, const int32_t* gcnt, int max_groups,
                              hipStream_t st);
// totals[head] = {nnz, gnnz, nitems, nsplit, nparts}
constexpr int NTOT = 5;
// Work-item length per head: max(min_chunk, ceil(gnnz_head / items_per_head),
// avg_factor x the head's average group union) (avg_factor 0: no such floor).
hipError_t launch_blocks_scan(const HeadDev* heads, int nheads, int min_chunk, int items_per_head, int avg_factor,
                              int64_t* totals, hipStream_t st);
hipError_t launch_blocks_fill(const HeadDev* heads, int nheads, int max_nbq, int R, int max_groups,
                              hipStream_t st);
// Modelled cost of each work item (its union entries: one staged K/V block
// each, plus one computed block per member that selects it).
hipError_t launch_item_cost(const HeadDev* heads, const WorkItem* items, int64_t nitems, float* cost,
                            hipStream_t st);
hipError_t launch_work_fill(const HeadDev* heads, int nheads, const int64_t* item_base,
                            const int64_t* part_base, const int64_t* split_base, int max_groups,
                            WorkItem* items, SplitRow* splits, hipStream_t st);
// k_attention.hip
struct AttnArgs {
  Tensor q, k, v;
  void* o; int64_t o_ss, o_sh;
  float* lse;                 // [Hq][S] or nullptr
  int32_t S;
  const HeadDev* heads;
  const WorkItem* items;
  int64_t nitems;
  const int32_t* item_map;    // [8][map_len]: work items of each XCD in order, -1 = none
  int64_t map_len;
  float* part_o;              // [nparts][R*64][128], each row normalised by its bf16-P sum
  float* part_ml;             // [nparts][R*64][4]: running max m, bf16-P sum lo, fp32-P sum l, unused
  int32_t R;                  // query blocks per row group (1, 2 or 4)
};
hipError_t launch_attention(const AttnArgs& a, hipStream_t st);
hipError_t launch_combine(const AttnArgs& a, const SplitRow* splits, int64_t nsplit, hipStream_t st);
// k_search.hip: out[h * n_class + c] = sum over x with cls[x] == c of |a[x,h] - b[x,h]|^2
hipError_t launch_sqerr(const void* a, const void* b, int64_t ss, int64_t sh, const uint8_t* cls, int n_class,
                        int S, int H, double* out, hipStream_t st);
// k_permute.hip
hipError_t launch_permute(const void* src, int64_t ss, void* dst, int64_t ds, const int32_t* perm,
                          int64_t n, int64_t row_bytes, int inverse, hipStream_t st);

// k_stats.hip: useful query-key pairs of one head's selected blocks, added to *out
hipError_t launch_pair_count(const HeadDev* heads, int head, int R, int ngroups, unsigned long long* out,
                             hipStream_t st);

// ---------------------------------------------------------------- check.hip
// Host consistency checks of a plan's tables: empty, or the first violation.
std::string check_index(const mmi_index_view& v);
std::string check_work(const mmi_work_view& w);

// The pattern search of Algorithm 4 (search.hip) over plans of this library;
// the problem is already validated, out has prob.Hq entries.
void search_layer(mmi_ctx* ctx, const mmi_problem& prob, const void* q, const void* k, const void* v,
                  const mmi_op* cands, int nc, const mmi_op* xc, int nx, const mmi_op& target, hipStream_t st,
                  mmi_head_cfg* out, mmi_search_report* rep);

}  // namespace mmi
