/*
 * mmi.h - C-ABI of the MI355X modality-aware permutation sparse attention
 * library (libmmi.so): the pre-filling hot path of MMInference
 * (arXiv 2504.16083).
 *
 * Problem statement (Section 3, Algorithms 1-3): inputs are Q, K, V of one
 * attention layer, the modality type index i_m of every token and the
 * per-head pattern chosen offline (Algorithm 4 outputs it; here it is an
 * input); the output is the attention output y (and optionally each row's
 * log-sum-exp). For each head the library estimates the pattern parameters
 * online from the last queries, builds the Q/K/V permutation and the block
 * index, runs a block-sparse causal FlashAttention-style kernel over the
 * selected 64x64 blocks and writes the output back in original token order.
 *
 * Conventions shared by every entry point:
 *   - All functions return an int status (MMI_OK or a negative MMI_ERR_*).
 *     On error nothing is written to caller buffers; mmi_last_error() gives
 *     a thread-local message. No C++ exception crosses this boundary.
 *   - Tensor pointers are DEVICE pointers owned by the caller; the library
 *     never frees them nor keeps them past the call that receives them.
 *     Work is enqueued asynchronously on the caller's HIP stream
 *     (hipStream_t passed as void*, NULL = the default stream); every
 *     argument is validated on the host before the first launch.
 *   - Shapes: one layer, batch 1, head_dim D = 128, block size 64, causal,
 *     bfloat16 Q/K/V/O. Hq query heads share Hkv KV heads (GQA): query head
 *     h reads KV head h / (Hq / Hkv). Element strides are given per token
 *     and per head; the head dimension must be contiguous and every row
 *     16-byte aligned. Stride 0 means the packed [S, H, 128] layout.
 *     S times the K or V token stride must stay below 2^31 elements, and
 *     the K and V token strides themselves below 2^23 elements.
 *   - The output O must not alias Q, K or V. A plan is not thread-safe.
 */
#ifndef MMI_H
#define MMI_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MMI_ABI_VERSION 1
#define MMI_MAX_MODALITIES 8
#define MMI_HEAD_DIM 128
#define MMI_BLOCK 64
#define MMI_LAST_Q 64          /* estimation rows, Section 4.1 (last_q = 64) */
#define MMI_MAX_STRIDE 1024    /* Grid max stride, Appendix C.5 table */
#define MMI_MAX_SEQ (1 << 21)  /* largest supported S (2,097,152 tokens) */
/* Device scratch of mmi_attention_noalloc: a static array of this many bytes
 * that each GPU the library runs on holds until the process ends. */
#define MMI_NOALLOC_SCRATCH_BYTES ((size_t)256 << 20)

/* status codes */
#define MMI_OK 0
#define MMI_ERR_INVALID_ARG -1  /* NULL pointer, negative size, bad stride  */
#define MMI_ERR_UNSUPPORTED -2  /* D != 128, block != 64, Hq % Hkv != 0, S too large */
#define MMI_ERR_BAD_CONFIG -3   /* an op/head kind or parameter out of range */
#define MMI_ERR_OOM -4          /* device allocation failed */
#define MMI_ERR_HIP -5          /* a HIP runtime call failed (text in mmi_last_error) */
#define MMI_ERR_STATE -6        /* call out of order (e.g. export before create) */
#define MMI_ERR_INTERNAL -7

/* Op kinds. One op describes a token predicate pred(q, k) in one coordinate
 * system; the selected blocks are the causal block lift of it (see
 * mmi_plan_create). */
#define MMI_OP_NONE 0    /* no key selected (2D-Boundary cross pairs only) */
#define MMI_OP_DENSE 1   /* every causal key */
#define MMI_OP_ASHAPE 2  /* k < sink or q - k < local (Appendix C.3)                */
#define MMI_OP_VSLASH 3  /* k in top-n_vertical columns or q - k in top-n_slash      */
                         /* diagonals of the estimate (Appendix C.3)                */
#define MMI_OP_GRID 4    /* Grid head (Algorithm 1): stride/phase searched over      */
                         /* [stride_lo, stride_hi]; q = k (mod s) if use_s, k = p   */
                         /* (mod s) if use_v, q = p (mod s) if use_h                */
#define MMI_OP_VERT 5    /* k in the top-n_vertical key columns of the key modality, */
                         /* estimated from the query modality's final queries        */
                         /* (2D-Boundary cross pairs only)                            */
/* Static baseline patterns (Section 4.1 "Baselines"; Appendix, table of baseline
 * hyperparameters). No estimation; same coordinates as ASHAPE. */
#define MMI_OP_SF_FIXED 6    /* Sparse Transformer, fixed: floor(q/local) == floor(k/local) */
                             /* (same segment) or k = 0 (mod stride_lo) (segment heads)     */
#define MMI_OP_SF_STRIDED 7  /* Sparse Transformer, strided: q - k < local or              */
                             /* q - k = 0 (mod stride_lo)                                   */
#define MMI_OP_TRISHAPE 8    /* A-shape plus every key for the final `bottom` queries:     */
                             /* k < sink or q - k < local or q >= L - bottom (L = extent   */
                             /* of the op's coordinates: S, or the modality's length)      */
/* Neighborhood attention over a token grid (Appendix F: the 2D/3D sliding windows
 * of DiT models made block-dense by a permutation). Global heads only; the one
 * bidirectional op (no k <= q condition). Tokens form a grid_t x grid_h x grid_w
 * grid in raster order (position (t*grid_h + h)*grid_w + w; grid_t = 1 for
 * images). Along an axis of length n with odd window k, coordinate c sees the k
 * coordinates from min(max(c - k/2, 0), n - k). Queries and keys are permuted
 * tile by tile (tile_t x tile_h x tile_w = 64 tokens, tiles and the tokens inside
 * a tile in raster order, border tiles padded), so tile i is block i; query tile
 * i selects every key tile that meets the union of its tokens' windows. */
#define MMI_OP_NATTEN 9

/* Head kinds. */
#define MMI_HEAD_GLOBAL 0     /* one op over all rows: No-Boundary / K-Boundary (Sec. 3.2) */
#define MMI_HEAD_QBOUNDARY 1  /* Algorithm 2: queries grouped by modality, op per modality */
#define MMI_HEAD_2D 2         /* Algorithm 3: Q and K grouped by modality, op per pair    */
/* No-Boundary and K-Boundary heads (Section 3.2; Appendix B.1): the sparse
 * index stays continuous along the query axis, so the head's intra-modality
 * op applies to all rows at no extra cost. Both names are the global kind. */
#define MMI_HEAD_NO_BOUNDARY MMI_HEAD_GLOBAL
#define MMI_HEAD_K_BOUNDARY MMI_HEAD_GLOBAL

typedef struct mmi_op {
  int32_t kind;                  /* MMI_OP_* */
  int32_t sink, local;           /* ASHAPE: sink >= 0, local >= 0 */
  int32_t n_vertical, n_slash;   /* VSLASH (both), VERT (n_vertical); >= 0 */
  int32_t stride_lo, stride_hi;  /* GRID: 1 <= lo <= hi <= MMI_MAX_STRIDE */
  int32_t use_h, use_v, use_s;   /* GRID line flags (0/1) */
  int32_t bottom;                /* TRISHAPE: final queries with full attention, >= 0 */
  int32_t grid_t, grid_h, grid_w;  /* NATTEN: token grid, product == S */
  int32_t win_t, win_h, win_w;     /* NATTEN: odd window per axis, 1 <= win <= grid */
  int32_t tile_t, tile_h, tile_w;  /* NATTEN: permutation tile, each >= 1, product 64; the
                                      number of tiles must not exceed MMI_MAX_SEQ / 64 */
} mmi_op;

typedef struct mmi_head_cfg {
  int32_t kind;                  /* MMI_HEAD_* */
  mmi_op global;                 /* HEAD_GLOBAL: DENSE, ASHAPE, VSLASH, GRID, NATTEN or a static baseline */
  mmi_op intra[MMI_MAX_MODALITIES];
  /* QBOUNDARY: intra[m] in DENSE, ASHAPE, VSLASH, GRID or a static baseline (global
   * positions; VSLASH and GRID estimated from modality m's final queries). A GRID
   * modality's queries are ordered by phase and its keys are read in the Grid order
   * of all S positions: the head's key slots are key layouts of ceil(S/64) blocks
   * each, position order first (if some modality is not GRID), then one Grid order
   * per GRID modality in ascending m. layouts * ceil(S/64) must not exceed
   * MMI_MAX_SEQ / 64 (MMI_ERR_UNSUPPORTED otherwise).
   * 2D: intra[m] in DENSE, ASHAPE, VSLASH, GRID or a static baseline (modality-local
   * coordinates). Static baselines: SF_FIXED, SF_STRIDED (local >= 1, stride_lo >= 1),
   * TRISHAPE (sink, local, bottom >= 0). */
  mmi_op cross[MMI_MAX_MODALITIES][MMI_MAX_MODALITIES];
  /* 2D: cross[mq][mk], mq != mk, in NONE, DENSE, VERT. */
} mmi_head_cfg;

typedef struct mmi_problem {
  int64_t S;                     /* tokens, 1 <= S <= MMI_MAX_SEQ */
  int32_t Hq, Hkv;               /* query / KV heads, Hq % Hkv == 0 */
  int32_t D;                     /* must be 128 */
  int32_t block;                 /* must be 64 */
  int64_t q_stride_s, q_stride_h;  /* element strides; 0,0 = packed [S,Hq,128] */
  int64_t k_stride_s, k_stride_h;  /* packed [S,Hkv,128] */
  int64_t v_stride_s, v_stride_h;
  int64_t o_stride_s, o_stride_h;  /* packed [S,Hq,128] */
  const uint8_t* modality;       /* HOST array [S] of modality ids < n_modalities, or NULL */
  int32_t n_modalities;          /* 1..MMI_MAX_MODALITIES (ignored if modality == NULL) */
} mmi_problem;

typedef struct mmi_ctx mmi_ctx;
typedef struct mmi_plan mmi_plan;

typedef struct mmi_head_stats {
  int32_t kind;                  /* head kind */
  int32_t n_qblocks, n_kblocks;  /* permuted query / key blocks (incl. padding) */
  int64_t nnz_blocks;            /* selected (query block, key block) pairs */
  int64_t causal_blocks;         /* query-block x key-block pairs with a causal element */
  int32_t split_rows;            /* query blocks split across work items */
  int32_t sigma[MMI_MAX_MODALITIES];  /* chosen Grid stride per op slot (0 = not Grid / dense fallback) */
  int32_t phase[MMI_MAX_MODALITIES];
  int32_t group_stride;          /* query-block stride of the attention row groups: 1, 2, 4, 8, or for
                                    NATTEN heads the tile count of a tile row or of a tile layer */
  int64_t loaded_blocks;         /* key blocks staged for this head (sum of the row-group unions) */
  int64_t blocks_by_modality[MMI_MAX_MODALITIES][MMI_MAX_MODALITIES];
  /* selected blocks by [query modality][key modality], a block taking the modality of its
     first token (the selected-block cost per modality and per modality pair that the pattern
     search budgets; query and key blocks are modality-pure in 2D-Boundary heads, query blocks
     in Q-Boundary heads) */
} mmi_head_stats;

/* Stage durations of a plan, from HIP events recorded on the plan's stream
 * (Section 4.5 "Latency" and Appendix E "Latency Breakdown" report latency
 * including the index building).
 * create_* cover mmi_plan_create, attn/combine the last mmi_plan_execute. */
typedef struct mmi_plan_timing {
  float est_ms;        /* estimation passes (row LSE, column/diagonal scores) */
  float select_ms;     /* Grid stride/phase search, vertical/slash top-k */
  float index_ms;      /* permutations, block index, work list (incl. one host sync) */
  float attn_ms;       /* block-sparse attention kernel */
  float combine_ms;    /* merge of split query blocks */
  int64_t computed_blocks;  /* selected 64x64 blocks over all heads */
  int64_t work_items;
  int64_t loaded_blocks;    /* K/V blocks staged by the attention kernel (union entries of all row groups) */
  int64_t device_bytes;     /* device memory the plan holds (its buffers, before allocator rounding) */
} mmi_plan_timing;

/* export kinds for mmi_plan_export (host copies; the call synchronises) */
#define MMI_EXPORT_QPERM 0       /* int32[n_qblocks*64]: slot -> position or -1 */
#define MMI_EXPORT_KPERM 1       /* int32[n_kblocks*64] (Q-Boundary with GRID: the layouts in order) */
#define MMI_EXPORT_ROW_PTR 2     /* int32[n_qblocks+1] */
#define MMI_EXPORT_COL_IDX 3     /* int32[nnz_blocks], ascending within a row */
#define MMI_EXPORT_V_SCORES 4    /* float[L_c]: column scores of the estimate */
#define MMI_EXPORT_U_SCORES 5    /* float[L_c]: diagonal scores */
#define MMI_EXPORT_FOLD 6        /* float[(hi-lo+1)*1024]: Grid fold c_s[p] at [s-lo][p] */
#define MMI_EXPORT_VSEL 7        /* int32[n]: selected vertical coordinates, ascending */
#define MMI_EXPORT_SSEL 8        /* int32[n]: selected slash offsets, ascending */
#define MMI_EXPORT_PARAMS 9      /* int32[4]: {sigma, phase, L_c, n_rows} (sigma 0 = dense) */
#define MMI_EXPORT_EST_LSE 10    /* float[n_rows]: natural-log LSE of the estimation rows */
#define MMI_EXPORT_UNION_PTR 11  /* int32[n_groups+1]: entry offsets of the attention row groups */
#define MMI_EXPORT_UNION 12      /* int32[loaded_blocks]: row-group union entries, per group the key
                                    blocks every member selects, then the others, each ascending:
                                    key block | select bits << 16 | mask bits << 24 (bit r: member r
                                    selects the block / the block holds a key position above member
                                    r's smallest query position, or padding) */

int mmi_version(void);
const char* mmi_status_str(int status);   /* static string, never NULL */
const char* mmi_last_error(void);         /* thread-local detail of the last error */

/* Context: binds a device, owns a cache of device workspace. */
int mmi_ctx_create(int device, mmi_ctx** out);
int mmi_ctx_destroy(mmi_ctx* ctx);

/* Estimation, choices, permutations and block index of every head
 * (Algorithms 1-3 up to the kernel launch). Enqueued on `stream`; the call
 * synchronises once with it (to size the block index). q, k: device
 * tensors described by `prob`; cfgs: host array [Hq]. Block (i, j) is
 * selected iff some query of permuted query block i and key of permuted key
 * block j satisfy k <= q in original positions and the head's predicate, or
 * block j holds the diagonal key of one of block i's queries. The plan owns
 * its device buffers until mmi_plan_destroy. */
int mmi_plan_create(mmi_ctx* ctx, const mmi_problem* prob, const mmi_head_cfg* cfgs,
                    const void* q, const void* k, void* stream, mmi_plan** out);

/* Block-sparse causal attention over the plan (Algorithms 5-7): gathers
 * permuted Q/K/V rows inside the kernel, online softmax in fp32, P rounded
 * to bf16 for the PV product, O written as bf16 (round to nearest even) in
 * original token order. lse: device float [Hq][S] natural-log LSE, or NULL. */
int mmi_plan_execute(mmi_plan* plan, const void* q, const void* k, const void* v,
                     void* o, float* lse, void* stream);

int mmi_plan_stats(mmi_plan* plan, int head, mmi_head_stats* out);

/* Copy one plan array of `head` to host memory. slot selects the op:
 * 0 for a global head, m for modality m (QBOUNDARY / 2D intra), and
 * 8 + mq*8 + mk for a 2D cross pair. If host_dst is NULL or bytes is too
 * small, only *needed is written (and MMI_OK returned if dst is NULL). */
int mmi_plan_export(mmi_plan* plan, int head, int what, int slot, void* host_dst,
                    size_t bytes, size_t* needed);

/* Work of one head (Section 4.1 reports attention FLOPs relative to dense):
 * *computed = query-key pairs in its selected blocks (nnz_blocks x 4096,
 * every pair of a selected block is computed); *useful = those the output
 * uses: live (non-padding) query and key rows, k <= q in original positions
 * (any live pair for a bidirectional head). Synchronises with the plan's
 * stream; the plan is not changed. */
int mmi_plan_pair_counts(mmi_plan* plan, int head, int64_t* useful, int64_t* computed);

/* Stage durations (synchronises with the plan's stream). */
int mmi_plan_timing_get(mmi_plan* plan, mmi_plan_timing* out);

int mmi_plan_destroy(mmi_plan* plan);

/* create + execute + destroy. */
int mmi_attention(mmi_ctx* ctx, const mmi_problem* prob, const mmi_head_cfg* cfgs,
                  const void* q, const void* k, const void* v, void* o, float* lse,
                  void* stream);

/* mmi_attention for callers that cannot allocate device memory (serving
 * loops, harnesses that forbid allocation): the same plan and kernels, but
 * every device buffer of the plan (estimation scores, permutations, block
 * index, work list, split partials) is carved from the library's static
 * scratch of MMI_NOALLOC_SCRATCH_BYTES on the context's device. The call
 * makes no hipMalloc, hipFree, hipHostMalloc or event creation (host heap
 * memory only for the plan's host-side tables) and returns after its work on
 * `stream` has finished. Results are bitwise those of mmi_attention.
 * Returns MMI_ERR_UNSUPPORTED, without writing o or lse, when the plan needs
 * more than the scratch (the message names the limit; mmi_plan_timing_get's
 * device_bytes tells a plan's need). Calls on one device are serialised by
 * the library; the scratch keeps the last call's contents, and every buffer
 * a call reads is written earlier in that same call. */
int mmi_attention_noalloc(mmi_ctx* ctx, const mmi_problem* prob, const mmi_head_cfg* cfgs,
                          const void* q, const void* k, const void* v, void* o, float* lse,
                          void* stream);

/* Every causal block of every head through the same kernel: the dense
 * causal attention baseline on the same GPU. */
int mmi_dense_attention(mmi_ctx* ctx, const mmi_problem* prob, const void* q,
                        const void* k, const void* v, void* o, float* lse, void* stream);

/* Explicit row permutation (the Q/K/V permutation of Algorithms 1-3 done as
 * a separate pass): dst row x = src row perm[x] (perm[x] = -1 -> zero row),
 * for x in [0, n_dst). unpermute: dst row perm[x] = src row x for perm[x] >= 0.
 * Rows are row_bytes long (multiple of 16), strides in bytes, perm is a
 * device int32 array. */
int mmi_permute_rows(const void* src, int64_t src_stride, void* dst, int64_t dst_stride,
                     const int32_t* perm, int64_t n_dst, int64_t row_bytes, void* stream);
int mmi_unpermute_rows(const void* src, int64_t src_stride, void* dst, int64_t dst_stride,
                       const int32_t* perm, int64_t n_src, int64_t row_bytes, void* stream);

/* Objective of the modality-aware pattern search (Appendix A, Algorithm 4:
 * candidates are scored on the attention output): per head and token class,
 * out[h * n_class + c] = sum over positions x with cls[x] == c of
 * sum_d (a[x, h, d] - b[x, h, d])^2, differences in fp32, sums in fp64 in a
 * fixed order (bitwise reproducible). a, b: device bf16 outputs laid out as O
 * in `prob` (o strides; prob->modality is not read); cls: device uint8 [S],
 * positions with cls >= n_class are skipped; out: device double [Hq * n_class],
 * written on `stream`. 1 <= n_class <= MMI_MAX_MODALITIES. */
int mmi_output_sqerr(const mmi_problem* prob, const void* a, const void* b, const uint8_t* cls,
                     int32_t n_class, double* out, void* stream);

/* ------------------------------------------------------------ pattern search
 * Modality-aware offline pattern search (Appendix A, Algorithm 4; the search
 * space of Appendix C.5) for every head of one layer on a calibration sample
 * (q, k, v device bf16 laid out as in `prob`; prob->modality on the host).
 * Every candidate configuration is one plan of this library for all heads,
 * executed on the sample: its cost over a set of query rows is the blocks
 * its plan selects there (mmi_head_stats.blocks_by_modality: the work the
 * attention kernel runs), its error the squared difference of its output
 * from a reference output over those rows (mmi_output_sqerr). A candidate is
 * admissible iff its cost does not exceed the cost of `target` (the FLOPs
 * target pattern, e.g. A-shape with 1k sink and 4k local tokens) over the
 * same rows in the same coordinates; the choice is the admissible candidate
 * of smallest error (the earlier one on equal errors), else the target.
 * With the n modalities present in the sample, in ascending id:
 *   1. intra, per modality m: 2D-Boundary heads whose cross pairs select
 *      nothing, candidate c on every modality; reference: dense intra ops;
 *      rows: modality m.
 *   2. cross, in rounds r = 1 .. n-1: 2D-Boundary heads with the chosen
 *      intra ops, cross candidate x on the pairs (mods[i], mods[(i+r) % n]),
 *      the other pairs DENSE; reference: dense causal attention; cost: the
 *      pair's blocks; budget: mods[i]'s step-1 budget minus the cost of its
 *      chosen intra op; none admissible -> NONE on that pair.
 *   3. inter: the best global op (chosen as in step 1 over all rows, budget
 *      = the global target head's cost), the Q-Boundary head with the chosen
 *      intra ops, the 2D-Boundary head with the chosen intra and cross ops;
 *      the smallest error among those within that budget (in that order on
 *      ties), else the cheapest.
 * cands[n_cands]: intra candidates in table order (n_cands >= 0); xc[n_xc]:
 * cross candidates (NONE, VERT, DENSE); out: host [Hq], the chosen
 * configuration of every head. Builds 8 + 2 n_cands + (n - 1) n_xc plans on
 * `stream` and synchronises with it; allocates device buffers for two
 * outputs (2 S Hq 128 bytes each) for the duration of the call. `report`
 * (or NULL) receives the search's steps: each array may be NULL; the index
 * i is the position of a modality in report->mods. */
typedef struct mmi_search_report {
  int32_t n_mod;                        /* out: modalities present */
  int32_t mods[MMI_MAX_MODALITIES];     /* out: their ids ascending, -1 after n_mod */
  int64_t plans;                        /* out: plans built */
  int64_t* budget1;     /* [Hq][8]: target cost of modality i's rows (step 1) */
  int64_t* step1_cost;  /* [Hq][n_cands][8] */
  double* step1_err;    /* [Hq][n_cands][8] */
  int32_t* intra;       /* [Hq][8]: chosen intra candidate of modality i, -1 = target */
  int64_t* step2_cost;  /* [Hq][7][n_xc][8]: round r-1, candidate x, rows of modality i */
  double* step2_err;    /* [Hq][7][n_xc][8] */
  int32_t* cross;       /* [Hq][8][8]: chosen cross candidate of pair (i, j), -1 = NONE */
  int64_t* budget3;     /* [Hq]: cost of the global target head */
  int64_t* step3g_cost; /* [Hq][n_cands]: global heads, all rows */
  double* step3g_err;   /* [Hq][n_cands] */
  int32_t* global;      /* [Hq]: chosen global candidate, -1 = target */
  int64_t* step3_cost;  /* [Hq][3]: global, Q-Boundary, 2D-Boundary */
  double* step3_err;    /* [Hq][3] */
  int32_t* kind;        /* [Hq]: chosen kind, 0 global, 1 Q-Boundary, 2 2D-Boundary */
} mmi_search_report;

int mmi_search(mmi_ctx* ctx, const mmi_problem* prob, const void* q, const void* k, const void* v,
               const mmi_op* cands, int32_t n_cands, const mmi_op* xc, int32_t n_xc, const mmi_op* target,
               void* stream, mmi_head_cfg* out, mmi_search_report* report);

/* ------------------------------------------------------------ debug checks
 * Host-side consistency checks of a plan's tables: when they pass, every
 * index the attention kernel derives from the tables (permutation slots,
 * key blocks, union entries, work items, partial slots, the per-XCD item
 * map) lies inside its buffers. With MMI_DEBUG=1 in the environment when a
 * context is created, every plan creation of that context runs
 * mmi_plan_check before it returns, and every execute synchronises with its
 * stream and reports a failed launch itself. A violation returns
 * MMI_ERR_INTERNAL; mmi_last_error names the table, head, index and value.
 * Plain host code: the two view checks need no device. */

/* One head's block index, as mmi_plan_export returns it (host arrays). */
typedef struct mmi_index_view {
  int32_t S;
  int32_t n_qblocks, n_kblocks;  /* mmi_head_stats */
  int32_t n_layouts;             /* key layouts kperm holds one after another (Q-Boundary heads with
                                    Grid modalities: more than 1), each n_kblocks / n_layouts blocks */
  int32_t causal;                /* 0: bidirectional head (mask bits mark padding only) */
  const int32_t* qperm;          /* [n_qblocks*64] slot -> position or -1, NULL = identity */
  const int32_t* kperm;          /* [n_kblocks*64], NULL = identity */
  const int32_t* row_ptr;        /* [n_qblocks+1] */
  const int32_t* col_idx;        /* [row_ptr[n_qblocks]] */
  int32_t group_size;            /* query blocks per row group (1, 2 or 4) */
  int32_t group_stride;          /* mmi_head_stats.group_stride */
  int32_t n_groups;              /* 0: the row-group checks are skipped */
  const int32_t* union_ptr;      /* [n_groups+1] (MMI_EXPORT_UNION_PTR) */
  const int32_t* union_ent;      /* [union_ptr[n_groups]] (MMI_EXPORT_UNION) */
} mmi_index_view;

/* Checks: qperm and each kperm layout hold every position of [0, S)
 * exactly once (other slots -1); row_ptr starts at 0 and never decreases,
 * column indices lie in [0, n_kblocks) and ascend within a row; per row
 * group (member r = query block (g / rho) R rho + g % rho + r rho): union_ptr
 * starts at 0 and never decreases, each entry names a key block once, its
 * select bits name live members only, the blocks of every live member come
 * first, each part ascending, member r's select bits mark exactly its query
 * block's column indices, and its mask bit is set exactly where the block
 * holds a key position above the member's smallest query position (or
 * padding; a bidirectional head: padding only). */
int mmi_check_index(const mmi_index_view* v);

/* The attention work list of a plan (host arrays). */
typedef struct mmi_work_view {
  int32_t n_heads;
  const int32_t* n_groups;             /* [n_heads] row groups per head */
  const int32_t* const* union_ptr;     /* [n_heads] -> [n_groups[h]+1] */
  int64_t n_items;
  const int32_t* items;                /* [n_items][5]: head, group, first and end union entry, partial
                                          slot (-1: the item writes O itself) */
  int64_t n_parts;                     /* partial slots */
  int64_t n_splits;
  const int32_t* splits;               /* [n_splits][4]: head, group, first partial slot, partials */
  int64_t map_len;
  const int32_t* item_map;             /* [8][map_len]: item indices per XCD, -1 = none */
} mmi_work_view;

/* Checks: the items of a row group follow each other in head and group
 * order and cut its union entries into consecutive ranges that cover it; a
 * group of one item writes O, a group of several gets consecutive unused
 * partial slots and exactly one split row naming them; every group with
 * union entries has items; the item map holds every item exactly once. */
int mmi_check_work(const mmi_work_view* w);

/* Both checks on a created plan: copies its tables to the host (synchronises
 * with the plan's stream) and checks every head and the work list. */
int mmi_plan_check(mmi_plan* plan);

#ifdef __cplusplus
}
#endif
#endif /* MMI_H */
