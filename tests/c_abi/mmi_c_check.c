/* C-only check of the libmmi ABI (test infrastructure): no Python, no torch.
 *   1. status codes and messages for invalid arguments;
 *   2. a global A-shape head whose window covers every key selects every
 *      causal block, so mmi_attention must equal mmi_dense_attention bitwise;
 *   3. plan statistics of that head (every causal block selected) and the
 *      host consistency checks of its tables;
 *   4. sampled rows of the output against plain causal softmax attention
 *      computed here in double precision (|dO| <= 2e-2, |dLSE| <= 1e-3);
 *   5. the pattern search (Algorithm 4) over two intra candidates: the
 *      number of plans it builds, and a chosen configuration that is the
 *      one its report names.
 * Prints "c abi ok" and exits 0 on success. */
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "../../include/mmi.h"

#define CHECK(x)                                                                         \
  do {                                                                                   \
    int rc_ = (x);                                                                       \
    if (rc_ != MMI_OK) {                                                                 \
      fprintf(stderr, "%s:%d: %s -> %d (%s)\n", __FILE__, __LINE__, #x, rc_, mmi_last_error()); \
      exit(1);                                                                           \
    }                                                                                    \
  } while (0)
#define HCHECK(x)                                                                        \
  do {                                                                                   \
    if ((x) != hipSuccess) { fprintf(stderr, "%s:%d: HIP call failed\n", __FILE__, __LINE__); exit(1); } \
  } while (0)
#define EXPECT(c)                                                                        \
  do {                                                                                   \
    if (!(c)) { fprintf(stderr, "%s:%d: expected %s\n", __FILE__, __LINE__, #c); exit(1); } \
  } while (0)

static uint64_t rng = 0x9E3779B97F4A7C15ull;
static double uniform(void) {      /* xorshift64*, uniform in (0, 1) */
  rng ^= rng >> 12; rng ^= rng << 25; rng ^= rng >> 27;
  return ((rng * 0x2545F4914F6CDD1Dull) >> 11) * (1.0 / 9007199254740992.0) + 1e-300;
}
static double normal(void) { return sqrt(-2.0 * log(uniform())) * cos(6.283185307179586 * uniform()); }

static uint16_t to_bf16(float f) {  /* round to nearest even */
  uint32_t u;
  memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
static double from_bf16(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

int main(void) {
  const int S = 3000, Hq = 4, Hkv = 2, D = 128, G = Hq / Hkv;
  printf("libmmi ABI version %d\n", mmi_version());
  EXPECT(mmi_version() == MMI_ABI_VERSION);
  EXPECT(strcmp(mmi_status_str(MMI_OK), "ok") == 0);

  const size_t nq = (size_t)S * Hq * D, nk = (size_t)S * Hkv * D;
  uint16_t *hq = malloc(nq * 2), *hk = malloc(nk * 2), *hv = malloc(nk * 2), *o1 = malloc(nq * 2),
           *o2 = malloc(nq * 2);
  float *l1 = malloc((size_t)Hq * S * 4), *l2 = malloc((size_t)Hq * S * 4);
  for (size_t i = 0; i < nq; ++i) hq[i] = to_bf16((float)normal());
  for (size_t i = 0; i < nk; ++i) hk[i] = to_bf16((float)normal());
  for (size_t i = 0; i < nk; ++i) hv[i] = to_bf16((float)normal());
  void *dq, *dk, *dv, *do1, *do2;
  float *dl1, *dl2;
  HCHECK(hipMalloc(&dq, nq * 2)); HCHECK(hipMalloc(&dk, nk * 2)); HCHECK(hipMalloc(&dv, nk * 2));
  HCHECK(hipMalloc(&do1, nq * 2)); HCHECK(hipMalloc(&do2, nq * 2));
  HCHECK(hipMalloc((void**)&dl1, (size_t)Hq * S * 4)); HCHECK(hipMalloc((void**)&dl2, (size_t)Hq * S * 4));
  HCHECK(hipMemcpy(dq, hq, nq * 2, hipMemcpyHostToDevice));
  HCHECK(hipMemcpy(dk, hk, nk * 2, hipMemcpyHostToDevice));
  HCHECK(hipMemcpy(dv, hv, nk * 2, hipMemcpyHostToDevice));

  mmi_problem p;
  memset(&p, 0, sizeof p);
  p.S = S; p.Hq = Hq; p.Hkv = Hkv; p.D = D; p.block = 64;
  mmi_head_cfg* cfgs = calloc(Hq, sizeof(mmi_head_cfg));
  for (int h = 0; h < Hq; ++h) {
    cfgs[h].kind = MMI_HEAD_GLOBAL;
    cfgs[h].global.kind = MMI_OP_ASHAPE;
    cfgs[h].global.sink = 0;
    cfgs[h].global.local = S;          /* the window covers every key */
  }

  /* 1. invalid arguments */
  mmi_ctx* ctx = NULL;
  mmi_plan* plan = NULL;
  EXPECT(mmi_plan_create(NULL, &p, cfgs, dq, dk, NULL, &plan) == MMI_ERR_INVALID_ARG);
  CHECK(mmi_ctx_create(0, &ctx));
  mmi_problem bad = p;
  bad.D = 64;
  EXPECT(mmi_plan_create(ctx, &bad, cfgs, dq, dk, NULL, &plan) == MMI_ERR_UNSUPPORTED);
  EXPECT(strlen(mmi_last_error()) > 0);
  cfgs[0].global.kind = 99;
  EXPECT(mmi_plan_create(ctx, &p, cfgs, dq, dk, NULL, &plan) == MMI_ERR_BAD_CONFIG);
  cfgs[0].global.kind = MMI_OP_ASHAPE;
  EXPECT(mmi_search(ctx, &p, dq, dk, dv, NULL, 0, NULL, 0, NULL, NULL, cfgs, NULL) == MMI_ERR_INVALID_ARG);

  /* 2. full-window A-shape == dense, bitwise */
  CHECK(mmi_attention(ctx, &p, cfgs, dq, dk, dv, do1, dl1, NULL));
  CHECK(mmi_dense_attention(ctx, &p, dq, dk, dv, do2, dl2, NULL));
  HCHECK(hipDeviceSynchronize());
  HCHECK(hipMemcpy(o1, do1, nq * 2, hipMemcpyDeviceToHost));
  HCHECK(hipMemcpy(o2, do2, nq * 2, hipMemcpyDeviceToHost));
  HCHECK(hipMemcpy(l1, dl1, (size_t)Hq * S * 4, hipMemcpyDeviceToHost));
  HCHECK(hipMemcpy(l2, dl2, (size_t)Hq * S * 4, hipMemcpyDeviceToHost));
  EXPECT(memcmp(o1, o2, nq * 2) == 0);
  EXPECT(memcmp(l1, l2, (size_t)Hq * S * 4) == 0);

  /* 3. statistics */
  CHECK(mmi_plan_create(ctx, &p, cfgs, dq, dk, NULL, &plan));
  mmi_head_stats st;
  CHECK(mmi_plan_stats(plan, 1, &st));
  CHECK(mmi_plan_check(plan));     /* the plan's tables pass the host consistency checks */
  {                                /* and a block index with a key block out of range fails them */
    int32_t rp[2] = {0, 1}, col[1] = {1};
    mmi_index_view iv;
    memset(&iv, 0, sizeof iv);
    iv.S = 64; iv.n_qblocks = 1; iv.n_kblocks = 1; iv.n_layouts = 1; iv.causal = 1;
    iv.row_ptr = rp; iv.col_idx = col;
    EXPECT(mmi_check_index(&iv) == MMI_ERR_INTERNAL);
    col[0] = 0;
    CHECK(mmi_check_index(&iv));
  }
  EXPECT(st.kind == MMI_HEAD_GLOBAL && st.nnz_blocks == st.causal_blocks);
  CHECK(mmi_plan_destroy(plan));

  /* 4. sampled rows against plain causal attention in double precision */
  const int rows[] = {0, 1, 63, 64, 65, 1000, 2047, 2999};
  double max_do = 0.0, max_dl = 0.0;
  double* s = malloc((size_t)S * sizeof(double));
  for (int h = 0; h < Hq; ++h) {
    const int g = h / G;
    for (size_t ri = 0; ri < sizeof rows / sizeof rows[0]; ++ri) {
      const int q = rows[ri];
      double m = -INFINITY, l = 0.0;
      for (int kk = 0; kk <= q; ++kk) {
        double dot = 0.0;
        for (int d = 0; d < D; ++d)
          dot += from_bf16(hq[((size_t)q * Hq + h) * D + d]) * from_bf16(hk[((size_t)kk * Hkv + g) * D + d]);
        s[kk] = dot / sqrt((double)D);
        if (s[kk] > m) m = s[kk];
      }
      for (int kk = 0; kk <= q; ++kk) l += exp(s[kk] - m);
      for (int d = 0; d < D; ++d) {
        double acc = 0.0;
        for (int kk = 0; kk <= q; ++kk) acc += exp(s[kk] - m) * from_bf16(hv[((size_t)kk * Hkv + g) * D + d]);
        const double diff = fabs(acc / l - from_bf16(o1[((size_t)q * Hq + h) * D + d]));
        if (diff > max_do) max_do = diff;
      }
      const double lse = m + log(l);
      const double dl = fabs(lse - l1[(size_t)h * S + q]) / fmax(1.0, fabs(lse));
      if (dl > max_dl) max_dl = dl;
    }
  }
  printf("max |dO| %.3g, max rel |dLSE| %.3g\n", max_do, max_dl);
  EXPECT(max_do <= 2e-2 && max_dl <= 1e-3);

  /* 5. search: one modality, intra candidates {dense, A-shape(64, 128)},
   * no cross candidates, target A-shape(64, 256): 8 + 2*2 + 0 plans */
  {
    mmi_op cand[2], target;
    memset(cand, 0, sizeof cand);
    memset(&target, 0, sizeof target);
    cand[0].kind = MMI_OP_DENSE;
    cand[1].kind = MMI_OP_ASHAPE; cand[1].sink = 64; cand[1].local = 128;
    target.kind = MMI_OP_ASHAPE; target.sink = 64; target.local = 256;
    mmi_head_cfg* chosen = calloc(Hq, sizeof(mmi_head_cfg));
    int32_t kind[8], glob[8], intra[8 * MMI_MAX_MODALITIES];
    int64_t budget3[8], cost3[8 * 3];
    mmi_search_report rep;
    memset(&rep, 0, sizeof rep);
    rep.kind = kind; rep.global = glob; rep.intra = intra; rep.budget3 = budget3; rep.step3_cost = cost3;
    EXPECT(Hq <= 8);
    CHECK(mmi_search(ctx, &p, dq, dk, dv, cand, 2, NULL, 0, &target, NULL, chosen, &rep));
    EXPECT(rep.plans == 8 + 2 * 2 && rep.n_mod == 1 && rep.mods[0] == 0 && rep.mods[1] == -1);
    for (int h = 0; h < Hq; ++h) {
      EXPECT(kind[h] >= 0 && kind[h] <= 2 && chosen[h].kind == kind[h]);
      /* dense exceeds the target's cost over all rows, so a chosen global op is the A-shape */
      EXPECT(glob[h] == 1 && intra[h * MMI_MAX_MODALITIES] == 1);
      if (kind[h] == MMI_HEAD_GLOBAL) EXPECT(chosen[h].global.kind == MMI_OP_ASHAPE && chosen[h].global.local == 128);
      EXPECT(cost3[h * 3 + kind[h]] <= budget3[h]);
    }
    free(chosen);
  }

  CHECK(mmi_ctx_destroy(ctx));
  HCHECK(hipFree(dq)); HCHECK(hipFree(dk)); HCHECK(hipFree(dv)); HCHECK(hipFree(do1)); HCHECK(hipFree(do2));
  HCHECK(hipFree(dl1)); HCHECK(hipFree(dl2));
  printf("c abi ok\n");
  return 0;
}
