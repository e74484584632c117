// Modality-aware offline pattern search (Appendix A, Algorithm 4) for every
// head of one layer on a calibration sample, over this library's own plans.
// Each candidate configuration is one plan for all heads (one configuration
// per head), executed on the sample; its cost is the blocks the plan selects
// (the work the attention kernel runs, from the plan's per-modality block
// counts), its error the squared difference of its output from a reference
// output (the output-difference kernel, per head and query modality). Host
// code only: the plans, the attention and the objective run on the device.
//
// Rules (Appendix A and C.5; the parts the paper leaves open are readings):
//   cost of a configuration over a set of query rows = its selected blocks
//   there; admissible iff it does not exceed the cost of the FLOPs target
//   pattern over the same rows in the same coordinates; choice = admissible
//   candidate of smallest error (the earlier one on equal errors), else the
//   target pattern.
//   1. intra, per modality m: 2D-Boundary heads whose cross pairs select
//      nothing, the candidate on every modality at once; reference: every
//      intra op dense; rows: modality m.
//   2. cross, in rounds k = 1 .. n-1: 2D-Boundary heads with the chosen intra
//      ops, the candidate on the pairs (a, a + k mod n), the other pairs
//      dense; reference: dense causal attention; cost: the pair's blocks;
//      budget: a's intra budget minus the cost of its chosen intra op; none
//      admissible -> no cross blocks.
//   3. inter: the best global op (No-/K-Boundary kind, chosen like step 1 on
//      all rows), the Q-Boundary head with the chosen intra ops and the
//      2D-Boundary head with the chosen intra and cross ops; the smallest
//      error among those within the global target cost (that order on
//      ties), else the cheapest.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <memory>
#include <string>
#include <vector>

#include "internal.hpp"

namespace mmi {

namespace {

void call(int rc) {
  if (rc != MMI_OK) throw Error(rc, mmi_last_error());
}

void hipcall(hipError_t e, const char* what) {
  if (e != hipSuccess) throw Error(MMI_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

struct DevBuf {
  void* p = nullptr;
  explicit DevBuf(size_t bytes) {
    const hipError_t e = hipMalloc(&p, std::max<size_t>(bytes, 1));
    if (e == hipErrorOutOfMemory) throw Error(MMI_ERR_OOM, "device allocation of the search's buffers failed");
    hipcall(e, "hipMalloc");
  }
  ~DevBuf() {
    if (p) (void)hipFree(p);
  }
  DevBuf(const DevBuf&) = delete;
  DevBuf& operator=(const DevBuf&) = delete;
};

mmi_op op_of(int kind) {
  mmi_op o;
  std::memset(&o, 0, sizeof o);
  o.kind = kind;
  return o;
}

// Head configurations: ops not given are dense (intra) or select nothing
// (cross); the global op of a non-global head is unused and left dense.
mmi_head_cfg cfg_base(int kind) {
  mmi_head_cfg c;
  std::memset(&c, 0, sizeof c);     // every cross op MMI_OP_NONE
  c.kind = kind;
  c.global = op_of(MMI_OP_DENSE);
  for (int m = 0; m < MMI_MAX_MODALITIES; ++m) c.intra[m] = op_of(MMI_OP_DENSE);
  return c;
}

mmi_head_cfg global_head(const mmi_op& op) {
  mmi_head_cfg c = cfg_base(MMI_HEAD_GLOBAL);
  c.global = op;
  return c;
}

// Cost of one head in one plan: selected blocks of the head, of modality
// a's query rows, and of a's query rows against b's keys.
struct Cost {
  int64_t all = 0;
  int64_t mod[MMI_MAX_MODALITIES] = {};
  int64_t pair[MMI_MAX_MODALITIES][MMI_MAX_MODALITIES] = {};
};

class Runner {
 public:
  Runner(mmi_ctx* ctx, const mmi_problem& prob, const void* q, const void* k, const void* v, hipStream_t st)
      : ctx_(ctx), prob_(prob), q_(q), k_(k), v_(v), st_(st) {
    prob_.o_stride_s = prob_.o_stride_h = 0;          // the runner's outputs are packed
    const int64_t S = prob.S;
    bool present[MMI_MAX_MODALITIES] = {};
    for (int64_t i = 0; i < S; ++i) present[prob.modality ? prob.modality[i] : 0] = true;
    int cls_of[MMI_MAX_MODALITIES];
    for (int m = 0; m < MMI_MAX_MODALITIES; ++m) {
      cls_of[m] = -1;
      if (present[m]) {
        cls_of[m] = (int)mods.size();
        mods.push_back(m);
      }
    }
    std::vector<uint8_t> cls((size_t)S);
    for (int64_t i = 0; i < S; ++i) cls[(size_t)i] = (uint8_t)cls_of[prob.modality ? prob.modality[i] : 0];
    const size_t obytes = (size_t)S * prob.Hq * MMI_HEAD_DIM * 2;
    o_.reset(new DevBuf(obytes));
    ref_.reset(new DevBuf(obytes));
    cls_.reset(new DevBuf((size_t)S));
    err_.reset(new DevBuf(sizeof(double) * prob.Hq * mods.size()));
    hipcall(hipMemcpyAsync(cls_->p, cls.data(), (size_t)S, hipMemcpyHostToDevice, st_), "cls copy");
    hipcall(hipStreamSynchronize(st_), "cls copy");
  }

  std::vector<int> mods;       // modality ids present, ascending
  int64_t plans = 0;

  // Plans and executes one configuration per head into the candidate output
  // (or the reference), then reads each head's costs.
  std::vector<Cost> run(const std::vector<mmi_head_cfg>& heads, bool into_ref = false) {
    mmi_plan* plan = nullptr;
    call(mmi_plan_create(ctx_, &prob_, heads.data(), q_, k_, st_, &plan));
    std::vector<Cost> out(heads.size());
    int rc = mmi_plan_execute(plan, q_, k_, v_, into_ref ? ref_->p : o_->p, nullptr, st_);
    for (size_t h = 0; rc == MMI_OK && h < heads.size(); ++h) {
      mmi_head_stats s;
      rc = mmi_plan_stats(plan, (int)h, &s);
      if (rc != MMI_OK) break;
      Cost& c = out[h];
      c.all = s.nnz_blocks;
      for (int a = 0; a < MMI_MAX_MODALITIES; ++a)
        for (int b = 0; b < MMI_MAX_MODALITIES; ++b) {
          c.pair[a][b] = s.blocks_by_modality[a][b];
          c.mod[a] += s.blocks_by_modality[a][b];
        }
    }
    const std::string msg = rc == MMI_OK ? std::string() : std::string(mmi_last_error());
    const int rd = mmi_plan_destroy(plan);
    if (rc != MMI_OK) throw Error(rc, msg);
    call(rd);
    ++plans;
    return out;
  }

  // err[h][i]: squared difference of the candidate output from the
  // reference over the rows of modality mods[i], in float64.
  std::vector<std::vector<double>> sqerr() {
    const int n = (int)mods.size();
    call(mmi_output_sqerr(&prob_, o_->p, ref_->p, static_cast<const uint8_t*>(cls_->p), n,
                          static_cast<double*>(err_->p), st_));
    std::vector<double> e((size_t)prob_.Hq * n);
    hipcall(hipMemcpyAsync(e.data(), err_->p, sizeof(double) * e.size(), hipMemcpyDeviceToHost, st_), "err copy");
    hipcall(hipStreamSynchronize(st_), "err copy");
    std::vector<std::vector<double>> out((size_t)prob_.Hq, std::vector<double>(n));
    for (int h = 0; h < prob_.Hq; ++h)
      for (int i = 0; i < n; ++i) out[h][i] = e[(size_t)h * n + i];
    return out;
  }

 private:
  mmi_ctx* ctx_;
  mmi_problem prob_;
  const void *q_, *k_, *v_;
  hipStream_t st_;
  std::unique_ptr<DevBuf> o_, ref_, cls_, err_;
};

// Index of the admissible candidate (cost <= budget) of smallest error, the
// earliest on equal errors; -1 if none.
int choose(const std::vector<int64_t>& cost, const std::vector<double>& err, int64_t budget) {
  int best = -1;
  for (size_t i = 0; i < cost.size(); ++i)
    if (cost[i] <= budget && (best < 0 || err[i] < err[(size_t)best])) best = (int)i;
  return best;
}

}  // namespace

void search_layer(mmi_ctx* ctx, const mmi_problem& prob, const void* q, const void* k, const void* v,
                  const mmi_op* cands, int nc, const mmi_op* xc, int nx, const mmi_op& target, hipStream_t st,
                  mmi_head_cfg* out, mmi_search_report* rep) {
  Runner R(ctx, prob, q, k, v, st);
  const int Hq = prob.Hq, n = (int)R.mods.size();
  const std::vector<int>& mods = R.mods;
  constexpr int M = MMI_MAX_MODALITIES;
  auto d2 = [&](mmi_head_cfg c, const mmi_op* intra, const mmi_op (*cross)[M]) {
    c.kind = MMI_HEAD_2D;
    for (int m : mods) c.intra[m] = intra[m];
    for (int a : mods)
      for (int b : mods)
        if (a != b) c.cross[a][b] = cross[a][b];
    return c;
  };
  mmi_op none_x[M][M], dense_x[M][M], all_dense[M];
  for (int a = 0; a < M; ++a) {
    all_dense[a] = op_of(MMI_OP_DENSE);
    for (int b = 0; b < M; ++b) {
      none_x[a][b] = op_of(MMI_OP_NONE);
      dense_x[a][b] = op_of(MMI_OP_DENSE);
    }
  }
  const mmi_head_cfg base = cfg_base(MMI_HEAD_2D);
  auto every_mod = [&](const mmi_op& op) {
    std::vector<mmi_op> v2(M, op_of(MMI_OP_DENSE));
    for (int m : mods) v2[m] = op;
    return v2;
  };

  // 1. intra-modality
  std::vector<int64_t> budget1((size_t)Hq * n);
  std::vector<int64_t> c1((size_t)Hq * nc * n);
  std::vector<double> e1((size_t)Hq * nc * n);
  R.run(std::vector<mmi_head_cfg>(Hq, d2(base, all_dense, none_x)), true);
  {
    const std::vector<mmi_op> t = every_mod(target);
    const auto bc = R.run(std::vector<mmi_head_cfg>(Hq, d2(base, t.data(), none_x)));
    for (int h = 0; h < Hq; ++h)
      for (int i = 0; i < n; ++i) budget1[(size_t)h * n + i] = bc[h].mod[mods[i]];
  }
  for (int c = 0; c < nc; ++c) {
    const std::vector<mmi_op> ops = every_mod(cands[c]);
    const auto cc = R.run(std::vector<mmi_head_cfg>(Hq, d2(base, ops.data(), none_x)));
    const auto ee = R.sqerr();
    for (int h = 0; h < Hq; ++h)
      for (int i = 0; i < n; ++i) {
        c1[((size_t)h * nc + c) * n + i] = cc[h].mod[mods[i]];
        e1[((size_t)h * nc + c) * n + i] = ee[h][i];
      }
  }
  std::vector<int> intra_pick((size_t)Hq * n);
  std::vector<std::vector<mmi_op>> intra((size_t)Hq, std::vector<mmi_op>(M, op_of(MMI_OP_DENSE)));
  for (int h = 0; h < Hq; ++h)
    for (int i = 0; i < n; ++i) {
      std::vector<int64_t> cost(nc);
      std::vector<double> err(nc);
      for (int c = 0; c < nc; ++c) {
        cost[c] = c1[((size_t)h * nc + c) * n + i];
        err[c] = e1[((size_t)h * nc + c) * n + i];
      }
      const int pick = choose(cost, err, budget1[(size_t)h * n + i]);
      intra_pick[(size_t)h * n + i] = pick;
      intra[h][mods[i]] = pick >= 0 ? cands[pick] : target;
    }

  // 2. cross-modality
  const int rounds = std::max(n - 1, 0);
  std::vector<int64_t> c2((size_t)Hq * rounds * nx * n);
  std::vector<double> e2((size_t)Hq * rounds * nx * n);
  std::vector<int> cross_pick((size_t)Hq * n * n, -1);
  std::vector<std::vector<mmi_op>> cross((size_t)Hq, std::vector<mmi_op>((size_t)M * M, op_of(MMI_OP_NONE)));
  R.run(std::vector<mmi_head_cfg>(Hq, global_head(op_of(MMI_OP_DENSE))), true);
  std::vector<Cost> ic;
  {
    std::vector<mmi_head_cfg> heads(Hq);
    for (int h = 0; h < Hq; ++h) heads[h] = d2(base, intra[h].data(), none_x);
    ic = R.run(heads);
  }
  for (int kk = 1; kk <= rounds; ++kk) {
    for (int x = 0; x < nx; ++x) {
      mmi_op cx[M][M];
      std::memcpy(cx, dense_x, sizeof cx);
      for (int ai = 0; ai < n; ++ai) cx[mods[ai]][mods[(ai + kk) % n]] = xc[x];
      std::vector<mmi_head_cfg> heads(Hq);
      for (int h = 0; h < Hq; ++h) heads[h] = d2(base, intra[h].data(), cx);
      const auto cc = R.run(heads);
      const auto ee = R.sqerr();
      for (int h = 0; h < Hq; ++h)
        for (int ai = 0; ai < n; ++ai) {
          const size_t at = (((size_t)h * rounds + (kk - 1)) * nx + x) * n + ai;
          c2[at] = cc[h].pair[mods[ai]][mods[(ai + kk) % n]];
          e2[at] = ee[h][ai];
        }
    }
    for (int h = 0; h < Hq; ++h)
      for (int ai = 0; ai < n; ++ai) {
        const int bi = (ai + kk) % n;
        std::vector<int64_t> cost(nx);
        std::vector<double> err(nx);
        for (int x = 0; x < nx; ++x) {
          const size_t at = (((size_t)h * rounds + (kk - 1)) * nx + x) * n + ai;
          cost[x] = c2[at];
          err[x] = e2[at];
        }
        const int pick = choose(cost, err, budget1[(size_t)h * n + ai] - ic[h].mod[mods[ai]]);
        cross_pick[((size_t)h * n + ai) * n + bi] = pick;
        cross[h][(size_t)mods[ai] * M + mods[bi]] = pick >= 0 ? xc[pick] : op_of(MMI_OP_NONE);
      }
  }

  // 3. inter-modality
  std::vector<int64_t> budget3(Hq), c3g((size_t)Hq * nc), c3((size_t)Hq * 3);
  std::vector<double> e3g((size_t)Hq * nc), e3((size_t)Hq * 3);
  {
    const auto gc = R.run(std::vector<mmi_head_cfg>(Hq, global_head(target)));
    for (int h = 0; h < Hq; ++h) budget3[h] = gc[h].all;
  }
  auto total = [&](const std::vector<double>& e) {   // rows of every modality, in ascending order
    double t = 0.0;
    for (int i = 0; i < n; ++i) t += e[i];
    return t;
  };
  for (int c = 0; c < nc; ++c) {
    const auto cc = R.run(std::vector<mmi_head_cfg>(Hq, global_head(cands[c])));
    const auto ee = R.sqerr();
    for (int h = 0; h < Hq; ++h) {
      c3g[(size_t)h * nc + c] = cc[h].all;
      e3g[(size_t)h * nc + c] = total(ee[h]);
    }
  }
  std::vector<int> global_pick(Hq);
  std::vector<mmi_head_cfg> kinds[3];
  for (auto& v2 : kinds) v2.resize(Hq);
  for (int h = 0; h < Hq; ++h) {
    const int pick = choose(std::vector<int64_t>(c3g.begin() + (size_t)h * nc, c3g.begin() + (size_t)(h + 1) * nc),
                            std::vector<double>(e3g.begin() + (size_t)h * nc, e3g.begin() + (size_t)(h + 1) * nc),
                            budget3[h]);
    global_pick[h] = pick;
    kinds[0][h] = global_head(pick >= 0 ? cands[pick] : target);
    mmi_head_cfg qb = cfg_base(MMI_HEAD_QBOUNDARY);
    for (int m : mods) qb.intra[m] = intra[h][m];
    kinds[1][h] = qb;
    mmi_op cx[M][M];
    std::memcpy(cx, cross[h].data(), sizeof cx);
    kinds[2][h] = d2(base, intra[h].data(), cx);
  }
  for (int kd = 0; kd < 3; ++kd) {
    const auto cc = R.run(kinds[kd]);
    const auto ee = R.sqerr();
    for (int h = 0; h < Hq; ++h) {
      c3[(size_t)h * 3 + kd] = cc[h].all;
      e3[(size_t)h * 3 + kd] = total(ee[h]);
    }
  }
  std::vector<int> kind_pick(Hq);
  for (int h = 0; h < Hq; ++h) {
    const std::vector<int64_t> cost(c3.begin() + (size_t)h * 3, c3.begin() + (size_t)h * 3 + 3);
    int pick = choose(cost, std::vector<double>(e3.begin() + (size_t)h * 3, e3.begin() + (size_t)h * 3 + 3),
                      budget3[h]);
    if (pick < 0) pick = (int)(std::min_element(cost.begin(), cost.end()) - cost.begin());
    kind_pick[h] = pick;
    out[h] = kinds[pick][h];
  }

  if (!rep) return;
  rep->n_mod = n;
  for (int i = 0; i < M; ++i) rep->mods[i] = i < n ? mods[i] : -1;
  rep->plans = R.plans;
  for (int h = 0; h < Hq; ++h) {
    for (int i = 0; i < n; ++i) {
      if (rep->budget1) rep->budget1[(size_t)h * M + i] = budget1[(size_t)h * n + i];
      if (rep->intra) rep->intra[(size_t)h * M + i] = intra_pick[(size_t)h * n + i];
      for (int c = 0; c < nc; ++c) {
        if (rep->step1_cost) rep->step1_cost[((size_t)h * nc + c) * M + i] = c1[((size_t)h * nc + c) * n + i];
        if (rep->step1_err) rep->step1_err[((size_t)h * nc + c) * M + i] = e1[((size_t)h * nc + c) * n + i];
      }
      for (int j = 0; j < n; ++j)
        if (rep->cross) rep->cross[((size_t)h * M + i) * M + j] = cross_pick[((size_t)h * n + i) * n + j];
      for (int kk = 0; kk < rounds; ++kk)
        for (int x = 0; x < nx; ++x) {
          const size_t src = (((size_t)h * rounds + kk) * nx + x) * n + i;
          const size_t dst = (((size_t)h * (M - 1) + kk) * nx + x) * M + i;
          if (rep->step2_cost) rep->step2_cost[dst] = c2[src];
          if (rep->step2_err) rep->step2_err[dst] = e2[src];
        }
    }
    if (rep->budget3) rep->budget3[h] = budget3[h];
    for (int c = 0; c < nc; ++c) {
      if (rep->step3g_cost) rep->step3g_cost[(size_t)h * nc + c] = c3g[(size_t)h * nc + c];
      if (rep->step3g_err) rep->step3g_err[(size_t)h * nc + c] = e3g[(size_t)h * nc + c];
    }
    for (int kd = 0; kd < 3; ++kd) {
      if (rep->step3_cost) rep->step3_cost[(size_t)h * 3 + kd] = c3[(size_t)h * 3 + kd];
      if (rep->step3_err) rep->step3_err[(size_t)h * 3 + kd] = e3[(size_t)h * 3 + kd];
    }
    if (rep->global) rep->global[h] = global_pick[h];
    if (rep->kind) rep->kind[h] = kind_pick[h];
  }
}

}  // namespace mmi
