// Host runtime of libmmi: argument validation, modality layout, the plan
// (estimation jobs, choices, permutations, block index, work list), launch
// sequencing on the caller's stream, a caching device allocator, and the
// C entry points declared in include/mmi.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <memory>
#include <mutex>
#include <stdexcept>
#include <string>
#include <functional>
#include <vector>

#include "device.hpp"
#include "internal.hpp"

namespace mmi {

// ------------------------------------------------------------------ errors
static thread_local std::string g_last_error;

[[noreturn]] static void fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  throw Error(code, buf);
}

#define HIPCHK(expr)                                                                          \
  do {                                                                                        \
    hipError_t e_ = (expr);                                                                   \
    if (e_ != hipSuccess) fail(MMI_ERR_HIP, "%s: %s (%s:%d)", #expr, hipGetErrorString(e_), \
                               __FILE__, __LINE__);                                           \
  } while (0)

// ------------------------------------------------------------------ allocator
// Device memory cache owned by a context: freed blocks are kept per exact
// size and handed out again, so repeated plans of one shape allocate once.
class Allocator {
 public:
  ~Allocator() { release(); }
  void* get(size_t bytes) {
    bytes = round(bytes);
    {
      std::lock_guard<std::mutex> lk(mu_);
      auto it = free_.find(bytes);
      if (it != free_.end()) {
        void* p = it->second;
        free_.erase(it);
        return p;
      }
    }
    void* p = nullptr;
    if (hipMalloc(&p, bytes) != hipSuccess) {
      (void)hipGetLastError();
      release();
      if (hipMalloc(&p, bytes) != hipSuccess) {
        (void)hipGetLastError();
        fail(MMI_ERR_OOM, "device allocation of %zu bytes failed", bytes);
      }
    }
    return p;
  }
  void put(void* p, size_t bytes) {
    if (!p) return;
    std::lock_guard<std::mutex> lk(mu_);
    free_.emplace(round(bytes), p);
  }
  void release() {
    std::lock_guard<std::mutex> lk(mu_);
    for (auto& kv : free_) (void)hipFree(kv.second);
    free_.clear();
  }

 private:
  static size_t round(size_t b) {
    if (b < 256) return 256;
    size_t r = 256;
    while (r < b && r < ((size_t)1 << 24)) r <<= 1;
    if (r >= b) return r;
    return (b + ((size_t)1 << 24) - 1) & ~(((size_t)1 << 24) - 1);
  }
  std::mutex mu_;
  std::multimap<size_t, void*> free_;
};

}  // namespace mmi

// ------------------------------------------------------------------ no-allocation scratch
// Device memory of mmi_attention_noalloc: one static array, which every GPU
// the library runs on holds (its own copy) until the process ends. Host code
// never passes the array's name as an address: its address on each device
// comes from hipGetSymbolAddress, taken once per device when the first
// context on that device is created.
static __device__ __align__(256) uint8_t scratch[MMI_NOALLOC_SCRATCH_BYTES];

namespace mmi {
constexpr int MAX_DEVICES = 64;
static std::mutex g_scratch_mu;                      // guards g_scratch_ptr
static uint8_t* g_scratch_ptr[MAX_DEVICES] = {};     // address of `scratch` on each device
static std::mutex g_scratch_call_mu[MAX_DEVICES];    // one no-allocation call at a time per device

static void scratch_setup(int device) {              // device is current
  if (device >= MAX_DEVICES) return;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch_ptr[device]) return;
  void* ptr = nullptr;
  HIPCHK(hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)));
  g_scratch_ptr[device] = static_cast<uint8_t*>(ptr);
}
}  // namespace mmi

struct mmi_ctx {
  int device = 0;
  int chunk_blocks = 64;           // smallest work-item length (union entries)
  int items_per_layer = 8192;      // target number of work items per layer
  int split_above_avg = 6;         // with enough row groups, split only groups above this many times
                                   // their head's average union (0: always split to the item target)
  int row_group = 4;               // query blocks per attention work item (1, 2 or 4)
  int live_plans = 0;              // plans created from this context and not destroyed
  bool debug = false;              // MMI_DEBUG: check every plan's tables, synchronise every execute
  mmi::Allocator alloc;
  int64_t* pinned = nullptr;       // host staging for totals
  size_t pinned_n = 0;
};

namespace mmi {

// ------------------------------------------------------------------ plan
struct Buf {
  void* p = nullptr;
  size_t n = 0;
};

struct EstInfo {       // host view of one estimation job
  int job = -1;
  int rowset = -1;
  int L_c = 0, nrows = 0, row0 = 0;
  float* v = nullptr;
  float* u = nullptr;
  float* fold = nullptr;
  int lo = 0, hi = -1;
  int32_t* params = nullptr;
  int32_t* vsel = nullptr;
  int32_t* ssel = nullptr;
  int nv = 0, ns = 0;
};

struct HostHead {
  int kind = 0;
  int op0 = 0, nops = 0;
  std::vector<int> op_slot;      // op index -> export slot
  std::vector<EstInfo> est;      // per op
  int64_t nnz = 0, gnnz = 0, nitems = 0, nsplit = 0, nparts = 0;
};

}  // namespace mmi

struct mmi_plan {
  mmi_ctx* ctx = nullptr;
  hipStream_t stream = nullptr;
  mmi_problem prob{};
  int S = 0, Hq = 0, Hkv = 0;
  mmi::Groups groups{};
  std::vector<mmi::Buf> bufs;
  std::vector<mmi::HeadDev> heads;
  std::vector<mmi::OpDev> ops;
  std::vector<mmi::HostHead> hh;
  mmi::HeadDev* d_heads = nullptr;
  mmi::OpDev* d_ops = nullptr;
  mmi::WorkItem* d_items = nullptr;
  mmi::SplitRow* d_splits = nullptr;
  float* d_part_o = nullptr;
  float* d_part_ml = nullptr;
  int64_t nitems = 0, nsplit = 0, nparts = 0;
  int32_t* d_item_map = nullptr;  // [8][map_len] work items per XCD
  int64_t map_len = 0;
  int R = 1;                      // query blocks per attention work item
  int32_t* d_tpos = nullptr;
  std::vector<uint8_t> mod;       // host modality of every position (all 0 without a layout)
  std::vector<float*> est_lse2;  // per rowset
  std::vector<std::vector<uint8_t>> keep;   // host sources of asynchronous uploads
  hipEvent_t ev[7] = {};          // stage boundaries: create 0..3, execute 4..6
  int64_t nnz_all = 0;
  int64_t gnnz_all = 0;
  bool executed = false;
  std::vector<int> rowset_n;
  int64_t device_bytes = 0;       // device memory the plan holds
  uint8_t* scratch = nullptr;     // non-null: buffers come from the no-allocation scratch
  size_t scratch_used = 0;
};

namespace mmi {

template <typename T>
static T* dalloc(mmi_plan* P, size_t count) {
  size_t bytes = std::max<size_t>(count, 1) * sizeof(T);
  if (P->scratch) {                      // bump allocation inside the static scratch
    const size_t off = (P->scratch_used + 255) & ~(size_t)255;
    if (bytes > MMI_NOALLOC_SCRATCH_BYTES || off > MMI_NOALLOC_SCRATCH_BYTES - bytes)
      fail(MMI_ERR_UNSUPPORTED,
           "the plan needs more than the %zu bytes of no-allocation scratch (S = %d, Hq = %d); "
           "use mmi_attention", (size_t)MMI_NOALLOC_SCRATCH_BYTES, P->S, P->Hq);
    P->scratch_used = off + bytes;
    P->device_bytes = (int64_t)P->scratch_used;
    return reinterpret_cast<T*>(P->scratch + off);
  }
  void* p = P->ctx->alloc.get(bytes);
  P->bufs.push_back({p, bytes});
  P->device_bytes += (int64_t)bytes;
  return reinterpret_cast<T*>(p);
}

// Stage boundary event (plans in scratch mode create no events).
static void mark(mmi_plan* P, int i, hipStream_t st) {
  if (P->ev[i]) HIPCHK(hipEventRecord(P->ev[i], st));
}

// Several host arrays sent as one device allocation and one copy (fewer
// small host-to-device copies per plan); each array's device address is
// handed to its setter when the pack is sent. The host copy is kept in the
// plan until it is destroyed, so the asynchronous copy never reads freed
// memory.
struct Pack {
  std::vector<uint8_t> host;
  std::vector<std::function<void(uint8_t*)>> set;
  template <typename T>
  void add(const std::vector<T>& v, T*& out) {
    const size_t off = (host.size() + 255) & ~(size_t)255;
    host.resize(off + std::max<size_t>(v.size(), 1) * sizeof(T));
    if (!v.empty()) std::memcpy(host.data() + off, v.data(), v.size() * sizeof(T));
    T** slot = &out;
    set.emplace_back([slot, off](uint8_t* d) { *slot = reinterpret_cast<T*>(d + off); });
  }
};

static void send(mmi_plan* P, Pack& pk) {
  uint8_t* d = dalloc<uint8_t>(P, pk.host.size());
  P->keep.push_back(std::move(pk.host));
  HIPCHK(hipMemcpyAsync(d, P->keep.back().data(), P->keep.back().size(), hipMemcpyHostToDevice, P->stream));
  for (auto& f : pk.set) f(d);
}

static void free_plan_buffers(mmi_plan* P) {
  for (auto& b : P->bufs) P->ctx->alloc.put(b.p, b.n);
  P->bufs.clear();
}

// ------------------------------------------------------------------ validation
static void check_op(const mmi_op& op, std::initializer_list<int> allowed, const char* where, int h) {
  bool ok = false;
  for (int a : allowed) ok |= (op.kind == a);
  if (!ok) fail(MMI_ERR_BAD_CONFIG, "head %d: op kind %d not allowed for %s", h, op.kind, where);
  if (op.kind == MMI_OP_ASHAPE && (op.sink < 0 || op.local < 0))
    fail(MMI_ERR_BAD_CONFIG, "head %d: A-shape sink/local must be >= 0", h);
  if ((op.kind == MMI_OP_VSLASH || op.kind == MMI_OP_VERT) && (op.n_vertical < 0 || op.n_slash < 0))
    fail(MMI_ERR_BAD_CONFIG, "head %d: vertical/slash sizes must be >= 0", h);
  if (op.kind == MMI_OP_GRID &&
      (op.stride_lo < 1 || op.stride_hi < op.stride_lo || op.stride_hi > MMI_MAX_STRIDE))
    fail(MMI_ERR_BAD_CONFIG, "head %d: grid stride range [%d, %d] outside [1, %d]", h, op.stride_lo,
         op.stride_hi, MMI_MAX_STRIDE);
  if ((op.kind == MMI_OP_SF_FIXED || op.kind == MMI_OP_SF_STRIDED) && (op.local < 1 || op.stride_lo < 1))
    fail(MMI_ERR_BAD_CONFIG, "head %d: Sparse Transformer local and stride must be >= 1", h);
  if (op.kind == MMI_OP_TRISHAPE && (op.sink < 0 || op.local < 0 || op.bottom < 0))
    fail(MMI_ERR_BAD_CONFIG, "head %d: Tri-shape sink/local/bottom must be >= 0", h);
}

static void aligned16(const void* p, const char* name) {
  if (reinterpret_cast<uintptr_t>(p) % 16) fail(MMI_ERR_INVALID_ARG, "%s is not 16-byte aligned", name);
}

static mmi_problem normalise(const mmi_problem* pr) {
  if (!pr) fail(MMI_ERR_INVALID_ARG, "problem is NULL");
  mmi_problem p = *pr;
  if (p.S < 1) fail(MMI_ERR_INVALID_ARG, "S must be >= 1");
  if (p.S > MMI_MAX_SEQ) fail(MMI_ERR_UNSUPPORTED, "S = %lld exceeds %d", (long long)p.S, MMI_MAX_SEQ);
  if (p.Hq < 1 || p.Hkv < 1) fail(MMI_ERR_INVALID_ARG, "head counts must be >= 1");
  if (p.Hq % p.Hkv) fail(MMI_ERR_UNSUPPORTED, "Hq %% Hkv != 0");
  if (p.D != MMI_HEAD_DIM) fail(MMI_ERR_UNSUPPORTED, "head dim %d (only 128)", p.D);
  if (p.block != MMI_BLOCK) fail(MMI_ERR_UNSUPPORTED, "block %d (only 64)", p.block);
  auto def = [](int64_t& ss, int64_t& sh, int H) {
    if (ss == 0 && sh == 0) { ss = (int64_t)H * 128; sh = 128; }
  };
  def(p.q_stride_s, p.q_stride_h, p.Hq);
  def(p.k_stride_s, p.k_stride_h, p.Hkv);
  def(p.v_stride_s, p.v_stride_h, p.Hkv);
  def(p.o_stride_s, p.o_stride_h, p.Hq);
  const int64_t st[8] = {p.q_stride_s, p.q_stride_h, p.k_stride_s, p.k_stride_h,
                         p.v_stride_s, p.v_stride_h, p.o_stride_s, p.o_stride_h};
  for (int i = 0; i < 8; ++i)
    if (st[i] <= 0 || st[i] % 8) fail(MMI_ERR_INVALID_ARG, "strides must be positive multiples of 8 elements");
  // the attention kernel forms K/V row offsets as 32-bit byte offsets, the
  // token stride in bytes entering a 24-bit multiply
  if (2 * p.S * p.k_stride_s > (int64_t)UINT32_MAX || 2 * p.S * p.v_stride_s > (int64_t)UINT32_MAX)
    fail(MMI_ERR_UNSUPPORTED, "S x K/V token stride must stay below 2^31 elements");
  if (2 * p.k_stride_s >= ((int64_t)1 << 24) || 2 * p.v_stride_s >= ((int64_t)1 << 24))
    fail(MMI_ERR_UNSUPPORTED, "K/V token stride must stay below 2^23 elements");
  if (p.modality) {
    if (p.n_modalities < 1 || p.n_modalities > MMI_MAX_MODALITIES)
      fail(MMI_ERR_INVALID_ARG, "n_modalities must be in [1, %d]", MMI_MAX_MODALITIES);
    for (int64_t i = 0; i < p.S; ++i)
      if (p.modality[i] >= p.n_modalities) fail(MMI_ERR_INVALID_ARG, "modality[%lld] = %d out of range",
                                                (long long)i, (int)p.modality[i]);
  }
  return p;
}

// ------------------------------------------------------------------ layout (host)
struct Layout {
  std::vector<Segment> segs;
  Groups g{};
  int gidx_of_mod[MMI_MAX_MODALITIES];
  std::vector<std::vector<int>> seg_of_group;   // segment indices per group, ascending
};

static Layout make_layout(const mmi_problem& p) {
  Layout L;
  const int S = (int)p.S;
  int count[MMI_MAX_MODALITIES] = {0};
  if (!p.modality) {
    L.segs.push_back({0, S, 0, 0});
    count[0] = S;
  } else {
    int i = 0;
    while (i < S) {
      int j = i;
      const int m = p.modality[i];
      while (j < S && p.modality[j] == m) ++j;
      L.segs.push_back({i, j - i, count[m], m});
      count[m] += j - i;
      i = j;
    }
  }
  std::fill(L.gidx_of_mod, L.gidx_of_mod + MMI_MAX_MODALITIES, -1);
  int off = 0, toff = 0;
  for (int m = 0; m < MMI_MAX_MODALITIES; ++m) {
    if (!count[m]) continue;
    const int gi = L.g.n++;
    L.gidx_of_mod[m] = gi;
    L.g.mod[gi] = m;
    L.g.off[gi] = off;
    L.g.len[gi] = count[m];
    L.g.toff[gi] = toff;
    off += (count[m] + B - 1) / B * B;
    toff += count[m];
  }
  L.seg_of_group.resize(L.g.n);
  for (int s = 0; s < (int)L.segs.size(); ++s) L.seg_of_group[L.gidx_of_mod[L.segs[s].mod]].push_back(s);
  return L;
}

// final <= 64 positions of the last run of group gi -> (row0, nrows, local index of row0)
static void final_rows(const Layout& L, int gi, int& row0, int& nrows, int& loc0) {
  const Segment& s = L.segs[L.seg_of_group[gi].back()];
  nrows = std::min(LASTQ, s.len);
  row0 = s.pos + s.len - nrows;
  loc0 = s.loc + s.len - nrows;
}

// number of positions of group gi that are <= pos
static int count_le(const Layout& L, int gi, int pos) {
  int c = 0;
  for (int s : L.seg_of_group[gi]) {
    const Segment& sg = L.segs[s];
    if (sg.pos > pos) break;
    c += std::min(sg.len, pos - sg.pos + 1);
  }
  return c;
}

// ------------------------------------------------------------------ plan create
struct Builder {
  mmi_plan* P;
  Layout L;
  std::vector<RowSet> rowsets;
  std::vector<EstJob> jobs;
  std::vector<GridJob> gjobs;
  std::vector<TopkJob> tjobs;
  std::map<std::pair<int, int>, int> rowset_of;   // (head, row0) -> index
  int chunk_keys = 4096;
  int max_tiles = 0, max_L = 0, max_chunks = 0, max_cands = 0, max_sel = 0;
  int32_t* d_tpos = nullptr;

  int rowset(int head, int kvh, int row0, int nrows) {
    auto key = std::make_pair(head, row0);
    auto it = rowset_of.find(key);
    if (it != rowset_of.end()) return it->second;
    RowSet r{};
    r.head = head; r.kvh = kvh; r.row0 = row0; r.nrows = nrows;
    r.nchunks = (row0 + nrows + chunk_keys - 1) / chunk_keys;
    r.part = dalloc<float>(P, (size_t)r.nchunks * LASTQ * 2);
    r.lse2 = dalloc<float>(P, LASTQ);
    max_chunks = std::max(max_chunks, r.nchunks);
    rowsets.push_back(r);
    P->est_lse2.push_back(r.lse2);
    P->rowset_n.push_back(nrows);
    return rowset_of[key] = (int)rowsets.size() - 1;
  }

  // estimation job; gi_key = key group (-1 = global positions)
  EstInfo est(int head, int kvh, int row0, int nrows, int coord0, int gi_key, int L_c, bool need_u) {
    EstInfo e;
    e.rowset = rowset(head, kvh, row0, nrows);
    EstJob j{};
    j.head = head; j.kvh = kvh; j.row0 = row0; j.nrows = nrows; j.rowset = e.rowset;
    j.coord0 = coord0;
    j.keymap = gi_key >= 0 ? d_tpos + L.g.toff[gi_key] : nullptr;
    j.L_c = L_c;
    j.ntiles = (L_c + B - 1) / B;
    j.v = dalloc<float>(P, L_c);
    j.u = need_u ? dalloc<float>(P, L_c) : nullptr;
    j.dpart = need_u ? dalloc<float>(P, (size_t)j.ntiles * 128) : nullptr;
    max_tiles = std::max(max_tiles, j.ntiles);
    max_L = std::max(max_L, L_c);
    e.job = (int)jobs.size();
    e.L_c = L_c; e.nrows = nrows; e.row0 = row0;
    e.v = j.v; e.u = j.u;
    jobs.push_back(j);
    return e;
  }

  void grid(EstInfo& e, const mmi_op& op, int32_t* params) {
    GridJob gj{};
    gj.v = e.v;
    gj.L_c = e.L_c;
    gj.lo = std::max(1, op.stride_lo);
    gj.hi = std::min(op.stride_hi, e.L_c / 2);
    const int nc = std::max(0, gj.hi - gj.lo + 1);
    gj.fold = dalloc<float>(P, (size_t)std::max(nc, 1) * FOLD_W);
    gj.score = dalloc<float>(P, std::max(nc, 1));
    gj.pick = dalloc<int32_t>(P, std::max(nc, 1));
    gj.params = params;
    gj.nrows = e.nrows;
    max_cands = std::max(max_cands, nc);
    e.fold = gj.fold; e.lo = gj.lo; e.hi = gj.hi; e.params = params;
    gjobs.push_back(gj);
  }

  int32_t* topk(const float* x, int L, int n) {
    n = std::min(n, L);
    int32_t* out = dalloc<int32_t>(P, std::max(n, 1));
    if (n > 0) tjobs.push_back({x, L, n, out});
    max_sel = std::max(max_sel, n);
    return out;
  }
};

static_assert(sizeof(mmi_op) == 80 && sizeof(mmi_head_cfg) == 4 + 73 * 80, "mmi.h struct layout");

static int natten_tiles(const mmi_op& o) {
  return ((o.grid_t + o.tile_t - 1) / o.tile_t) * ((o.grid_h + o.tile_h - 1) / o.tile_h) *
         ((o.grid_w + o.tile_w - 1) / o.tile_w);
}

static void check_natten(const mmi_op& o, int64_t S, int h) {
  const int g[3] = {o.grid_t, o.grid_h, o.grid_w}, w[3] = {o.win_t, o.win_h, o.win_w};
  const int t[3] = {o.tile_t, o.tile_h, o.tile_w};
  for (int a = 0; a < 3; ++a) {
    if (g[a] < 1 || t[a] < 1) fail(MMI_ERR_BAD_CONFIG, "head %d: NATTEN grid and tile sizes must be >= 1", h);
    if (w[a] < 1 || w[a] > g[a] || w[a] % 2 == 0)
      fail(MMI_ERR_BAD_CONFIG, "head %d: NATTEN window %d on an axis of %d (odd, 1..axis)", h, w[a], g[a]);
  }
  if ((int64_t)g[0] * g[1] * g[2] != S)
    fail(MMI_ERR_BAD_CONFIG, "head %d: NATTEN grid %dx%dx%d != S", h, g[0], g[1], g[2]);
  if (t[0] * t[1] * t[2] != B) fail(MMI_ERR_BAD_CONFIG, "head %d: NATTEN tile must hold 64 tokens", h);
  if ((int64_t)natten_tiles(o) > MMI_MAX_SEQ / B)
    fail(MMI_ERR_UNSUPPORTED, "head %d: %d NATTEN tiles exceed %d blocks", h, natten_tiles(o), MMI_MAX_SEQ / B);
}

// Key layouts of a Q-Boundary head: the position order (if some modality is
// not Grid) and one Grid order per Grid modality.
static int qb_grid_mods(const Groups& g, const mmi_head_cfg& c) {
  int n = 0;
  for (int gi = 0; gi < g.n; ++gi) n += c.intra[g.mod[gi]].kind == MMI_OP_GRID;
  return n;
}

static int qb_layouts(const Groups& g, const mmi_head_cfg& c) {
  const int n = qb_grid_mods(g, c);
  return n + (n < g.n ? 1 : 0);
}

static void validate_cfgs(const Groups& g, const mmi_problem& p, const mmi_head_cfg* cfgs) {
  for (int h = 0; h < p.Hq; ++h) {
    const mmi_head_cfg& c = cfgs[h];
    if (c.kind == MMI_HEAD_GLOBAL) {
      check_op(c.global, {MMI_OP_DENSE, MMI_OP_ASHAPE, MMI_OP_VSLASH, MMI_OP_GRID, MMI_OP_SF_FIXED,
                          MMI_OP_SF_STRIDED, MMI_OP_TRISHAPE, MMI_OP_NATTEN}, "a global head", h);
      if (c.global.kind == MMI_OP_NATTEN) check_natten(c.global, p.S, h);
    } else if (c.kind == MMI_HEAD_QBOUNDARY) {
      for (int gi = 0; gi < g.n; ++gi)
        check_op(c.intra[g.mod[gi]], {MMI_OP_DENSE, MMI_OP_ASHAPE, MMI_OP_VSLASH, MMI_OP_GRID, MMI_OP_SF_FIXED,
                                      MMI_OP_SF_STRIDED, MMI_OP_TRISHAPE}, "a Q-Boundary modality", h);
      const int nlay = qb_layouts(g, c);
      const int64_t nb = (p.S + B - 1) / B;
      if (nlay > 1 && nlay * nb > MMI_MAX_SEQ / B)
        fail(MMI_ERR_UNSUPPORTED, "head %d: %d key layouts of %lld blocks exceed %d key blocks", h, nlay,
             (long long)nb, MMI_MAX_SEQ / B);
    } else if (c.kind == MMI_HEAD_2D) {
      for (int a = 0; a < g.n; ++a)
        for (int b2 = 0; b2 < g.n; ++b2) {
          if (a == b2)
            check_op(c.intra[g.mod[a]], {MMI_OP_DENSE, MMI_OP_ASHAPE, MMI_OP_VSLASH, MMI_OP_GRID, MMI_OP_SF_FIXED,
                                         MMI_OP_SF_STRIDED, MMI_OP_TRISHAPE}, "a 2D-Boundary intra pair", h);
          else
            check_op(c.cross[g.mod[a]][g.mod[b2]], {MMI_OP_NONE, MMI_OP_DENSE, MMI_OP_VERT},
                     "a 2D-Boundary cross pair", h);
        }
    } else {
      fail(MMI_ERR_BAD_CONFIG, "head %d: unknown head kind %d", h, c.kind);
    }
  }

}

static void validate_inputs(const mmi_problem* prob, const mmi_head_cfg* cfgs, const void* q, const void* k) {
  const mmi_problem p = normalise(prob);
  if (!cfgs) fail(MMI_ERR_INVALID_ARG, "cfgs is NULL");
  if (!q || !k) fail(MMI_ERR_INVALID_ARG, "q/k is NULL");
  aligned16(q, "q");
  aligned16(k, "k");
  const Layout L = make_layout(p);
  validate_cfgs(L.g, p, cfgs);
}

static void build_item_map(mmi_plan* P, hipStream_t st);

static void plan_create_impl(mmi_ctx* ctx, const mmi_problem* prob_in, const mmi_head_cfg* cfgs, const void* q,
                             const void* k, hipStream_t st, mmi_plan* P) {
  const mmi_problem p = normalise(prob_in);
  if (!cfgs) fail(MMI_ERR_INVALID_ARG, "cfgs is NULL");
  if (!q || !k) fail(MMI_ERR_INVALID_ARG, "q/k is NULL");
  aligned16(q, "q");
  aligned16(k, "k");
  P->ctx = ctx;
  P->stream = st;
  P->prob = p;
  P->prob.modality = nullptr;
  P->mod.assign((size_t)p.S, 0);
  if (p.modality) std::copy(p.modality, p.modality + p.S, P->mod.begin());
  P->S = (int)p.S; P->Hq = p.Hq; P->Hkv = p.Hkv;
  const int S = P->S, G = p.Hq / p.Hkv;
  Builder bd;
  bd.P = P;
  bd.L = make_layout(p);
  const Layout& L = bd.L;
  const Groups& g = L.g;
  P->groups = g;
  validate_cfgs(g, p, cfgs);

  HIPCHK(hipSetDevice(ctx->device));
  // positions of each modality
  std::vector<int32_t> toff_by_mod(MMI_MAX_MODALITIES, 0);
  for (int gi = 0; gi < g.n; ++gi) toff_by_mod[g.mod[gi]] = g.toff[gi];
  Segment* d_segs = nullptr;
  int32_t* d_toff = nullptr;
  {
    Pack pk;
    pk.add(L.segs, d_segs);
    pk.add(toff_by_mod, d_toff);
    send(P, pk);
  }
  bd.d_tpos = P->d_tpos = dalloc<int32_t>(P, S);
  bool qb_grid = false;
  for (int h = 0; h < p.Hq; ++h) qb_grid |= cfgs[h].kind == MMI_HEAD_QBOUNDARY && qb_grid_mods(g, cfgs[h]) > 0;
  uint8_t* d_modpos = qb_grid ? dalloc<uint8_t>(P, S) : nullptr;
  HIPCHK(launch_positions(d_segs, (int)L.segs.size(), d_toff, bd.d_tpos, d_modpos, S, st));
  std::vector<QbOrderJob> qjobs;

  const int nb_all = (S + B - 1) / B;
  int nb_groups = 0;
  for (int gi = 0; gi < g.n; ++gi) nb_groups += (g.len[gi] + B - 1) / B;

  P->hh.resize(p.Hq);
  int max_slots = 0, max_nbq = 0, max_nbk = 0, max_groups = 0;
  const int R = ctx->row_group;
  P->R = R;
  for (int h = 0; h < p.Hq; ++h) {
    const mmi_head_cfg& c = cfgs[h];
    HostHead& H = P->hh[h];
    HeadDev hd{};
    hd.kind = c.kind;
    hd.kvh = h / G;
    hd.S = S;
    hd.op0 = (int)P->ops.size();
    H.kind = c.kind;
    H.op0 = hd.op0;
    auto base_op = [&](const mmi_op& o) {
      OpDev d{};
      d.kind = o.kind;
      d.sink = o.sink; d.local = o.local;
      d.use_h = o.use_h != 0; d.use_v = o.use_v != 0; d.use_s = o.use_s != 0;
      d.stride = o.stride_lo; d.bottom = o.bottom;
      d.grid[0] = o.grid_t; d.grid[1] = o.grid_h; d.grid[2] = o.grid_w;
      d.win[0] = o.win_t; d.win[1] = o.win_h; d.win[2] = o.win_w;
      d.tile[0] = o.tile_t; d.tile[1] = o.tile_h; d.tile[2] = o.tile_w;
      return d;
    };
    hd.causal = 1;
    if (c.kind == MMI_HEAD_GLOBAL && c.global.kind == MMI_OP_NATTEN) {
      // tile-permuted queries and keys, one block per tile, bidirectional
      hd.nbq = hd.nbk = natten_tiles(c.global);
      hd.causal = 0;
      hd.qperm = dalloc<int32_t>(P, (size_t)hd.nbq * B);
      hd.kperm = hd.qperm;
      hd.kminpos = dalloc<int32_t>(P, hd.nbk);
      hd.kmaxpos = dalloc<int32_t>(P, hd.nbk);
      OpDev d = base_op(c.global);
      d.L = S; d.kbase = 0; d.nkblk = hd.nbk;
      P->ops.push_back(d);
      H.est.push_back(EstInfo{});
      H.op_slot.push_back(0);
    } else if (c.kind == MMI_HEAD_GLOBAL) {
      hd.nbq = hd.nbk = nb_all;
      OpDev d = base_op(c.global);
      d.L = S; d.kbase = 0; d.nkblk = nb_all;
      EstInfo e;
      const int nrows = std::min(LASTQ, S), row0 = S - nrows;
      if (c.global.kind == MMI_OP_GRID || c.global.kind == MMI_OP_VSLASH) {
        e = bd.est(h, hd.kvh, row0, nrows, row0, -1, S, c.global.kind == MMI_OP_VSLASH);
        if (c.global.kind == MMI_OP_GRID) {
          int32_t* params = dalloc<int32_t>(P, 4);
          bd.grid(e, c.global, params);
          d.params = params;
        } else {
          e.vsel = bd.topk(e.v, e.L_c, c.global.n_vertical);
          e.ssel = bd.topk(e.u, e.L_c, c.global.n_slash);
          e.nv = std::min(c.global.n_vertical, e.L_c);
          e.ns = std::min(c.global.n_slash, e.L_c);
          d.vsel = e.vsel; d.nv = e.nv; d.ssel = e.ssel; d.ns = e.ns;
          d.selpb = dalloc<int2>(P, d.nv);
        }
      }
      if (c.global.kind == MMI_OP_GRID) {
        hd.qperm = dalloc<int32_t>(P, (size_t)nb_all * B);
        hd.kperm = hd.qperm;
        hd.kminpos = dalloc<int32_t>(P, nb_all);
        hd.kmaxpos = dalloc<int32_t>(P, nb_all);
      }
      P->ops.push_back(d);
      H.est.push_back(e);
      H.op_slot.push_back(0);
    } else if (c.kind == MMI_HEAD_QBOUNDARY) {
      hd.nbq = nb_groups;
      hd.qperm = dalloc<int32_t>(P, (size_t)nb_groups * B);
      const int ngrid = qb_grid_mods(g, c);
      hd.nbk = ngrid ? qb_layouts(g, c) * nb_all : nb_all;
      if (ngrid) {          // key layouts: [position order] then one Grid order per Grid modality
        hd.kperm = dalloc<int32_t>(P, (size_t)hd.nbk * B);
        hd.kminpos = dalloc<int32_t>(P, hd.nbk);
        hd.kmaxpos = dalloc<int32_t>(P, hd.nbk);
      }
      int next_layout = ngrid < g.n ? 1 : 0;
      for (int gi = 0; gi < g.n; ++gi) {
        const mmi_op& o = c.intra[g.mod[gi]];
        OpDev d = base_op(o);
        d.L = S; d.nkblk = nb_all;
        d.kbase = o.kind == MMI_OP_GRID ? (next_layout++) * nb_all : 0;
        EstInfo e;
        if (o.kind == MMI_OP_GRID) {
          int row0, nrows, loc0;
          final_rows(L, gi, row0, nrows, loc0);
          e = bd.est(h, hd.kvh, row0, nrows, row0, -1, row0 + nrows, false);
          int32_t* params = dalloc<int32_t>(P, 4);
          bd.grid(e, o, params);
          d.params = params;
          qjobs.push_back({params, hd.qperm + g.off[gi], g.mod[gi], dalloc<int32_t>(P, qb_order_chunks(S))});
        } else if (o.kind == MMI_OP_VSLASH) {
          int row0, nrows, loc0;
          final_rows(L, gi, row0, nrows, loc0);
          e = bd.est(h, hd.kvh, row0, nrows, row0, -1, row0 + nrows, true);
          e.vsel = bd.topk(e.v, e.L_c, o.n_vertical);
          e.ssel = bd.topk(e.u, e.L_c, o.n_slash);
          e.nv = std::min(o.n_vertical, e.L_c);
          e.ns = std::min(o.n_slash, e.L_c);
          d.vsel = e.vsel; d.nv = e.nv; d.ssel = e.ssel; d.ns = e.ns;
          d.selpb = dalloc<int2>(P, d.nv);
        }
        P->ops.push_back(d);
        H.est.push_back(e);
        H.op_slot.push_back(g.mod[gi]);
      }
    } else {
      hd.nbq = hd.nbk = nb_groups;
      hd.qperm = dalloc<int32_t>(P, (size_t)nb_groups * B);
      hd.kperm = hd.qperm;
      hd.kminpos = dalloc<int32_t>(P, nb_groups);
      hd.kmaxpos = dalloc<int32_t>(P, nb_groups);
      const int n0 = (int)P->ops.size();
      P->ops.resize(n0 + g.n * g.n);
      H.est.resize(g.n * g.n);
      H.op_slot.resize(g.n * g.n);
      // intra ops first (cross VERT into a Grid group needs that group's params)
      for (int gi = 0; gi < g.n; ++gi) {
        const mmi_op& o = c.intra[g.mod[gi]];
        OpDev d = base_op(o);
        d.L = g.len[gi]; d.kbase = g.off[gi] / B; d.nkblk = (g.len[gi] + B - 1) / B;
        d.keymap = bd.d_tpos + g.toff[gi];
        d.koff = g.off[gi];
        EstInfo e;
        if (o.kind == MMI_OP_GRID || o.kind == MMI_OP_VSLASH) {
          int row0, nrows, loc0;
          final_rows(L, gi, row0, nrows, loc0);
          e = bd.est(h, hd.kvh, row0, nrows, loc0, gi, g.len[gi], o.kind == MMI_OP_VSLASH);
          if (o.kind == MMI_OP_GRID) {
            int32_t* params = dalloc<int32_t>(P, 4);
            bd.grid(e, o, params);
            d.params = params;
          } else {
            e.vsel = bd.topk(e.v, e.L_c, o.n_vertical);
            e.ssel = bd.topk(e.u, e.L_c, o.n_slash);
            e.nv = std::min(o.n_vertical, e.L_c);
            e.ns = std::min(o.n_slash, e.L_c);
            d.vsel = e.vsel; d.nv = e.nv; d.ssel = e.ssel; d.ns = e.ns;
            d.selpb = dalloc<int2>(P, d.nv);
          }
        }
        P->ops[n0 + gi * g.n + gi] = d;
        H.est[gi * g.n + gi] = e;
        H.op_slot[gi * g.n + gi] = g.mod[gi];
      }
      for (int a = 0; a < g.n; ++a)
        for (int b2 = 0; b2 < g.n; ++b2) {
          if (a == b2) continue;
          const mmi_op& o = c.cross[g.mod[a]][g.mod[b2]];
          OpDev d = base_op(o);
          d.L = g.len[b2]; d.kbase = g.off[b2] / B; d.nkblk = (g.len[b2] + B - 1) / B;
          d.keymap = bd.d_tpos + g.toff[b2];
          d.koff = g.off[b2];
          const OpDev& kintra = P->ops[n0 + b2 * g.n + b2];
          d.kgrid = kintra.kind == MMI_OP_GRID ? 1 : 0;
          d.kparams = kintra.params;
          EstInfo e;
          if (o.kind == MMI_OP_VERT) {
            int row0, nrows, loc0;
            final_rows(L, a, row0, nrows, loc0);
            const int Lc = count_le(L, b2, row0 + nrows - 1);
            if (Lc > 0) {
              e = bd.est(h, hd.kvh, row0, nrows, 0, b2, Lc, false);
              e.vsel = bd.topk(e.v, e.L_c, o.n_vertical);
              e.nv = std::min(o.n_vertical, e.L_c);
            }
            d.vsel = e.vsel; d.nv = e.nv;
            d.selpb = dalloc<int2>(P, d.nv);
          }
          P->ops[n0 + a * g.n + b2] = d;
          H.est[a * g.n + b2] = e;
          H.op_slot[a * g.n + b2] = 8 + g.mod[a] * 8 + g.mod[b2];
        }
    }
    H.nops = (int)P->ops.size() - H.op0;
    hd.nwords = (hd.nbk + 31) / 32;
    hd.counts = dalloc<int32_t>(P, hd.nbq);
    hd.rowptr = dalloc<int32_t>(P, hd.nbq + 1);
    hd.bitmap = dalloc<uint32_t>(P, (size_t)hd.nbq * hd.nwords);
    if (c.kind == MMI_HEAD_GLOBAL && c.global.kind == MMI_OP_NATTEN) {
      // neighbouring tiles along h and along t as row-group members
      const int ntw = (c.global.grid_w + c.global.tile_w - 1) / c.global.tile_w;
      const int nth = (c.global.grid_h + c.global.tile_h - 1) / c.global.tile_h;
      hd.rho_alt[0] = ntw > 8 ? ntw : 0;
      hd.rho_alt[1] = nth * ntw > 8 && nth > 1 ? nth * ntw : 0;
    }
    const int max_rho = std::max(8, std::max(hd.rho_alt[0], hd.rho_alt[1]));
    hd.gcap = (hd.nbq + R - 1) / R + max_rho;   // >= groups_for(nbq, R, rho) for every candidate
    hd.gp = dalloc<int32_t>(P, 3);
    hd.gcount = dalloc<int32_t>(P, hd.gcap);
    hd.growptr = dalloc<int32_t>(P, hd.gcap + 1);
    hd.chunklen = dalloc<int32_t>(P, 1);
    hd.chunks = dalloc<int32_t>(P, hd.gcap);
    hd.itembase = dalloc<int32_t>(P, hd.gcap);
    hd.splitoff = dalloc<int32_t>(P, hd.gcap);
    hd.partoff = dalloc<int32_t>(P, hd.gcap);
    max_slots = std::max(max_slots, std::max(hd.nbq, hd.nbk) * B);
    max_nbq = std::max(max_nbq, hd.nbq);
    max_groups = std::max(max_groups, hd.gcap);
    max_nbk = std::max(max_nbk, hd.nbk);
    P->heads.push_back(hd);
  }

  // estimation -> choices
  const Tensor tq{q, p.q_stride_s, p.q_stride_h}, tk{k, p.k_stride_s, p.k_stride_h};
  if (!P->scratch)
    for (auto& e : P->ev) HIPCHK(hipEventCreate(&e));
  // members of the estimation groups that read the same keys: row sets per
  // KV head, score jobs per (KV head, key map)
  auto grouped = [](int n, auto key_of, int& ngrp, int& nr) {
    std::map<std::pair<int64_t, int64_t>, std::vector<int32_t>> by;
    for (int i = 0; i < n; ++i) by[key_of(i)].push_back(i);
    ngrp = (int)by.size();
    nr = 1;
    for (const auto& kv : by) nr = std::max(nr, (int)kv.second.size());
    std::vector<int32_t> order((size_t)std::max(ngrp, 1) * nr, -1);
    int gi = 0;
    for (const auto& kv : by) {
      std::copy(kv.second.begin(), kv.second.end(), order.begin() + (size_t)gi * nr);
      ++gi;
    }
    return order;
  };
  int rs_ngrp = 0, rs_nr = 1, job_ngrp = 0, job_nr = 1;
  const std::vector<int32_t> rs_order = grouped((int)bd.rowsets.size(), [&](int i) {
    return std::make_pair((int64_t)bd.rowsets[i].kvh, (int64_t)0); }, rs_ngrp, rs_nr);
  const std::vector<int32_t> job_order = grouped((int)bd.jobs.size(), [&](int i) {
    return std::make_pair((int64_t)bd.jobs[i].kvh, (int64_t)(intptr_t)bd.jobs[i].keymap); }, job_ngrp, job_nr);
  int32_t *d_rs_order = nullptr, *d_job_order = nullptr;
  RowSet* d_rs = nullptr;
  EstJob* d_jobs = nullptr;
  GridJob* d_g = nullptr;
  TopkJob* d_t = nullptr;
  QbOrderJob* d_qj = nullptr;
  {
    Pack pk;
    pk.add(bd.rowsets, d_rs);
    pk.add(bd.jobs, d_jobs);
    pk.add(bd.gjobs, d_g);
    pk.add(bd.tjobs, d_t);
    pk.add(P->heads, P->d_heads);
    pk.add(P->ops, P->d_ops);
    pk.add(qjobs, d_qj);
    pk.add(rs_order, d_rs_order);
    pk.add(job_order, d_job_order);
    send(P, pk);
  }
  mark(P, 0, st);
  HIPCHK(launch_est_lse(d_rs, (int)bd.rowsets.size(), d_rs_order, rs_ngrp, rs_nr, bd.max_chunks, tq, tk,
                        bd.chunk_keys, st));
  HIPCHK(launch_est_scores(d_jobs, (int)bd.jobs.size(), d_job_order, job_ngrp, job_nr, bd.max_tiles, d_rs, tq,
                           tk, st));
  HIPCHK(launch_est_udiag(d_jobs, (int)bd.jobs.size(), bd.max_L, st));
  mark(P, 1, st);
  HIPCHK(launch_grid_search(d_g, (int)bd.gjobs.size(), bd.max_cands, st));
  int32_t* d_tscr = dalloc<int32_t>(P, topk_scratch_ints((int)bd.tjobs.size()));
  HIPCHK(launch_topk(d_t, (int)bd.tjobs.size(), d_tscr, st));
  mark(P, 2, st);

  // permutations, key summaries, block counts
  HIPCHK(launch_perms(P->d_heads, p.Hq, P->d_ops, g, bd.d_tpos, S, max_slots, st));
  HIPCHK(launch_qb_order(d_qj, (int)qjobs.size(), d_modpos, S, st));
  HIPCHK(launch_key_summaries(P->d_heads, p.Hq, P->d_ops, (int)P->ops.size(), g, max_nbk, bd.max_sel, st));
  const int chunk = ctx->chunk_blocks;
  HIPCHK(launch_blocks_count(P->d_heads, p.Hq, P->d_ops, g, max_nbq, st));
  int64_t* d_cand = dalloc<int64_t>(P, (size_t)p.Hq * NRHO);
  int32_t* d_gcnt = dalloc<int32_t>(P, (size_t)p.Hq * NRHO * std::max(max_groups, 1));
  bool extra_rho = false;
  for (const HeadDev& hd : P->heads) extra_rho = extra_rho || hd.rho_alt[0] > 0 || hd.rho_alt[1] > 0;
  HIPCHK(launch_group_stride(P->d_heads, p.Hq, R, max_groups, max_nbq, extra_rho, d_cand, d_gcnt, st));
  HIPCHK(launch_group_count(P->d_heads, p.Hq, d_gcnt, max_groups, st));
  const size_t ntot = (size_t)p.Hq * NTOT;
  int64_t* d_tot = dalloc<int64_t>(P, ntot);
  const int items_per_head = std::max(1, ctx->items_per_layer / p.Hq);
  // When the row groups alone already give the target number of work items,
  // only groups far above their head's average are split (a split puts
  // chunks of one union side by side on an XCD, which share no key blocks,
  // in place of neighbouring groups, which do).
  int64_t groups_all = 0;
  for (const auto& hd : P->heads) groups_all += (hd.nbq + R - 1) / R;
  const int split_above_avg = groups_all >= ctx->items_per_layer ? ctx->split_above_avg : 0;
  HIPCHK(launch_blocks_scan(P->d_heads, p.Hq, chunk, items_per_head, split_above_avg, d_tot, st));
  std::vector<int64_t> tot_host;
  const int64_t* tot = nullptr;
  if (P->scratch) {                      // pageable host copy: no pinned allocation
    tot_host.resize(ntot);
    HIPCHK(hipMemcpyAsync(tot_host.data(), d_tot, sizeof(int64_t) * ntot, hipMemcpyDeviceToHost, st));
    tot = tot_host.data();
  } else {
    if (ctx->pinned_n < ntot) {
      if (ctx->pinned) HIPCHK(hipHostFree(ctx->pinned));
      ctx->pinned = nullptr;
      HIPCHK(hipHostMalloc((void**)&ctx->pinned, sizeof(int64_t) * ntot));
      ctx->pinned_n = ntot;
    }
    HIPCHK(hipMemcpyAsync(ctx->pinned, d_tot, sizeof(int64_t) * ntot, hipMemcpyDeviceToHost, st));
    tot = ctx->pinned;
  }
  HIPCHK(hipStreamSynchronize(st));

  // sizes known: column pools, work items, partials
  std::vector<int64_t> item_base(p.Hq), part_base(p.Hq), split_base(p.Hq);
  int64_t nnz_all = 0, gnnz_all = 0;
  for (int h = 0; h < p.Hq; ++h) {
    HostHead& H = P->hh[h];
    const int64_t* t = tot + (size_t)h * NTOT;
    H.nnz = t[0];
    H.gnnz = t[1];
    H.nitems = t[2];
    H.nsplit = t[3];
    H.nparts = t[4];
    gnnz_all += H.gnnz;
    item_base[h] = P->nitems;
    part_base[h] = P->nparts;
    split_base[h] = P->nsplit;
    P->nitems += H.nitems;
    P->nparts += H.nparts;
    P->nsplit += H.nsplit;
    nnz_all += H.nnz;
  }
  if (P->nitems > 0x7fffffff || P->nparts > 0x7fffffff)
    fail(MMI_ERR_UNSUPPORTED, "work list too large (%lld items)", (long long)P->nitems);
  int32_t* col = dalloc<int32_t>(P, nnz_all);
  int32_t* gcol = dalloc<int32_t>(P, gnnz_all);
  int64_t off = 0, goff = 0;
  for (int h = 0; h < p.Hq; ++h) {
    P->heads[h].col = col + off;
    P->heads[h].gcol = gcol + goff;
    off += P->hh[h].nnz;
    goff += P->hh[h].gnnz;
  }
  P->keep.emplace_back(reinterpret_cast<const uint8_t*>(P->heads.data()),
                       reinterpret_cast<const uint8_t*>(P->heads.data()) + sizeof(HeadDev) * p.Hq);
  HIPCHK(hipMemcpyAsync(P->d_heads, P->keep.back().data(), sizeof(HeadDev) * p.Hq, hipMemcpyHostToDevice, st));
  HIPCHK(launch_blocks_fill(P->d_heads, p.Hq, max_nbq, R, max_groups, st));
  P->d_items = dalloc<WorkItem>(P, P->nitems);
  P->d_splits = dalloc<SplitRow>(P, P->nsplit);
  P->d_part_o = dalloc<float>(P, (size_t)std::max<int64_t>(P->nparts, 1) * B * R * D);
  P->d_part_ml = dalloc<float>(P, (size_t)std::max<int64_t>(P->nparts, 1) * B * R * 4);
  int64_t *d_ib = nullptr, *d_pb = nullptr, *d_sb = nullptr;
  {
    Pack pk;
    pk.add(item_base, d_ib);
    pk.add(part_base, d_pb);
    pk.add(split_base, d_sb);
    send(P, pk);
  }
  HIPCHK(launch_work_fill(P->d_heads, p.Hq, d_ib, d_pb, d_sb, max_groups, P->d_items, P->d_splits, st));
  build_item_map(P, st);
  mark(P, 3, st);
  P->nnz_all = nnz_all;
  P->gnnz_all = gnnz_all;
}

// Work items of each XCD. Items (row groups, or chunks of long ones, in head
// and group order) are cut into runs of consecutive items, which share key
// blocks; the runs are dealt to the 8 XCDs longest first, each to the XCD
// with the least modelled cost so far (at most a quarter more runs than the
// average per XCD), and each XCD runs its runs in that order. Runs are 32
// items, fewer for small layers so that every XCD gets some.
static void build_item_map(mmi_plan* P, hipStream_t st) {
  const int64_t n = P->nitems;
  if (n <= 0) return;
  float* d_cost = dalloc<float>(P, n);
  HIPCHK(launch_item_cost(P->d_heads, P->d_items, n, d_cost, st));
  std::vector<float> cost(n);
  HIPCHK(hipMemcpyAsync(cost.data(), d_cost, sizeof(float) * n, hipMemcpyDeviceToHost, st));
  HIPCHK(hipStreamSynchronize(st));
  const int64_t run = std::max<int64_t>(1, std::min<int64_t>(32, n / 64));
  const int64_t nruns = (n + run - 1) / run;
  std::vector<double> rc(nruns, 0.0);
  for (int64_t i = 0; i < n; ++i) rc[i / run] += cost[i];
  std::vector<int64_t> order(nruns);
  for (int64_t j = 0; j < nruns; ++j) order[j] = j;
  std::stable_sort(order.begin(), order.end(), [&](int64_t x, int64_t y) { return rc[x] > rc[y]; });
  const int64_t avg = (nruns + 7) / 8, cap = avg + std::max<int64_t>(1, avg / 4);
  double load[8] = {0};
  std::vector<int64_t> runs_of[8];
  for (int64_t j : order) {
    int best = -1;
    for (int x = 0; x < 8; ++x)
      if ((int64_t)runs_of[x].size() < cap && (best < 0 || load[x] < load[best])) best = x;
    runs_of[best].push_back(j);
    load[best] += rc[j];
  }
  int64_t len = 0;
  std::vector<int64_t> items_of(8, 0);
  for (int x = 0; x < 8; ++x) {
    for (int64_t j : runs_of[x]) items_of[x] += std::min(run, n - j * run);
    len = std::max(len, items_of[x]);
  }
  std::vector<int32_t> map((size_t)8 * len, -1);
  for (int x = 0; x < 8; ++x) {
    int64_t k = 0;
    for (int64_t j : runs_of[x])
      for (int64_t i = j * run; i < std::min(n, (j + 1) * run); ++i) map[(size_t)x * len + k++] = (int32_t)i;
  }
  Pack pk;
  pk.add(map, P->d_item_map);
  send(P, pk);
  P->map_len = len;
}

// The debug check of a plan: its tables copied to the host, each head's
// block index and row-group unions, then the work list and item map.
static void plan_check(mmi_plan* P) {
  HIPCHK(hipSetDevice(P->ctx->device));
  HIPCHK(hipStreamSynchronize(P->stream));
  auto get = [](const int32_t* src, size_t n) {
    std::vector<int32_t> v(std::max<size_t>(n, 1));
    if (n) HIPCHK(hipMemcpy(v.data(), src, n * 4, hipMemcpyDeviceToHost));
    return v;
  };
  const int nb_all = (P->S + B - 1) / B;
  std::vector<int32_t> ngroups(P->Hq);
  std::vector<std::vector<int32_t>> uptr(P->Hq);
  for (int h = 0; h < P->Hq; ++h) {
    const HeadDev& hd = P->heads[h];
    const HostHead& H = P->hh[h];
    const std::vector<int32_t> gp = get(hd.gp, 3);
    if (gp[0] < 1 || gp[1] < 0 || gp[1] > hd.gcap)
      fail(MMI_ERR_INTERNAL, "plan check, head %d: row stride %d, %d row groups (capacity %d)", h, gp[0], gp[1],
           hd.gcap);
    const std::vector<int32_t> qp = hd.qperm ? get(hd.qperm, (size_t)hd.nbq * B) : std::vector<int32_t>();
    const std::vector<int32_t> kp = hd.kperm ? get(hd.kperm, (size_t)hd.nbk * B) : std::vector<int32_t>();
    const std::vector<int32_t> rp = get(hd.rowptr, hd.nbq + 1), col = get(hd.col, H.nnz);
    uptr[h] = get(hd.growptr, (size_t)gp[1] + 1);
    const std::vector<int32_t> ent = get(hd.gcol, H.gnnz);
    if (rp[hd.nbq] != H.nnz || uptr[h][gp[1]] != H.gnnz)
      fail(MMI_ERR_INTERNAL, "plan check, head %d: %d / %d entries, the plan sized %lld / %lld", h, rp[hd.nbq],
           uptr[h][gp[1]], (long long)H.nnz, (long long)H.gnnz);
    mmi_index_view v{};
    v.S = P->S;
    v.n_qblocks = hd.nbq;
    v.n_kblocks = hd.nbk;
    v.n_layouts = H.kind == MMI_HEAD_QBOUNDARY && hd.kperm ? hd.nbk / nb_all : 1;
    v.causal = hd.causal;
    v.qperm = hd.qperm ? qp.data() : nullptr;
    v.kperm = hd.kperm ? kp.data() : nullptr;
    v.row_ptr = rp.data();
    v.col_idx = col.data();
    v.group_size = P->R;
    v.group_stride = gp[0];
    v.n_groups = gp[1];
    v.union_ptr = uptr[h].data();
    v.union_ent = ent.data();
    const std::string e = check_index(v);
    if (!e.empty()) fail(MMI_ERR_INTERNAL, "plan check, head %d: %s", h, e.c_str());
    ngroups[h] = gp[1];
  }
  std::vector<WorkItem> items(std::max<int64_t>(P->nitems, 1));
  std::vector<SplitRow> splits(std::max<int64_t>(P->nsplit, 1));
  if (P->nitems) HIPCHK(hipMemcpy(items.data(), P->d_items, sizeof(WorkItem) * P->nitems, hipMemcpyDeviceToHost));
  if (P->nsplit) HIPCHK(hipMemcpy(splits.data(), P->d_splits, sizeof(SplitRow) * P->nsplit, hipMemcpyDeviceToHost));
  const std::vector<int32_t> map = P->map_len ? get(P->d_item_map, (size_t)8 * P->map_len) : std::vector<int32_t>();
  std::vector<int32_t> it5((size_t)5 * std::max<int64_t>(P->nitems, 1)), sp4((size_t)4 * std::max<int64_t>(P->nsplit, 1));
  for (int64_t i = 0; i < P->nitems; ++i) {
    const WorkItem& w = items[i];
    const int32_t r[5] = {w.head, w.group, w.e0, w.e1, w.part};
    std::copy(r, r + 5, it5.begin() + 5 * i);
  }
  for (int64_t i = 0; i < P->nsplit; ++i) {
    const SplitRow& sr = splits[i];
    const int32_t r[4] = {sr.head, sr.group, sr.part0, sr.nparts};
    std::copy(r, r + 4, sp4.begin() + 4 * i);
  }
  std::vector<const int32_t*> up(P->Hq);
  for (int h = 0; h < P->Hq; ++h) up[h] = uptr[h].data();
  mmi_work_view w{};
  w.n_heads = P->Hq;
  w.n_groups = ngroups.data();
  w.union_ptr = up.data();
  w.n_items = P->nitems;
  w.items = it5.data();
  w.n_parts = P->nparts;
  w.n_splits = P->nsplit;
  w.splits = sp4.data();
  w.map_len = P->map_len;
  w.item_map = map.empty() ? nullptr : map.data();
  const std::string e = check_work(w);
  if (!e.empty()) fail(MMI_ERR_INTERNAL, "plan check, work list: %s", e.c_str());
}

static void plan_execute_impl(mmi_plan* P, const void* q, const void* k, const void* v, void* o, float* lse,
                              hipStream_t st) {
  if (!q || !k || !v || !o) fail(MMI_ERR_INVALID_ARG, "q/k/v/o is NULL");
  aligned16(q, "q"); aligned16(k, "k"); aligned16(v, "v"); aligned16(o, "o");
  if (o == q || o == k || o == v) fail(MMI_ERR_INVALID_ARG, "o aliases an input");
  HIPCHK(hipSetDevice(P->ctx->device));
  const mmi_problem& p = P->prob;
  AttnArgs a{};
  a.q = {q, p.q_stride_s, p.q_stride_h};
  a.k = {k, p.k_stride_s, p.k_stride_h};
  a.v = {v, p.v_stride_s, p.v_stride_h};
  a.o = o; a.o_ss = p.o_stride_s; a.o_sh = p.o_stride_h;
  a.lse = lse;
  a.S = P->S;
  a.heads = P->d_heads;
  a.items = P->d_items;
  a.nitems = P->nitems;
  a.part_o = P->d_part_o;
  a.part_ml = P->d_part_ml;
  a.item_map = P->d_item_map;
  a.map_len = P->map_len;
  a.R = P->R;
  mark(P, 4, st);
  HIPCHK(launch_attention(a, st));
  mark(P, 5, st);
  HIPCHK(launch_combine(a, P->d_splits, P->nsplit, st));
  mark(P, 6, st);
  P->stream = st;
  P->executed = true;
}

}  // namespace mmi

// ====================================================================== C ABI
using namespace mmi;

template <typename F>
static int guarded(F&& f) {
  try {
    f();
    return MMI_OK;
  } catch (const Error& e) {
    g_last_error = e.what();
    return e.code;
  } catch (const std::bad_alloc&) {
    g_last_error = "host allocation failed";
    return MMI_ERR_OOM;
  } catch (const std::exception& e) {
    g_last_error = e.what();
    return MMI_ERR_INTERNAL;
  } catch (...) {
    g_last_error = "unknown error";
    return MMI_ERR_INTERNAL;
  }
}

extern "C" {

int mmi_version(void) { return MMI_ABI_VERSION; }

const char* mmi_status_str(int s) {
  switch (s) {
    case MMI_OK: return "ok";
    case MMI_ERR_INVALID_ARG: return "invalid argument";
    case MMI_ERR_UNSUPPORTED: return "unsupported shape";
    case MMI_ERR_BAD_CONFIG: return "bad head config";
    case MMI_ERR_OOM: return "out of device memory";
    case MMI_ERR_HIP: return "HIP runtime error";
    case MMI_ERR_STATE: return "invalid state";
    case MMI_ERR_INTERNAL: return "internal error";
    default: return "unknown status";
  }
}

const char* mmi_last_error(void) { return g_last_error.c_str(); }

int mmi_ctx_create(int device, mmi_ctx** out) {
  return guarded([&] {
    if (!out) fail(MMI_ERR_INVALID_ARG, "out is NULL");
    int n = 0;
    HIPCHK(hipGetDeviceCount(&n));
    if (device < 0 || device >= n) fail(MMI_ERR_INVALID_ARG, "device %d of %d", device, n);
    HIPCHK(hipSetDevice(device));
    scratch_setup(device);
    auto* c = new mmi_ctx();
    c->device = device;
    if (const char* e = getenv("MMI_CHUNK_BLOCKS")) {
      const int v = atoi(e);
      if (v >= 1) c->chunk_blocks = v;
    }
    if (const char* e = getenv("MMI_ITEMS_PER_LAYER")) {
      const int v = atoi(e);
      if (v >= 1) c->items_per_layer = v;
    }
    if (const char* e = getenv("MMI_SPLIT_ABOVE_AVG")) {
      const int v = atoi(e);
      if (v >= 0) c->split_above_avg = v;
    }
    if (const char* e = getenv("MMI_DEBUG")) c->debug = e[0] != '\0' && strcmp(e, "0") != 0;
    if (const char* e = getenv("MMI_ROW_GROUP")) {
      const int v = atoi(e);
      if (v == 1 || v == 2 || v == 4) c->row_group = v;
    }
    *out = c;
  });
}

int mmi_ctx_destroy(mmi_ctx* ctx) {
  return guarded([&] {
    if (!ctx) fail(MMI_ERR_INVALID_ARG, "ctx is NULL");
    if (ctx->live_plans > 0)
      fail(MMI_ERR_STATE, "context still has %d live plan(s); destroy them first", ctx->live_plans);
    (void)hipSetDevice(ctx->device);
    (void)hipDeviceSynchronize();
    if (ctx->pinned) (void)hipHostFree(ctx->pinned);
    delete ctx;
  });
}

// Plan creation shared by mmi_plan_create (scratch_base NULL: buffers from the
// context's allocator) and mmi_attention_noalloc (buffers in the scratch).
static int create_plan(mmi_ctx* ctx, const mmi_problem* prob, const mmi_head_cfg* cfgs, const void* q,
                       const void* k, void* stream, uint8_t* scratch_base, mmi_plan** out) {
  mmi_plan* P = nullptr;
  int rc = guarded([&] {
    validate_inputs(prob, cfgs, q, k);     // host-only checks first
    if (!ctx || !out) fail(MMI_ERR_INVALID_ARG, "ctx/out is NULL");
    P = new mmi_plan();
    P->scratch = scratch_base;
    plan_create_impl(ctx, prob, cfgs, q, k, (hipStream_t)stream, P);
    if (ctx->debug) plan_check(P);
  });
  if (rc != MMI_OK) {
    if (P) {
      if (P->ctx) {
        (void)hipStreamSynchronize((hipStream_t)stream);
        free_plan_buffers(P);
      }
      for (auto& e : P->ev)
        if (e) (void)hipEventDestroy(e);
      delete P;
    }
    return rc;
  }
  ++ctx->live_plans;
  *out = P;
  return MMI_OK;
}

int mmi_plan_create(mmi_ctx* ctx, const mmi_problem* prob, const mmi_head_cfg* cfgs, const void* q,
                    const void* k, void* stream, mmi_plan** out) {
  return create_plan(ctx, prob, cfgs, q, k, stream, nullptr, out);
}

int mmi_plan_execute(mmi_plan* plan, const void* q, const void* k, const void* v, void* o, float* lse,
                     void* stream) {
  return guarded([&] {
    if (!plan) fail(MMI_ERR_STATE, "plan is NULL");
    plan_execute_impl(plan, q, k, v, o, lse, (hipStream_t)stream);
    if (plan->ctx->debug) {   // a failed launch is reported by the call that made it
      HIPCHK(hipStreamSynchronize((hipStream_t)stream));
      HIPCHK(hipGetLastError());
    }
  });
}

int mmi_plan_destroy(mmi_plan* plan) {
  return guarded([&] {
    if (!plan) fail(MMI_ERR_INVALID_ARG, "plan is NULL");
    (void)hipSetDevice(plan->ctx->device);
    HIPCHK(hipStreamSynchronize(plan->stream));
    free_plan_buffers(plan);
    for (auto& e : plan->ev)
      if (e) (void)hipEventDestroy(e);
    --plan->ctx->live_plans;
    delete plan;
  });
}

int mmi_plan_stats(mmi_plan* P, int head, mmi_head_stats* out) {
  return guarded([&] {
    if (!P || !out) fail(MMI_ERR_INVALID_ARG, "plan/out is NULL");
    if (head < 0 || head >= P->Hq) fail(MMI_ERR_INVALID_ARG, "head %d out of range", head);
    HIPCHK(hipSetDevice(P->ctx->device));
    HIPCHK(hipStreamSynchronize(P->stream));
    const HostHead& H = P->hh[head];
    const HeadDev& hd = P->heads[head];
    mmi_head_stats s{};
    s.kind = H.kind;
    s.n_qblocks = hd.nbq;
    s.n_kblocks = hd.nbk;
    s.nnz_blocks = H.nnz;
    const int64_t nb = (P->S + B - 1) / B;
    s.causal_blocks = nb * (nb + 1) / 2;
    s.split_rows = (int32_t)H.nsplit;
    for (int i = 0; i < H.nops; ++i) {
      const EstInfo& e = H.est[i];
      if (e.params) {
        int32_t prm[4];
        HIPCHK(hipMemcpy(prm, e.params, sizeof prm, hipMemcpyDeviceToHost));
        const int slot = H.op_slot[i];
        if (slot < MMI_MAX_MODALITIES) { s.sigma[slot] = prm[0]; s.phase[slot] = prm[1]; }
      }
    }
    int32_t gp[2];
    HIPCHK(hipMemcpy(gp, hd.gp, sizeof gp, hipMemcpyDeviceToHost));
    s.group_stride = gp[0];
    s.loaded_blocks = H.gnnz;
    // selected blocks by (query modality, key modality), from the block index
    auto block_mods = [&](const int32_t* perm, int nblk) {
      std::vector<int32_t> slots((size_t)nblk * B);
      if (perm) HIPCHK(hipMemcpy(slots.data(), perm, slots.size() * 4, hipMemcpyDeviceToHost));
      else for (size_t x = 0; x < slots.size(); ++x) slots[x] = x < (size_t)P->S ? (int32_t)x : -1;
      std::vector<int> m(nblk, -1);
      for (int j = 0; j < nblk; ++j)
        for (int x = 0; x < B && m[j] < 0; ++x)
          if (slots[(size_t)j * B + x] >= 0) m[j] = P->mod[slots[(size_t)j * B + x]];
      return m;
    };
    const std::vector<int> qm = block_mods(hd.qperm, hd.nbq), km = block_mods(hd.kperm, hd.nbk);
    std::vector<int32_t> rp(hd.nbq + 1), col(std::max<int64_t>(H.nnz, 1));
    HIPCHK(hipMemcpy(rp.data(), hd.rowptr, rp.size() * 4, hipMemcpyDeviceToHost));
    if (H.nnz) HIPCHK(hipMemcpy(col.data(), hd.col, (size_t)H.nnz * 4, hipMemcpyDeviceToHost));
    for (int i = 0; i < hd.nbq; ++i) {
      if (qm[i] < 0) continue;
      for (int e = rp[i]; e < rp[i + 1]; ++e)
        if (km[col[e]] >= 0) ++s.blocks_by_modality[qm[i]][km[col[e]]];
    }
    *out = s;
  });
}

int mmi_plan_pair_counts(mmi_plan* P, int head, int64_t* useful, int64_t* computed) {
  return guarded([&] {
    if (!P || !useful || !computed) fail(MMI_ERR_INVALID_ARG, "plan/useful/computed is NULL");
    if (head < 0 || head >= P->Hq) fail(MMI_ERR_INVALID_ARG, "head %d out of range", head);
    HIPCHK(hipSetDevice(P->ctx->device));
    HIPCHK(hipStreamSynchronize(P->stream));
    int32_t gp[2];
    HIPCHK(hipMemcpy(gp, P->heads[head].gp, sizeof gp, hipMemcpyDeviceToHost));
    void* d = P->ctx->alloc.get(sizeof(unsigned long long));
    unsigned long long n = 0;
    hipError_t e = hipMemcpyAsync(d, &n, sizeof n, hipMemcpyHostToDevice, P->stream);
    if (e == hipSuccess) e = launch_pair_count(P->d_heads, head, P->R, gp[1], static_cast<unsigned long long*>(d), P->stream);
    if (e == hipSuccess) e = hipMemcpyAsync(&n, d, sizeof n, hipMemcpyDeviceToHost, P->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(P->stream);
    P->ctx->alloc.put(d, sizeof(unsigned long long));
    HIPCHK(e);
    *useful = (int64_t)n;
    *computed = P->hh[head].nnz * (int64_t)(B * B);
  });
}

int mmi_plan_timing_get(mmi_plan* P, mmi_plan_timing* out) {
  return guarded([&] {
    if (!P || !out) fail(MMI_ERR_INVALID_ARG, "plan/out is NULL");
    HIPCHK(hipSetDevice(P->ctx->device));
    HIPCHK(hipStreamSynchronize(P->stream));
    mmi_plan_timing t{};
    HIPCHK(hipEventElapsedTime(&t.est_ms, P->ev[0], P->ev[1]));
    HIPCHK(hipEventElapsedTime(&t.select_ms, P->ev[1], P->ev[2]));
    HIPCHK(hipEventElapsedTime(&t.index_ms, P->ev[2], P->ev[3]));
    if (P->executed) {
      HIPCHK(hipEventElapsedTime(&t.attn_ms, P->ev[4], P->ev[5]));
      HIPCHK(hipEventElapsedTime(&t.combine_ms, P->ev[5], P->ev[6]));
    }
    t.computed_blocks = P->nnz_all;
    t.work_items = P->nitems;
    t.loaded_blocks = P->gnnz_all;
    t.device_bytes = P->device_bytes;
    *out = t;
  });
}

int mmi_plan_export(mmi_plan* P, int head, int what, int slot, void* dst, size_t bytes, size_t* needed) {
  return guarded([&] {
    if (!P) fail(MMI_ERR_STATE, "plan is NULL");
    if (head < 0 || head >= P->Hq) fail(MMI_ERR_INVALID_ARG, "head %d out of range", head);
    HIPCHK(hipSetDevice(P->ctx->device));
    HIPCHK(hipStreamSynchronize(P->stream));
    const HostHead& H = P->hh[head];
    const HeadDev& hd = P->heads[head];
    const void* src = nullptr;
    size_t n = 0;
    std::vector<int32_t> tmp;
    const EstInfo* e = nullptr;
    if (what >= MMI_EXPORT_V_SCORES) {
      for (int i = 0; i < H.nops; ++i)
        if (H.op_slot[i] == slot) e = &H.est[i];
      if (!e) fail(MMI_ERR_INVALID_ARG, "head %d has no op in slot %d", head, slot);
    }
    switch (what) {
      case MMI_EXPORT_QPERM:
      case MMI_EXPORT_KPERM: {
        const int32_t* pm = what == MMI_EXPORT_QPERM ? hd.qperm : hd.kperm;
        const int nslots = (what == MMI_EXPORT_QPERM ? hd.nbq : hd.nbk) * B;
        n = (size_t)nslots * 4;
        if (pm) {
          src = pm;
        } else {
          tmp.resize(nslots);
          for (int x = 0; x < nslots; ++x) tmp[x] = x < P->S ? x : -1;
        }
        break;
      }
      case MMI_EXPORT_ROW_PTR: src = hd.rowptr; n = (size_t)(hd.nbq + 1) * 4; break;
      case MMI_EXPORT_COL_IDX: src = hd.col; n = (size_t)H.nnz * 4; break;
      case MMI_EXPORT_V_SCORES: src = e->v; n = e->v ? (size_t)e->L_c * 4 : 0; break;
      case MMI_EXPORT_U_SCORES: src = e->u; n = e->u ? (size_t)e->L_c * 4 : 0; break;
      case MMI_EXPORT_FOLD: src = e->fold; n = e->fold ? (size_t)std::max(0, e->hi - e->lo + 1) * FOLD_W * 4 : 0; break;
      case MMI_EXPORT_VSEL: src = e->vsel; n = (size_t)e->nv * 4; break;
      case MMI_EXPORT_SSEL: src = e->ssel; n = (size_t)e->ns * 4; break;
      case MMI_EXPORT_PARAMS: {
        tmp.assign(4, 0);
        if (e->params) HIPCHK(hipMemcpy(tmp.data(), e->params, 16, hipMemcpyDeviceToHost));
        else { tmp[2] = e->L_c; tmp[3] = e->nrows; }
        n = 16;
        break;
      }
      case MMI_EXPORT_EST_LSE: {
        if (e->rowset < 0) { n = 0; break; }
        n = (size_t)e->nrows * 4;
        std::vector<float> l2(e->nrows);
        HIPCHK(hipMemcpy(l2.data(), P->est_lse2[e->rowset], n, hipMemcpyDeviceToHost));
        tmp.resize(e->nrows);
        for (int r = 0; r < e->nrows; ++r) {
          const float x = l2[r] * LN2;
          std::memcpy(&tmp[r], &x, 4);
        }
        break;
      }
      case MMI_EXPORT_UNION_PTR:
      case MMI_EXPORT_UNION: {
        int32_t gp[2];
        HIPCHK(hipMemcpy(gp, hd.gp, sizeof gp, hipMemcpyDeviceToHost));
        if (what == MMI_EXPORT_UNION_PTR) { src = hd.growptr; n = (size_t)(gp[1] + 1) * 4; }
        else { src = hd.gcol; n = (size_t)H.gnnz * 4; }
        break;
      }
      default: fail(MMI_ERR_INVALID_ARG, "unknown export kind %d", what);
    }
    if (needed) *needed = n;
    if (!dst) return;
    if (bytes < n) fail(MMI_ERR_INVALID_ARG, "destination holds %zu bytes, %zu needed", bytes, n);
    if (n == 0) return;
    if (!tmp.empty()) std::memcpy(dst, tmp.data(), n);
    else HIPCHK(hipMemcpy(dst, src, n, hipMemcpyDeviceToHost));
  });
}

int mmi_attention(mmi_ctx* ctx, const mmi_problem* prob, const mmi_head_cfg* cfgs, const void* q, const void* k,
                  const void* v, void* o, float* lse, void* stream) {
  mmi_plan* P = nullptr;
  int rc = mmi_plan_create(ctx, prob, cfgs, q, k, stream, &P);
  if (rc != MMI_OK) return rc;
  rc = mmi_plan_execute(P, q, k, v, o, lse, stream);
  const int rc2 = mmi_plan_destroy(P);
  return rc != MMI_OK ? rc : rc2;
}

int mmi_attention_noalloc(mmi_ctx* ctx, const mmi_problem* prob, const mmi_head_cfg* cfgs, const void* q,
                          const void* k, const void* v, void* o, float* lse, void* stream) {
  if (!ctx) {
    g_last_error = "ctx is NULL";
    return MMI_ERR_INVALID_ARG;
  }
  if (ctx->device >= MAX_DEVICES || !g_scratch_ptr[ctx->device]) {
    g_last_error = "no-allocation scratch is not set up on this device";
    return MMI_ERR_UNSUPPORTED;
  }
  // one call at a time per device: the scratch holds one plan
  std::lock_guard<std::mutex> lk(g_scratch_call_mu[ctx->device]);
  mmi_plan* P = nullptr;
  int rc = create_plan(ctx, prob, cfgs, q, k, stream, g_scratch_ptr[ctx->device], &P);
  if (rc != MMI_OK) return rc;
  rc = mmi_plan_execute(P, q, k, v, o, lse, stream);
  const int rc2 = mmi_plan_destroy(P);      // waits for the stream: the scratch is free again
  return rc != MMI_OK ? rc : rc2;
}

int mmi_dense_attention(mmi_ctx* ctx, const mmi_problem* prob, const void* q, const void* k, const void* v,
                        void* o, float* lse, void* stream) {
  if (!prob) {
    g_last_error = "problem is NULL";
    return MMI_ERR_INVALID_ARG;
  }
  if (prob->Hq < 1 || prob->Hq > (1 << 16)) {
    g_last_error = "Hq out of range";
    return MMI_ERR_INVALID_ARG;
  }
  std::vector<mmi_head_cfg> cfgs(prob->Hq);
  for (auto& c : cfgs) {
    std::memset(&c, 0, sizeof c);
    c.kind = MMI_HEAD_GLOBAL;
    c.global.kind = MMI_OP_DENSE;
  }
  return mmi_attention(ctx, prob, cfgs.data(), q, k, v, o, lse, stream);
}

int mmi_permute_rows(const void* src, int64_t src_stride, void* dst, int64_t dst_stride, const int32_t* perm,
                     int64_t n_dst, int64_t row_bytes, void* stream) {
  return guarded([&] {
    if (!src || !dst || !perm) fail(MMI_ERR_INVALID_ARG, "NULL pointer");
    if (n_dst < 0 || row_bytes <= 0 || row_bytes % 16 || src_stride % 16 || dst_stride % 16)
      fail(MMI_ERR_INVALID_ARG, "rows and strides must be positive multiples of 16 bytes");
    aligned16(src, "src"); aligned16(dst, "dst");
    HIPCHK(launch_permute(src, src_stride, dst, dst_stride, perm, n_dst, row_bytes, 0, (hipStream_t)stream));
  });
}

int mmi_unpermute_rows(const void* src, int64_t src_stride, void* dst, int64_t dst_stride, const int32_t* perm,
                       int64_t n_src, int64_t row_bytes, void* stream) {
  return guarded([&] {
    if (!src || !dst || !perm) fail(MMI_ERR_INVALID_ARG, "NULL pointer");
    if (n_src < 0 || row_bytes <= 0 || row_bytes % 16 || src_stride % 16 || dst_stride % 16)
      fail(MMI_ERR_INVALID_ARG, "rows and strides must be positive multiples of 16 bytes");
    aligned16(src, "src"); aligned16(dst, "dst");
    HIPCHK(launch_permute(src, src_stride, dst, dst_stride, perm, n_src, row_bytes, 1, (hipStream_t)stream));
  });
}

int mmi_check_index(const mmi_index_view* v) {
  return guarded([&] {
    if (!v) fail(MMI_ERR_INVALID_ARG, "view is NULL");
    const std::string e = check_index(*v);
    if (!e.empty()) fail(MMI_ERR_INTERNAL, "%s", e.c_str());
  });
}

int mmi_check_work(const mmi_work_view* w) {
  return guarded([&] {
    if (!w) fail(MMI_ERR_INVALID_ARG, "view is NULL");
    const std::string e = check_work(*w);
    if (!e.empty()) fail(MMI_ERR_INTERNAL, "%s", e.c_str());
  });
}

int mmi_plan_check(mmi_plan* plan) {
  return guarded([&] {
    if (!plan) fail(MMI_ERR_STATE, "plan is NULL");
    plan_check(plan);
  });
}

int mmi_output_sqerr(const mmi_problem* prob, const void* a, const void* b, const uint8_t* cls, int32_t n_class,
                     double* out, void* stream) {
  return guarded([&] {
    if (!prob) fail(MMI_ERR_INVALID_ARG, "problem is NULL");
    mmi_problem p = *prob;
    p.modality = nullptr;          // not read here
    p = normalise(&p);
    if (!a || !b || !cls || !out) fail(MMI_ERR_INVALID_ARG, "NULL pointer");
    if (n_class < 1 || n_class > MMI_MAX_MODALITIES)
      fail(MMI_ERR_INVALID_ARG, "n_class must be in [1, %d]", MMI_MAX_MODALITIES);
    aligned16(a, "a"); aligned16(b, "b");
    HIPCHK(launch_sqerr(a, b, p.o_stride_s, p.o_stride_h, cls, n_class, (int)p.S, p.Hq, out, (hipStream_t)stream));
  });
}

int mmi_search(mmi_ctx* ctx, const mmi_problem* prob, const void* q, const void* k, const void* v,
               const mmi_op* cands, int32_t n_cands, const mmi_op* xc, int32_t n_xc, const mmi_op* target,
               void* stream, mmi_head_cfg* out, mmi_search_report* report) {
  return guarded([&] {
    if (!ctx || !q || !k || !v || !target || !out) fail(MMI_ERR_INVALID_ARG, "NULL pointer");
    if (n_cands < 0 || n_xc < 0 || (n_cands > 0 && !cands) || (n_xc > 0 && !xc))
      fail(MMI_ERR_INVALID_ARG, "candidate lists: negative count or NULL array");
    const mmi_problem p = normalise(prob);
    HIPCHK(hipSetDevice(ctx->device));
    search_layer(ctx, p, q, k, v, cands, n_cands, xc, n_xc, *target, (hipStream_t)stream, out, report);
  });
}

}  // extern "C"
