// Host side of the C ABI declared in include/rc.h: argument validation,
// device memory plumbing and kernel orchestration.  Every step of the
// method itself runs in the kernels of graph.hip, family.hip and fill.hip.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <memory>
#include <mutex>
#include <new>
#include <utility>
#include <vector>

#include "rc_internal.h"
#include "dominance.h"
#include "dual.h"

using namespace rcdp;

#define RC_HIP(x)                                     \
  do {                                                \
    hipError_t e_ = (x);                              \
    if (e_ != hipSuccess) {                           \
      rcdp::set_last_error(#x, e_);                   \
      return RC_E_DEVICE;                             \
    }                                                 \
  } while (0)

namespace rcdp {

static thread_local char g_last_error[512] = "";

void set_last_error(const char* what, hipError_t e) {
  std::snprintf(g_last_error, sizeof(g_last_error), "%s: %s", what, hipGetErrorString(e));
}

void set_last_error_msg(const char* msg) {
  std::snprintf(g_last_error, sizeof(g_last_error), "%s", msg);
}

int32_t jitter_seed() {
  const char* env = std::getenv("RCDP_JITTER");
  return env ? (int32_t)std::strtol(env, nullptr, 10) : 0;
}

namespace {
// Free pinned buffers, smallest first: a request takes the smallest that
// fits, or allocates a power of two of at least 64 KB.  Never destroyed, so
// that no buffer is released after the runtime has shut down.
struct StagingPool {
  std::mutex mu;
  std::vector<std::pair<size_t, char*>> free_list;
};
StagingPool& staging_pool() {
  static StagingPool* pool = new StagingPool();
  return *pool;
}
}  // namespace

Staging::Staging(size_t bytes) {
  StagingPool& pool = staging_pool();
  {
    std::lock_guard<std::mutex> lock(pool.mu);
    auto& fl = pool.free_list;
    for (size_t x = 0; x < fl.size(); x++) {
      if (fl[x].first >= bytes) {
        n_ = fl[x].first;
        p_ = fl[x].second;
        fl.erase(fl.begin() + (std::ptrdiff_t)x);
        return;
      }
    }
  }
  size_t n = (size_t)64 << 10;
  while (n < bytes) n <<= 1;
  void* p = nullptr;
  if (hipHostMalloc(&p, n, hipHostMallocDefault) != hipSuccess) return;
  p_ = static_cast<char*>(p);
  n_ = n;
}

Staging::~Staging() {
  if (!p_ || pending_) return;
  StagingPool& pool = staging_pool();
  std::lock_guard<std::mutex> lock(pool.mu);
  auto& fl = pool.free_list;
  auto it = fl.begin();
  while (it != fl.end() && it->first < n_) ++it;
  fl.insert(it, {n_, p_});
}

// Sizes of the memory-indexed table of one solve (rc_solve_dual): argument
// checks, the effective budget, the row width and the scratch it needs.
int dual_buffers(rc_family f, int64_t B, int32_t objective, DualBuffers* out) {
  if (!f || B < 0) return RC_E_ARG;
  if (objective != RC_TIME_CENTRIC && objective != RC_MEMORY_CENTRIC) return RC_E_ARG;
  const int64_t Beff = std::min<int64_t>(B, 2 * f->g->M_total);
  const int64_t W = std::min<int64_t>(Beff, f->g->M_total) + 1;
  if (f->g->T_total >= (int64_t)UINT32_MAX || W > INT32_MAX / 2 ||
      (double)f->F * (double)W > (double)((int64_t)1 << 31))
    return RC_E_OVERFLOW;
  *out = DualBuffers();
  out->Beff = Beff;
  out->W = W;
  out->cells = f->F * W;
  return RC_OK;
}

// The memory-indexed table, its selection and (when any schedule output is
// asked for) its traceback, in the device buffers of b; results to the host
// outputs.  Synchronises s.  e0 / e1 (may be null) bracket the table's
// kernels.  Allocates nothing.
int dual_solve(rc_family f, int32_t objective, const DualBuffers& b, hipEvent_t e0,
               hipEvent_t e1, hipStream_t s, int64_t* t_opt, int64_t* m_opt, int32_t* k,
               int32_t* chain_host, int32_t* seg_host, uint8_t* cached_host, int64_t* overhead,
               int64_t* peak, int64_t* cache_mem) {
  const hipError_t le = launch_dual(f, f->level_pairs, (int32_t)b.Beff, (int32_t)b.W, objective,
                                    b.D, b.st, e0, e1, s);
  if (le != hipSuccess) {
    set_last_error("dual table launch", le);
    return RC_E_DEVICE;
  }
  DevStatus hs;
  RC_HIP(hipMemcpyAsync(&hs, b.st, sizeof(hs), hipMemcpyDeviceToHost, s));
  RC_HIP(hipStreamSynchronize(s));
  const bool schedule = k || chain_host || seg_host || cached_host || overhead || peak || cache_mem;
  if (schedule && hs.t_sel >= 0) {
    const int n = f->g->n;
    const hipError_t te = launch_dual_trace(f, (int32_t)b.Beff, (int32_t)b.W, objective, b.D,
                                            b.st, b.chain, b.seg, b.cached, s);
    if (te != hipSuccess) {
      set_last_error("dual traceback launch", te);
      return RC_E_DEVICE;
    }
    DevStatus ts;
    RC_HIP(hipMemcpyAsync(&ts, b.st, sizeof(ts), hipMemcpyDeviceToHost, s));
    RC_HIP(hipStreamSynchronize(s));
    if (ts.error || ts.k < 0 || ts.k > f->F) {
      set_last_error_msg("dual traceback: the walk did not end at (empty set, 0, 0)");
      return RC_E_DEVICE;
    }
    if (chain_host && ts.k > 0)
      RC_HIP(hipMemcpyAsync(chain_host, b.chain, sizeof(int32_t) * (size_t)ts.k,
                            hipMemcpyDeviceToHost, s));
    if (seg_host && n > 0)
      RC_HIP(hipMemcpyAsync(seg_host, b.seg, sizeof(int32_t) * (size_t)n, hipMemcpyDeviceToHost,
                            s));
    if (cached_host && n > 0)
      RC_HIP(hipMemcpyAsync(cached_host, b.cached, (size_t)n, hipMemcpyDeviceToHost, s));
    RC_HIP(hipStreamSynchronize(s));
    if (k) *k = ts.k;
    if (overhead) *overhead = ts.overhead;
    if (peak) *peak = ts.peak;
    if (cache_mem) *cache_mem = ts.cache_mem;
  }
  if (t_opt) *t_opt = hs.t_sel;
  if (m_opt) *m_opt = hs.t_sel >= 0 ? hs.m_sel : -1;
  return hs.t_sel >= 0 ? RC_OK : RC_INFEASIBLE;
}

void* Arena::raw(size_t bytes) {
  void* p = nullptr;
  if (alloc) {
    p = alloc(bytes, user);
  } else if (hipMalloc(&p, bytes) != hipSuccess) {
    p = nullptr;
  }
  if (p) ptrs.push_back(p);
  return p;
}

// Small buffers are carved from chunks of kChunk bytes, so that a handle
// costs a few calls of the caller's allocator rather than one per buffer.
void* Arena::get(size_t bytes) {
  if (bytes == 0) bytes = 1;
  bytes = (bytes + 255) & ~size_t(255);
  if (bytes > kChunk / 4) return raw(bytes);
  if (cur + bytes > end) {
    char* c = static_cast<char*>(raw(kChunk));
    if (!c) return nullptr;
    cur = c;
    end = c + kChunk;
  }
  void* p = cur;
  cur += bytes;
  return p;
}

void Arena::release_all() {
  cur = end = nullptr;
  for (void* p : ptrs) {
    if (alloc) {
      if (free_fn) free_fn(p, user);
    } else {
      (void)hipFree(p);
    }
  }
  ptrs.clear();
}

}  // namespace rcdp

static hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

template <class T>
static int upload(Arena& a, const T* host, int64_t count, T** dev, hipStream_t s) {
  *dev = a.get_n<T>(count);
  if (!*dev) return RC_E_NOMEM;
  if (count > 0)
    RC_HIP(hipMemcpyAsync(*dev, host, sizeof(T) * (size_t)count, hipMemcpyHostToDevice, s));
  return RC_OK;
}

extern "C" {

const char* rc_last_error(void) { return g_last_error; }

const char* rc_status_str(int status) {
  switch (status) {
    case RC_OK: return "ok";
    case RC_INFEASIBLE: return "infeasible: no chain of lower sets meets the budget";
    case RC_E_ARG: return "invalid argument";
    case RC_E_CYCLE: return "the graph has a directed cycle or a self-loop";
    case RC_E_COST: return "a node cost is not positive";
    case RC_E_TOO_MANY_SETS: return "the lower-set family exceeds max_sets";
    case RC_E_OVERFLOW: return "a value exceeds the table's integer widths";
    case RC_E_NOMEM: return "device allocation failed";
    case RC_E_DEVICE: return "HIP runtime or kernel error";
    case RC_E_STATE: return "handle in the wrong state";
    case RC_E_SCRATCH: return "the solve needs more than the allocation-free scratch";
    default: return "unknown status";
  }
}

// ------------------------------------------------------------------ graph

int rc_graph_create(int32_t n, const int32_t* row_ptr, const int32_t* col_idx, const int32_t* T,
                    const int32_t* M, rc_alloc_fn alloc, rc_free_fn free_fn, void* user,
                    void* stream, rc_graph* out) {
  if (!out || n < 0 || n > kMaxNodes) return RC_E_ARG;
  if (n > 0 && (!row_ptr || !T || !M)) return RC_E_ARG;
  if (alloc && !free_fn) return RC_E_ARG;
  // -- validation of the CSR and costs (Section 2: T_v > 0, M_v > 0)
  int64_t nnz = 0;
  if (n > 0) {
    if (row_ptr[0] != 0) return RC_E_ARG;
    for (int v = 0; v < n; v++)
      if (row_ptr[v + 1] < row_ptr[v]) return RC_E_ARG;
    nnz = row_ptr[n];
    if (nnz > 0 && !col_idx) return RC_E_ARG;
    for (int64_t e = 0; e < nnz; e++)
      if (col_idx[e] < 0 || col_idx[e] >= n) return RC_E_ARG;
  }
  int64_t Ttot = 0, Mtot = 0;
  for (int v = 0; v < n; v++) {
    if (T[v] < 1 || M[v] < 1) return RC_E_COST;
    Ttot += T[v];
    Mtot += M[v];
  }
  if (Ttot >= (int64_t)INT32_MAX - 1 || Mtot >= ((int64_t)1 << 29)) return RC_E_OVERFLOW;
  // -- deduplicated predecessor lists and topological depth (Kahn by levels)
  std::vector<std::vector<int32_t>> preds(n);
  for (int v = 0; v < n; v++) {
    for (int64_t e = row_ptr[v]; e < row_ptr[v + 1]; e++) {
      int w = col_idx[e];
      if (w == v) return RC_E_CYCLE;
      preds[w].push_back(v);
    }
  }
  for (auto& p : preds) {
    std::sort(p.begin(), p.end());
    p.erase(std::unique(p.begin(), p.end()), p.end());
  }
  std::vector<int32_t> indeg(n), depth(n, 0), order;
  order.reserve(n);
  std::vector<std::vector<int32_t>> succs(n);
  for (int w = 0; w < n; w++)
    for (int v : preds[w]) succs[v].push_back(w);
  for (int v = 0; v < n; v++) {
    indeg[v] = (int32_t)preds[v].size();
    if (indeg[v] == 0) order.push_back(v);
  }
  for (size_t q = 0; q < order.size(); q++) {
    int v = order[q];
    for (int w : succs[v]) {
      depth[w] = std::max(depth[w], depth[v] + 1);
      if (--indeg[w] == 0) order.push_back(w);
    }
  }
  if ((int)order.size() != n) return RC_E_CYCLE;
  int32_t D = 0;
  for (int v = 0; v < n; v++) D = std::max(D, depth[v] + 1);
  std::vector<int32_t> by_depth(n), depth_ptr(D + 1, 0);
  for (int v = 0; v < n; v++) depth_ptr[depth[v] + 1]++;
  for (int d = 0; d < D; d++) depth_ptr[d + 1] += depth_ptr[d];
  {
    std::vector<int32_t> fill(depth_ptr.begin(), depth_ptr.end() - 1);
    for (int v = 0; v < n; v++) by_depth[fill[depth[v]]++] = v;
  }
  std::vector<int32_t> pred_ptr(n + 1, 0), pred_idx;
  for (int v = 0; v < n; v++) {
    pred_ptr[v + 1] = pred_ptr[v] + (int32_t)preds[v].size();
    pred_idx.insert(pred_idx.end(), preds[v].begin(), preds[v].end());
  }

  rc_graph g = new (std::nothrow) rc_graph_s();
  if (!g) return RC_E_NOMEM;
  g->n = n;
  g->words = (n + 63) / 64;
  g->T_total = Ttot;
  g->M_total = Mtot;
  g->arena.alloc = alloc;
  g->arena.free_fn = free_fn;
  g->arena.user = user;
  g->num_depths = D;
  for (int v = 0; v < n; v++) g->num_sinks += succs[v].empty() ? 1 : 0;
  hipStream_t s = as_stream(stream);
  int st = RC_OK;
  int32_t *d_row_ptr = nullptr, *d_col_idx = nullptr;
  std::vector<int32_t> rp(row_ptr ? row_ptr : nullptr, row_ptr ? row_ptr + n + 1 : nullptr);
  std::vector<int32_t> ci(col_idx ? col_idx : nullptr, col_idx ? col_idx + nnz : nullptr);
  if (st == RC_OK) st = upload(g->arena, T, n, &g->dT, s);
  if (st == RC_OK) st = upload(g->arena, M, n, &g->dM, s);
  if (st == RC_OK) st = upload(g->arena, pred_ptr.data(), n + 1, &g->dPredPtr, s);
  g->num_pred_edges = (int32_t)pred_idx.size();
  if (st == RC_OK) st = upload(g->arena, pred_idx.data(), (int64_t)pred_idx.size(), &g->dPredIdx, s);
  if (st == RC_OK) st = upload(g->arena, by_depth.data(), n, &g->dByDepth, s);
  if (st == RC_OK) st = upload(g->arena, depth_ptr.data(), D + 1, &g->dDepthPtr, s);
  if (st == RC_OK) st = upload(g->arena, rp.data(), (int64_t)rp.size(), &d_row_ptr, s);
  if (st == RC_OK) st = upload(g->arena, ci.data(), (int64_t)ci.size(), &d_col_idx, s);
  if (st == RC_OK) {
    g->dSucc = g->arena.get_n<uint64_t>((int64_t)n * g->words);
    g->dPred = g->arena.get_n<uint64_t>((int64_t)n * g->words);
    g->dAnc = g->arena.get_n<uint64_t>((int64_t)n * g->words);
    if (!g->dSucc || !g->dPred || !g->dAnc) st = RC_E_NOMEM;
  }
  if (st == RC_OK && n > 0 && launch_graph_masks(g, d_row_ptr, d_col_idx, s) != hipSuccess)
    st = RC_E_DEVICE;
  // the ancestor sets (Section 4.3's generators of the pruned family) are a
  // property of the graph: computed once here, read by every pruned family
  if (st == RC_OK && n > 0 && launch_ancestors(g, g->dAnc, s) != hipSuccess) st = RC_E_DEVICE;
  // the host vectors above must stay alive until the copies have completed
  if (st == RC_OK && hipStreamSynchronize(s) != hipSuccess) st = RC_E_DEVICE;
  if (st != RC_OK) {
    (void)hipStreamSynchronize(s);
    g->arena.release_all();
    delete g;
    return st;
  }
  *out = g;
  return RC_OK;
}

void rc_graph_free(rc_graph g) {
  if (!g) return;
  (void)hipDeviceSynchronize();
  g->arena.release_all();
  delete g;
}

// ----------------------------------------------------------------- family

// Which blocks the family's wavefront records use.  RCDP_FILL=wavefront
// forces the row-push fill's fixed blocks and RCDP_FILL=ghost the ghost-zone
// blocks (families of at most kGhostMaxSets sets).  Otherwise: fixed blocks
// for families beyond that size, for families of kWideMinSets sets and more
// and for tables with rows of 2^16 cells and more (where the split-panel
// fill measured fastest), ghost-zone blocks for the rest.
// shape_known: max_row and the levels are set (after the host copies).
static int32_t family_block_kind(rc_family f, bool shape_known) {
  const int64_t F = f->F;
  if (F < 2) return 0;
  const char* env = std::getenv("RCDP_FILL");
  if (F > kGhostMaxSets ||
      (env && (std::strcmp(env, "wavefront") == 0 || std::strcmp(env, "wide") == 0)))
    return kBlocksFixed;
  if (env && std::strcmp(env, "ghost") == 0) return kBlocksGhost;
  if (!shape_known) return -1;                 // decided once the table's shape is known
  // fixed blocks, so that the split-panel fill can take the family, for
  // rows of 2^16 cells and more and for families of kWideMinSets sets and
  // more (measured faster than the ghost-zone fill on every such shape
  // here, resnet50_t10's 175 sets included: the ghost blocks hold fewer
  // rows, so that each staged window serves fewer targets); ghost-zone
  // blocks for the smaller families
  return f->max_row >= 65536 || F >= kWideMinSets ? kBlocksFixed : kBlocksGhost;
}

// Block starts of the chosen kind (host).
static void cut_blocks(rc_family f, const std::vector<int32_t>& near_h) {
  f->bstart_host.clear();
  if (f->blk_kind == kBlocksGhost) {
    f->bstart_host = ghost_cut(f->F, near_h);
    return;
  }
  for (int64_t j = 1; j < f->F; j += kJB) f->bstart_host.push_back((int32_t)j);
  f->bstart_host.push_back((int32_t)f->F);
}

// Block starts to the device (through pinned memory), then the number of
// panel sources per block and their offsets (rec_ptr).  Uses the family
// arena; counts is scratch of at least nblk + 1 entries.  The staging
// buffer must stay alive until the stream has been synchronised.
static int upload_blocks(rc_family f, int64_t* counts, std::unique_ptr<Staging>& stage,
                         hipStream_t s) {
  Arena& A = f->arena;
  f->nblk = (int64_t)f->bstart_host.size() - 1;
  if (f->nblk <= 0) {
    f->nblk = 0;
    return RC_OK;
  }
  f->bstart = A.get_n<int32_t>(f->nblk + 1);
  f->rec_ptr = A.get_n<int64_t>(f->nblk + 1);
  if (!f->bstart || !f->rec_ptr) return RC_E_NOMEM;
  const size_t bytes = sizeof(int32_t) * (size_t)(f->nblk + 1);
  stage.reset(new (std::nothrow) Staging(bytes));
  if (!stage || !stage->data()) return RC_E_NOMEM;
  std::memcpy(stage->data(), f->bstart_host.data(), bytes);
  stage->in_flight();
  if (hipMemcpyAsync(f->bstart, stage->data(), bytes, hipMemcpyHostToDevice, s) != hipSuccess ||
      launch_blk_count(f, f->nblk, counts, s) != hipSuccess ||
      launch_scan(counts, f->rec_ptr, f->nblk, 1, s) != hipSuccess)
    return RC_E_DEVICE;
  return RC_OK;
}

// Sets of the pruned family: the n ancestor sets L^v (distinct, since v is
// the one maximal node of L^v), the empty set, and V unless V is one of the
// L^v, which happens exactly when the graph has a single sink (every node
// then reaches it).
static int64_t pruned_family_size(rc_graph g) {
  if (g->n == 0) return 1;
  return (int64_t)g->n + 1 + (g->num_sinks > 1 ? 1 : 0);
}

// Gathers L into the device buffer dev (at least bytes) and enqueues one
// copy of it into the staging buffer.
static int pack_to_host(const PackList& L, void* dev, size_t bytes, Staging& st, hipStream_t s) {
  if (launch_pack(L, dev, s) != hipSuccess) return RC_E_DEVICE;
  st.in_flight();
  if (hipMemcpyAsync(st.data(), dev, bytes, hipMemcpyDeviceToHost, s) != hipSuccess)
    return RC_E_DEVICE;
  return RC_OK;
}

// Record buffers up to this many records are sized from an upper bound
// (every record holds at least one pair) without waiting for their count.
constexpr int64_t kRecordBound = (int64_t)1 << 18;

static int build_family_impl(rc_family f, int64_t max_sets, hipStream_t s) {
  rc_graph g = f->g;
  const int n = g->n, words = g->words;
  Arena& A = f->arena;
  Arena tmp;                       // scratch released at the end of the build
  tmp.alloc = A.alloc;
  tmp.free_fn = A.free_fn;
  tmp.user = A.user;
  std::unique_ptr<Staging> up_stage;  // host -> device block starts
  struct TmpGuard {
    Arena& a;
    hipStream_t s;
    ~TmpGuard() {
      (void)hipStreamSynchronize(s);
      a.release_all();
    }
  } guard{tmp, s};
  // Host -> device and device -> host copies go through pinned buffers; a
  // build waits for the stream once for the family's size (exact family
  // only), once for its shape and pair count, once more for the near shifts
  // of a ghost-zone family, and once at the end.
  auto sync_landed = [&](Staging& st) -> int {
    if (hipStreamSynchronize(s) != hipSuccess) {
      set_last_error_msg("family build: stream synchronisation failed");
      return RC_E_DEVICE;
    }
    st.landed();
    return RC_OK;
  };

  f->status = A.get_n<DevStatus>(1);
  if (!f->status) return RC_E_NOMEM;
  RC_HIP(launch_zero(f->status, sizeof(DevStatus), s));

  // ---- a2: the family as bitmasks, in canonical order
  const bool pruned = f->mode == RC_FAMILY_PRUNED;
  const int64_t cap = pruned ? (int64_t)n + 2 : max_sets;
  f->fstride = cap;
  uint64_t* cand = tmp.get_n<uint64_t>(cap * words);
  int32_t* lvl = tmp.get_n<int32_t>(n + 3);
  f->bits = A.get_n<uint64_t>(cap * words);
  if (!cand || !lvl || !f->bits) return RC_E_NOMEM;
  if (pruned) {
    RC_HIP(launch_pruned_candidates(g, g->dAnc, cand, s));
  } else {
    RC_HIP(launch_enum_exact(g, cand, cap, lvl, f->status, s));
  }
  RC_HIP(launch_rank(g, f->mode, cand, cap, lvl, f->bits, f->fstride, f->status, s));
  int64_t F = 0;
  if (pruned) {
    F = pruned_family_size(g);          // checked against the device's count below
  } else {
    Staging st0(sizeof(DevStatus));
    if (!st0.data()) return RC_E_NOMEM;
    st0.in_flight();
    RC_HIP(hipMemcpyAsync(st0.data(), f->status, sizeof(DevStatus), hipMemcpyDeviceToHost, s));
    const int ss = sync_landed(st0);
    if (ss != RC_OK) return ss;
    const DevStatus& h0 = *st0.at<DevStatus>(0);
    if (h0.overflow) return RC_E_TOO_MANY_SETS;
    if (h0.error) return RC_E_DEVICE;
    F = h0.count;
  }
  if (F < 1 || F > max_sets) return RC_E_TOO_MANY_SETS;
  f->F = F;

  // ---- a3: per-set quantities
  f->size = A.get_n<int32_t>(F);
  f->Tsum = A.get_n<int32_t>(F);
  f->Msum = A.get_n<int32_t>(F);
  f->Tbd = A.get_n<int32_t>(F);
  f->Mbd = A.get_n<int32_t>(F);
  f->A = A.get_n<int32_t>(F);
  f->w = A.get_n<int32_t>(F);
  f->bd = A.get_n<uint64_t>(f->fstride * words);
  f->row_off = A.get_n<int64_t>(F + 1);
  f->pred_ptr = A.get_n<int64_t>(F + 1);
  int64_t* counts = tmp.get_n<int64_t>(F + 1);
  int64_t* padded = tmp.get_n<int64_t>(F + 1);
  int64_t* walg_t = tmp.get_n<int64_t>(F + 1);
  if (!f->size || !f->Tsum || !f->Msum || !f->Tbd || !f->Mbd || !f->A || !f->w || !f->bd ||
      !f->row_off || !f->pred_ptr || !counts || !padded || !walg_t)
    return RC_E_NOMEM;
  RC_HIP(launch_set_quantities(f, s));
  // row offsets: rows padded to kRowAlign cells
  RC_HIP(launch_row_widths(f, padded, s));
  RC_HIP(launch_scan(padded, f->row_off, F, 1, s));
  RC_HIP(launch_row_align(f, s));
  // ---- a4: predecessor pairs, counted per target
  RC_HIP(launch_pair_count(f, counts, s));
  RC_HIP(launch_scan(counts, f->pred_ptr, F, 1, s));

  // ---- the family's shape to the host: sizes, widths, row offsets, pairs
  StageLayout L1;
  const size_t o_st = L1.add<DevStatus>(1), o_size = L1.add<int32_t>(F),
               o_w = L1.add<int32_t>(F), o_off = L1.add<int64_t>(F + 1),
               o_pp = L1.add<int64_t>(F + 1);
  {
    Staging st1(L1.bytes);
    void* pk1 = tmp.get(L1.bytes);
    if (!st1.data() || !pk1) return RC_E_NOMEM;
    PackList P1;
    P1.add(f->status, sizeof(DevStatus), (int64_t)o_st);
    P1.add(f->size, sizeof(int32_t) * F, (int64_t)o_size);
    P1.add(f->w, sizeof(int32_t) * F, (int64_t)o_w);
    P1.add(f->row_off, sizeof(int64_t) * (F + 1), (int64_t)o_off);
    P1.add(f->pred_ptr, sizeof(int64_t) * (F + 1), (int64_t)o_pp);
    const int pc1 = pack_to_host(P1, pk1, L1.bytes, st1, s);
    if (pc1 != RC_OK) return pc1;
    const int ss = sync_landed(st1);
    if (ss != RC_OK) return ss;
    const DevStatus& h1 = *st1.at<DevStatus>(o_st);
    if (h1.overflow) return RC_E_TOO_MANY_SETS;
    if (h1.error) return RC_E_DEVICE;
    if (h1.count != F) {
      set_last_error_msg("family build: the device counted another family size");
      return RC_E_DEVICE;
    }
    const int32_t* size_h = st1.at<int32_t>(o_size);
    const int32_t* w_h = st1.at<int32_t>(o_w);
    const int64_t* off_h = st1.at<int64_t>(o_off);
    const int64_t* pp_h = st1.at<int64_t>(o_pp);
    f->w_host.assign(w_h, w_h + F);
    f->row_off_host.assign(off_h, off_h + F + 1);
    f->cells = off_h[F];
    f->cells_alloc = f->cells + kGuard;
    f->P = pp_h[F];
    if (f->P < 0 || f->P >= ((int64_t)1 << 40) || f->cells >= ((int64_t)1 << 40))
      return RC_E_OVERFLOW;
    f->level_ptr.clear();
    f->level_maxw.clear();
    f->max_row = 0;
    for (int64_t i = 0; i < F; i++) {
      if (i == 0 || size_h[i] != size_h[i - 1]) {
        f->level_ptr.push_back(i);
        f->level_maxw.push_back(0);
      }
      f->level_maxw.back() = std::max(f->level_maxw.back(), w_h[i]);
      f->max_row = std::max<int64_t>(f->max_row, w_h[i]);
    }
    f->level_ptr.push_back(F);
    // the most pairs of a target per size level (the memory-indexed table
    // runs that many pairs per level launch)
    f->level_pairs.clear();
    for (size_t l = 0; l + 1 < f->level_ptr.size(); l++) {
      int64_t most = 0;
      for (int64_t j = f->level_ptr[l]; j < f->level_ptr[l + 1]; j++)
        most = std::max(most, pp_h[j + 1] - pp_h[j]);
      f->level_pairs.push_back(most);
    }
  }

  // ---- a4: the pairs themselves and the relaxation count
  const int64_t P = f->P;
  f->pidx = A.get_n<int32_t>(P);
  f->pdt = A.get_n<int32_t>(P);
  f->pdm = A.get_n<int32_t>(P);
  f->pc = A.get_n<int32_t>(P);
  if (!f->pidx || !f->pdt || !f->pdm || !f->pc) return RC_E_NOMEM;
  RC_HIP(launch_pair_write(f, walg_t, s));
  RC_HIP(launch_sum(walg_t, F, &f->status->walg, s));

  // ---- blocks of the wavefront fills: kJB targets each for the row-push
  // fill; for the ghost-zone fill cut on the host from the shifts of near
  // pairs
  f->blk_kind = family_block_kind(f, true);
  if (f->blk_kind == kBlocksGhost) {
    int32_t* near_d = tmp.get_n<int32_t>(F * kNear);
    if (!near_d) return RC_E_NOMEM;
    RC_HIP(launch_near_shifts(f, near_d, s));
    Staging st2(sizeof(int32_t) * (size_t)(F * kNear));
    if (!st2.data()) return RC_E_NOMEM;
    st2.in_flight();
    RC_HIP(hipMemcpyAsync(st2.data(), near_d, sizeof(int32_t) * (size_t)(F * kNear),
                          hipMemcpyDeviceToHost, s));
    const int ss = sync_landed(st2);
    if (ss != RC_OK) return ss;
    const int32_t* nh = st2.at<int32_t>(0);
    cut_blocks(f, std::vector<int32_t>(nh, nh + F * kNear));
  } else if (f->blk_kind == kBlocksFixed) {
    cut_blocks(f, std::vector<int32_t>());
  }
  if (f->blk_kind != 0) {
    const int ub = upload_blocks(f, counts, up_stage, s);
    if (ub != RC_OK) return ub;
  }

  // ---- panel records: buffers sized from the bound P when it is small,
  // else from the count (one more wait)
  f->rec_total = 0;
  int64_t rec_cap = std::min<int64_t>(P, f->nblk * F);
  if (f->nblk > 0 && rec_cap > kRecordBound) {
    Staging st3(sizeof(int64_t));
    if (!st3.data()) return RC_E_NOMEM;
    st3.in_flight();
    RC_HIP(hipMemcpyAsync(st3.data(), f->rec_ptr + f->nblk, sizeof(int64_t),
                          hipMemcpyDeviceToHost, s));
    const int ss = sync_landed(st3);
    if (ss != RC_OK) return ss;
    rec_cap = *st3.at<int64_t>(0);
  }
  const bool records = f->nblk > 0 && rec_cap <= kMaxRecords;
  if (records) {
    BlockRecords& R = f->rec;
    const int64_t Rn = rec_cap, T3 = f->nblk * kJB * kJB;
    R.src = A.get_n<int32_t>(Rn);
    R.e = A.get_n<int32_t>(Rn * kJB);
    R.kadd = A.get_n<uint32_t>(Rn * kJB);
    R.c = A.get_n<int32_t>(Rn * kJB);
    R.tri_e = A.get_n<int32_t>(T3);
    R.tri_kadd = A.get_n<uint32_t>(T3);
    R.tri_c = A.get_n<int32_t>(T3);
    if (!R.src || !R.e || !R.kadd || !R.c || !R.tri_e || !R.tri_kadd || !R.tri_c)
      return RC_E_NOMEM;
    RC_HIP(launch_blk_fill(f, f->nblk, s));
    f->clu_ptr = A.get_n<int64_t>(f->nblk + 1);
    if (!f->clu_ptr) return RC_E_NOMEM;
    RC_HIP(launch_blk_clusters(f, counts, s));
    RC_HIP(launch_scan(counts, f->clu_ptr, f->nblk, 1, s));
  }
  // the split-panel fill: one record per (block, source, shift), a block's
  // records sorted in LDS, byte offsets of the table in 31 bits
  int64_t* wcounts = nullptr;
  if (records && f->blk_kind == kBlocksFixed) {
    f->wrec_ptr = A.get_n<int64_t>(f->nblk + 1);
    wcounts = tmp.get_n<int64_t>(f->nblk + 1);
    if (!f->wrec_ptr || !wcounts) return RC_E_NOMEM;
    RC_HIP(launch_wide_count(f, wcounts, s));
    RC_HIP(launch_scan(wcounts, f->wrec_ptr, f->nblk, 1, s));
  }

  // ---- the counts to the host: status (relaxations, errors), records
  StageLayout L4;
  const size_t q_st = L4.add<DevStatus>(1), q_rec = L4.add<int64_t>(1),
               q_clu = L4.add<int64_t>(1), q_wrec = L4.add<int64_t>(1),
               q_wc = L4.add<int64_t>(wcounts ? f->nblk : 0);
  Staging st4(L4.bytes);
  void* pk4 = tmp.get(L4.bytes);
  if (!st4.data() || !pk4) return RC_E_NOMEM;
  PackList P4;
  P4.add(f->status, sizeof(DevStatus), (int64_t)q_st);
  if (f->nblk > 0) P4.add(f->rec_ptr + f->nblk, sizeof(int64_t), (int64_t)q_rec);
  if (records) P4.add(f->clu_ptr + f->nblk, sizeof(int64_t), (int64_t)q_clu);
  if (wcounts) {
    P4.add(f->wrec_ptr + f->nblk, sizeof(int64_t), (int64_t)q_wrec);
    P4.add(wcounts, sizeof(int64_t) * f->nblk, (int64_t)q_wc);
  }
  const int pc4 = pack_to_host(P4, pk4, L4.bytes, st4, s);
  if (pc4 != RC_OK) return pc4;
  const int ss = sync_landed(st4);
  if (ss != RC_OK) return ss;
  if (up_stage) up_stage->landed();
  const DevStatus& h4 = *st4.at<DevStatus>(q_st);
  if (h4.error) return RC_E_DEVICE;
  f->relax = h4.walg;
  f->rec_total = f->nblk > 0 ? *st4.at<int64_t>(q_rec) : 0;
  if (f->rec_total > rec_cap) {
    set_last_error_msg("family build: more panel records than pairs");
    return RC_E_DEVICE;
  }
  f->has_records = records;
  f->clu_total = records ? *st4.at<int64_t>(q_clu) : 0;
  f->wrec_total = wcounts ? *st4.at<int64_t>(q_wrec) : 0;
  f->has_wide = wcounts && 2 * f->cells_alloc < INT32_MAX && f->wrec_total < ((int64_t)1 << 26);
  for (int64_t b = 0; wcounts && b < f->nblk; b++)
    f->has_wide = f->has_wide && st4.at<int64_t>(q_wc)[b] <= kWMaxRec;
  return RC_OK;
}

int rc_build_family(rc_graph g, int32_t mode, int64_t max_sets, void* stream, rc_family* out) {
  if (!g || !out) return RC_E_ARG;
  if (mode != RC_FAMILY_EXACT && mode != RC_FAMILY_PRUNED) return RC_E_ARG;
  if (max_sets < 1) return RC_E_ARG;
  max_sets = std::min<int64_t>(max_sets, kMaxSets);
  rc_family f = new (std::nothrow) rc_family_s();
  if (!f) return RC_E_NOMEM;
  f->g = g;
  f->mode = mode;
  f->arena.alloc = g->arena.alloc;
  f->arena.free_fn = g->arena.free_fn;
  f->arena.user = g->arena.user;
  int st = build_family_impl(f, max_sets, as_stream(stream));
  if (st != RC_OK) {
    (void)hipStreamSynchronize(as_stream(stream));
    f->arena.release_all();
    delete f;
    return st;
  }
  *out = f;
  return RC_OK;
}

int rc_family_stats(rc_family f, rc_family_info* info) {
  if (!f || !info) return RC_E_ARG;
  info->n = f->g->n;
  info->words = f->g->words;
  info->num_sets = f->F;
  info->num_pairs = f->P;
  info->num_levels = (int64_t)f->level_ptr.size() - 1;
  info->table_cells = 0;
  for (int32_t x : f->w_host) info->table_cells += x;
  info->relaxations = f->relax;
  info->T_total = f->g->T_total;
  info->M_total = f->g->M_total;
  info->max_row = f->max_row;
  return RC_OK;
}

int rc_min_budget(rc_family f, void* stream, int64_t* B_min) {
  if (!f || !B_min) return RC_E_ARG;
  const int64_t hi0 = 2 * f->g->M_total;           // the chain {V} peaks at 2 M(V)
  if (hi0 >= INT32_MAX) return RC_E_OVERFLOW;
  hipStream_t s = as_stream(stream);
  const size_t scratch = min_budget_scratch_bytes(f, (int32_t)hi0);
  if (scratch > 0 && !f->bmin_scratch) {
    f->bmin_scratch = static_cast<uint32_t*>(f->arena.get(scratch));
    if (!f->bmin_scratch) return RC_E_NOMEM;
  }
  RC_HIP(launch_min_budget(f, (int32_t)hi0, f->bmin_scratch, s));
  DevStatus hs;
  RC_HIP(hipMemcpyAsync(&hs, f->status, sizeof(hs), hipMemcpyDeviceToHost, s));
  RC_HIP(hipStreamSynchronize(s));
  *B_min = hs.bmin;
  return RC_OK;
}

int rc_solve_dual(rc_family f, int64_t B, int32_t objective, void* stream, int64_t* t_opt,
                  int64_t* m_opt, float* fill_ms, int32_t* k, int32_t* chain_host,
                  int32_t* seg_host, uint8_t* cached_host, int64_t* overhead, int64_t* peak,
                  int64_t* cache_mem) {
  DualBuffers need;
  const int st0 = dual_buffers(f, B, objective, &need);
  if (st0 != RC_OK) return st0;
  hipStream_t s = as_stream(stream);
  rcdp::Arena A;
  A.alloc = f->arena.alloc;
  A.free_fn = f->arena.free_fn;
  A.user = f->arena.user;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  auto finish = [&](int st) {
    (void)hipStreamSynchronize(s);
    if (e0) (void)hipEventDestroy(e0);
    if (e1) (void)hipEventDestroy(e1);
    A.release_all();
    return st;
  };
  DualBuffers buf = need;
  buf.D = A.get_n<uint32_t>(need.cells);
  buf.st = A.get_n<DevStatus>(1);
  buf.chain = A.get_n<int32_t>(f->F);
  buf.seg = A.get_n<int32_t>(f->g->n);
  buf.cached = A.get_n<uint8_t>(f->g->n);
  if (!buf.D || !buf.st || !buf.chain || !buf.seg || !buf.cached) return finish(RC_E_NOMEM);
  if (fill_ms && (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess))
    return finish(RC_E_DEVICE);
  const int st = dual_solve(f, objective, buf, e0, e1, s, t_opt, m_opt, k, chain_host, seg_host,
                            cached_host, overhead, peak, cache_mem);
  if (fill_ms && st >= 0) {
    float ms = -1.f;
    if (hipEventElapsedTime(&ms, e0, e1) != hipSuccess) ms = -1.f;
    *fill_ms = ms;
  }
  return finish(st);
}

int rc_family_sets(rc_family f, uint64_t* bits_host, void* stream) {
  if (!f || !bits_host) return RC_E_ARG;
  const int words = f->g->words;
  hipStream_t s = as_stream(stream);
  std::vector<uint64_t> wm((size_t)words * f->fstride);
  if (!wm.empty())
    RC_HIP(hipMemcpyAsync(wm.data(), f->bits, sizeof(uint64_t) * wm.size(), hipMemcpyDeviceToHost, s));
  RC_HIP(hipStreamSynchronize(s));
  for (int64_t i = 0; i < f->F; i++)
    for (int w = 0; w < words; w++) bits_host[i * words + w] = wm[(size_t)w * f->fstride + i];
  return RC_OK;
}

void rc_family_free(rc_family f) {
  if (!f) return;
  (void)hipDeviceSynchronize();
  f->arena.release_all();
  delete f;
}

// ------------------------------------------------------------------ solve

// Level launches suit narrow tables (few columns, many targets per level);
// the persistent wavefront suits wide ones.  RCDP_FILL=level|wavefront
// overrides the choice.
static void destroy_events(rc_solution sol) {
  for (hipEvent_t* e : {&sol->ev0, &sol->ev1, &sol->evk0, &sol->evk1})
    if (*e) {
      (void)hipEventDestroy(*e);
      *e = nullptr;
    }
}

static int choose_fill_path(rc_family f) {
  if (!f->has_records || f->F < 2) return 0;
  // the family's wavefront fill: ghost-zone blocks, or fixed blocks of kJB
  // with the split-panel fill when it can take the family
  const int wave = f->blk_kind == kBlocksGhost ? 2 : (f->has_wide ? 3 : 1);
  const char* env = std::getenv("RCDP_FILL");
  if (env && std::strcmp(env, "level") == 0) return 0;
  if (env && std::strcmp(env, "wavefront") == 0 && f->blk_kind == kBlocksFixed) return 1;
  if (env && (std::strcmp(env, "wide") == 0 || std::strcmp(env, "ghost") == 0)) return wave;
  if (wave == 1) return 0;
  // The wavefront against the level launches, by their measured costs on
  // this GPU.  The wavefront runs its 256-cell columns at most three (the
  // split-panel fill: four) per compute unit at a time, each through every
  // row of the table at about 2.5 us per row.  A level launch costs about 6 us, plus the source reads
  // of its pairs (2 bytes per relaxation) at about 4 TB/s.  Few levels of
  // many sets or of very long rows (the ladder and U-Net shapes) take the
  // level launches; many levels take the wavefront.
  const int64_t levels = (int64_t)f->level_ptr.size() - 1;
  const int64_t slots = (wave == 3 ? wide_slots_per_cu(3) : 3) * (int64_t)num_cus();
  const int64_t col_rounds = ((f->max_row + kWC - 1) / kWC + slots - 1) / slots;
  const double wave_us = 2.5 * (double)f->F * (double)col_rounds;
  const double level_us = 6.0 * (double)levels + 2.0 * (double)f->relax / 4.0e6;
  return level_us < wave_us ? 0 : wave;
}

}  // extern "C"

// A solution handle with its buffers and events; nothing enqueued yet.
static int new_solution(rc_family f, int64_t B, int32_t objective, rc_solution* out,
                        bool level_only = false) {
  if (!f || B < 0) return RC_E_ARG;
  if (objective != RC_TIME_CENTRIC && objective != RC_MEMORY_CENTRIC) return RC_E_ARG;
  const int64_t Beff = std::min<int64_t>(B, 2 * f->g->M_total);
  if (Beff > kMaxBudget32) return RC_E_OVERFLOW;
  // a budget beyond the 16-bit cells: 32-bit cells and the level fill
  const bool cell32 = Beff > kMaxBudget;
  rc_solution sol = new (std::nothrow) rc_solution_s();
  if (!sol) return RC_E_NOMEM;
  sol->f = f;
  sol->B = B;
  sol->Beff = Beff;
  sol->objective = objective;
  sol->arena.alloc = f->arena.alloc;
  sol->arena.free_fn = f->arena.free_fn;
  sol->arena.user = f->arena.user;
  auto fail = [&](int st) {
    destroy_events(sol);
    sol->arena.release_all();
    delete sol;
    return st;
  };
  sol->cell32 = cell32;
  if (cell32)
    sol->m32 = sol->arena.get_n<uint32_t>(f->cells_alloc);
  else
    sol->m = sol->arena.get_n<uint16_t>(f->cells_alloc);
  sol->status = sol->arena.get_n<DevStatus>(1);
  sol->chain = sol->arena.get_n<int32_t>(f->F);
  sol->seg = sol->arena.get_n<int32_t>(f->g->n);
  sol->cached = sol->arena.get_n<uint8_t>(f->g->n);
  if (!(sol->m || sol->m32) || !sol->status || !sol->chain || !sol->seg || !sol->cached)
    return fail(RC_E_NOMEM);
  if (hipEventCreate(&sol->ev0) != hipSuccess || hipEventCreate(&sol->ev1) != hipSuccess)
    return fail(RC_E_DEVICE);
  sol->fill_path = level_only || cell32 ? 0 : choose_fill_path(f);
  if (sol->fill_path != 0 &&
      (hipEventCreate(&sol->evk0) != hipSuccess || hipEventCreate(&sol->evk1) != hipSuccess))
    return fail(RC_E_DEVICE);
  if (sol->fill_path == 3) {
    const int64_t K = wide_columns(f), R = f->wrec_total;
    sol->progress = sol->arena.get_n<int32_t>(K);
    sol->ticket = sol->arena.get_n<int32_t>(1);
    sol->wkey = sol->arena.get_n<int64_t>(R);
    sol->wbl_tmp = sol->arena.get_n<int32_t>(2 * R);
    sol->wtd_tmp = sol->arena.get_n<int32_t>(kWTd * R);
    sol->wbl = sol->arena.get_n<int32_t>(2 * (R + kWPad));
    sol->wtd = sol->arena.get_n<int32_t>(kWTd * (R + kWPad));
    sol->wmeta = sol->arena.get_n<int32_t>(f->nblk * kWMeta);
    sol->wlive = sol->arena.get_n<int32_t>(f->nblk * K);
    sol->wpush = sol->arena.get_n<int32_t>(f->nblk * kJB * kWPush);
    if (!sol->progress || !sol->ticket || !sol->wkey || !sol->wbl_tmp || !sol->wtd_tmp ||
        !sol->wbl || !sol->wtd || !sol->wmeta || !sol->wlive || !sol->wpush)
      return fail(RC_E_NOMEM);
  } else if (sol->fill_path != 0) {
    const int64_t K = sol->fill_path == 2 ? ghost_columns(f) : blocked_columns(f);
    sol->progress = sol->arena.get_n<int32_t>(K);
    sol->ticket = sol->arena.get_n<int32_t>(1);
    sol->crec = sol->arena.get_n<int32_t>(f->clu_total * kRecInts);
    sol->crec_tmp = sol->arena.get_n<int32_t>(f->clu_total * kRecInts);
    sol->live_cap = (int32_t)std::min<int64_t>(K, kLiveCap);
    sol->live = sol->arena.get_n<int32_t>(f->nblk * sol->live_cap * 2);
    sol->blk_meta = sol->arena.get_n<int32_t>(f->nblk * kMetaInts);
    if (sol->fill_path == 2)
      sol->tri = sol->arena.get_n<int32_t>(f->nblk * kJB * kTriInts);
    else
      sol->push = sol->arena.get_n<int32_t>(f->nblk * kJB * kPushInts);
    sol->sentinel = sol->arena.get_n<uint16_t>(8);
    if (!sol->progress || !sol->ticket || !sol->crec || !sol->crec_tmp || !sol->live ||
        !sol->blk_meta || !(sol->push || sol->tri) || !sol->sentinel)
      return fail(RC_E_NOMEM);
  }
  *out = sol;
  return RC_OK;
}

static void drop_solution(rc_solution sol) {
  destroy_events(sol);
  sol->arena.release_all();
  delete sol;
}

// The selection result read back from the device, into the handle.
static int settle_solution(rc_solution sol, const DevStatus& hs, float fill_ms, float kernel_ms) {
  if (hs.error) {
    set_last_error_msg(hs.error == 3   ? "wavefront fill: a wait timed out (kernel aborted)"
                       : hs.error == 4 ? "ghost fill: an in-block shift exceeds the halo"
                                       : "DP fill kernel reported an inconsistency");
    return RC_E_DEVICE;
  }
  sol->fill_ms = fill_ms;
  sol->kernel_ms = kernel_ms;
  sol->t_star = hs.t_sel;
  sol->m_star = hs.t_sel >= 0 ? hs.m_sel : -1;
  sol->result = hs.t_sel >= 0 ? RC_OK : RC_INFEASIBLE;
  return sol->result;
}

static float elapsed(hipEvent_t a, hipEvent_t b) {
  float ms = -1.f;
  if (!a || !b || hipEventElapsedTime(&ms, a, b) != hipSuccess) return -1.f;
  return ms;
}

extern "C" {

}  // extern "C"

// rc_solve and rc_solve_dominance: one table fill, then the selection of t*.
static int solve_one(rc_family f, int64_t B, int32_t objective, void* stream, rc_solution* out,
                     int64_t* t_opt, int64_t* m_opt, bool dominance) {
  if (!f || !out) return RC_E_ARG;
  hipStream_t s = as_stream(stream);
  rc_solution sol = nullptr;
  const int st0 = new_solution(f, B, objective, &sol, dominance);
  if (st0 != RC_OK) return st0;
  if (dominance && sol->cell32) {      // the weak-front kernels take 16-bit cells only
    drop_solution(sol);
    return RC_E_OVERFLOW;
  }
  auto fail = [&](int st) {
    (void)hipStreamSynchronize(s);
    drop_solution(sol);
    return st;
  };
  if (launch_solve_init(sol, s) != hipSuccess) return fail(RC_E_DEVICE);
  int32_t* we = nullptr;              // the skip: end of each row's weak front
  if (dominance && !(we = sol->arena.get_n<int32_t>(f->F))) return fail(RC_E_NOMEM);
  if (hipEventRecord(sol->ev0, s) != hipSuccess) return fail(RC_E_DEVICE);
  const hipError_t fe = dominance               ? launch_fill_dominance(sol, we, s)
                        : sol->fill_path == 3   ? launch_fill_wide(sol, s)
                        : sol->fill_path == 2   ? launch_fill_ghost(sol, s)
                        : sol->fill_path == 1 ? launch_fill_blocked(sol, s)
                                              : launch_fill(sol, s);
  if (fe != hipSuccess) {
    set_last_error(sol->fill_path == 3   ? "split-panel fill launch"
                   : sol->fill_path == 2 ? "ghost fill launch"
                   : sol->fill_path == 1 ? "blocked fill launch"
                                         : "level fill launch",
                   fe);
    return fail(RC_E_DEVICE);
  }
  if (hipEventRecord(sol->ev1, s) != hipSuccess) return fail(RC_E_DEVICE);
  if (launch_select(sol, s) != hipSuccess) return fail(RC_E_DEVICE);
  Staging stage(sizeof(DevStatus));
  if (!stage.data()) return fail(RC_E_NOMEM);
  stage.in_flight();
  if (hipMemcpyAsync(stage.data(), sol->status, sizeof(DevStatus), hipMemcpyDeviceToHost, s) !=
          hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    return fail(RC_E_DEVICE);
  stage.landed();
  const DevStatus hs = *stage.at<DevStatus>(0);
  const float fill_ms = elapsed(sol->ev0, sol->ev1);
  const float kernel_ms = sol->evk0 ? elapsed(sol->evk0, sol->evk1) : fill_ms;
  const int st = settle_solution(sol, hs, fill_ms, kernel_ms);
  if (st < 0) return fail(st);
  if (t_opt) *t_opt = sol->t_star;
  if (m_opt) *m_opt = sol->m_star;
  *out = sol;
  return st;
}

extern "C" {

int rc_solve(rc_family f, int64_t B, int32_t objective, void* stream, rc_solution* out,
             int64_t* t_opt, int64_t* m_opt) {
  return solve_one(f, B, objective, stream, out, t_opt, m_opt, false);
}

int rc_solve_dominance(rc_family f, int64_t B, void* stream, rc_solution* out, int64_t* t_opt,
                       int64_t* m_opt) {
  return solve_one(f, B, RC_TIME_CENTRIC, stream, out, t_opt, m_opt, true);
}

int rc_solve_batch(rc_family f, const int64_t* B_host, int32_t nb, int32_t objective,
                   void* stream, rc_solution* out_host, int64_t* t_opt, int64_t* m_opt) {
  if (!f || !B_host || !out_host || nb <= 0) return RC_E_ARG;
  hipStream_t s = as_stream(stream);
  std::vector<rc_solution> sols;
  auto fail = [&](int st) {
    (void)hipStreamSynchronize(s);
    for (rc_solution x : sols) drop_solution(x);
    return st;
  };
  for (int32_t b = 0; b < nb; b++) {
    rc_solution x = nullptr;
    const int st = new_solution(f, B_host[b], objective, &x);
    if (st != RC_OK) return fail(st);
    sols.push_back(x);
  }
  for (rc_solution x : sols)
    if (launch_solve_init(x, s) != hipSuccess) return fail(RC_E_DEVICE);
  rc_solution s0 = sols[0];
  if (hipEventRecord(s0->ev0, s) != hipSuccess) return fail(RC_E_DEVICE);
  std::vector<BParams> host_prm;
  std::vector<GParams> host_gprm;
  std::vector<WParams> host_wprm;
  // one batched launch when every table takes the same fill (budgets beyond
  // the 16-bit cells take the level fill, one table at a time)
  bool same = true;
  for (rc_solution x : sols) same = same && x->fill_path == s0->fill_path;
  if (!same) {
    for (rc_solution x : sols) {
      const hipError_t fe = x->fill_path == 3   ? launch_fill_wide(x, s)
                            : x->fill_path == 2 ? launch_fill_ghost(x, s)
                            : x->fill_path == 1 ? launch_fill_blocked(x, s)
                                                : launch_fill(x, s);
      if (fe != hipSuccess) {
        set_last_error("fill launch", fe);
        return fail(RC_E_DEVICE);
      }
    }
  } else if (s0->fill_path == 3) {
    host_wprm.resize((size_t)nb);
    WParams* dev_prm = s0->arena.get_n<WParams>(nb);
    if (!dev_prm) return fail(RC_E_NOMEM);
    const hipError_t fe = launch_fill_wide_batch(sols.data(), nb, host_wprm.data(), dev_prm, s);
    if (fe != hipSuccess) {
      set_last_error("batched split-panel fill launch", fe);
      return fail(RC_E_DEVICE);
    }
  } else if (s0->fill_path == 2) {
    host_gprm.resize((size_t)nb);
    GParams* dev_prm = s0->arena.get_n<GParams>(nb);
    if (!dev_prm) return fail(RC_E_NOMEM);
    const hipError_t fe = launch_fill_ghost_batch(sols.data(), nb, host_gprm.data(), dev_prm, s);
    if (fe != hipSuccess) {
      set_last_error("batched ghost fill launch", fe);
      return fail(RC_E_DEVICE);
    }
  } else if (s0->fill_path == 1) {
    host_prm.resize((size_t)nb);
    BParams* dev_prm = s0->arena.get_n<BParams>(nb);
    if (!dev_prm) return fail(RC_E_NOMEM);
    const hipError_t fe = launch_fill_blocked_batch(sols.data(), nb, host_prm.data(), dev_prm, s);
    if (fe != hipSuccess) {
      set_last_error("batched blocked fill launch", fe);
      return fail(RC_E_DEVICE);
    }
  } else {
    for (rc_solution x : sols) {
      const hipError_t fe = launch_fill(x, s);
      if (fe != hipSuccess) {
        set_last_error("level fill launch", fe);
        return fail(RC_E_DEVICE);
      }
    }
  }
  if (hipEventRecord(s0->ev1, s) != hipSuccess) return fail(RC_E_DEVICE);
  for (rc_solution x : sols)
    if (launch_select(x, s) != hipSuccess) return fail(RC_E_DEVICE);
  Staging stage(sizeof(DevStatus) * (size_t)nb);
  if (!stage.data()) return fail(RC_E_NOMEM);
  stage.in_flight();
  for (int32_t b = 0; b < nb; b++)
    if (hipMemcpyAsync(stage.at<DevStatus>(0) + b, sols[b]->status, sizeof(DevStatus),
                       hipMemcpyDeviceToHost, s) != hipSuccess)
      return fail(RC_E_DEVICE);
  if (hipStreamSynchronize(s) != hipSuccess) return fail(RC_E_DEVICE);
  stage.landed();
  const float fill_ms = elapsed(s0->ev0, s0->ev1);
  const float kernel_ms = s0->evk0 ? elapsed(s0->evk0, s0->evk1) : fill_ms;
  for (int32_t b = 0; b < nb; b++) {
    const int st = settle_solution(sols[b], stage.at<DevStatus>(0)[b], fill_ms, kernel_ms);
    if (st < 0) return fail(st);
  }
  for (int32_t b = 0; b < nb; b++) {
    out_host[b] = sols[b];
    if (t_opt) t_opt[b] = sols[b]->t_star;
    if (m_opt) m_opt[b] = sols[b]->m_star;
  }
  return RC_OK;
}

int rc_solution_fill_ms(rc_solution s, float* ms) {
  if (!s || !ms) return RC_E_ARG;
  *ms = s->fill_ms;
  return RC_OK;
}

int rc_solution_fill_kernel_ms(rc_solution s, float* ms) {
  if (!s || !ms) return RC_E_ARG;
  *ms = s->kernel_ms;
  return RC_OK;
}

int rc_solution_fill_path(rc_solution s, int32_t* path) {
  if (!s || !path) return RC_E_ARG;
  *path = s->fill_path == 0 && s->cell32 ? 4 : s->fill_path;
  return RC_OK;
}

int rc_solution_trace_path(rc_solution s, int32_t* path) {
  if (!s || !path) return RC_E_ARG;
  *path = s->trace_path;
  return RC_OK;
}

int rc_reconstruct(rc_solution sol, void* stream, int32_t* k, int32_t* chain_host,
                   int32_t* seg_host, uint8_t* cached_host, int64_t* overhead, int64_t* peak,
                   int64_t* cache_mem) {
  if (!sol) return RC_E_ARG;
  if (sol->result != RC_OK) return RC_INFEASIBLE;
  hipStream_t s = as_stream(stream);
  rc_family f = sol->f;
  const int n = f->g->n;
  // the chain has at most min(F, n + 1) sets: every step adds a node
  const int64_t kmax = std::min<int64_t>(f->F, (int64_t)n + 1);
  StageLayout lay;
  const size_t o_st = lay.add<DevStatus>(1), o_ch = lay.add<int32_t>(kmax),
               o_sg = lay.add<int32_t>(n), o_ca = lay.add<uint8_t>(n);
  Staging stage(lay.bytes);
  if (!sol->pack) sol->pack = sol->arena.get(lay.bytes);
  if (!stage.data() || !sol->pack) return RC_E_NOMEM;
  const hipError_t te = launch_trace(sol, s);
  if (te == hipErrorOutOfMemory) return RC_E_NOMEM;
  if (te != hipSuccess) {
    set_last_error("traceback launch", te);
    return RC_E_DEVICE;
  }
  PackList PL;
  PL.add(sol->status, sizeof(DevStatus), (int64_t)o_st);
  PL.add(sol->chain, sizeof(int32_t) * kmax, (int64_t)o_ch);
  PL.add(sol->seg, sizeof(int32_t) * n, (int64_t)o_sg);
  PL.add(sol->cached, (n + 3) / 4 * 4, (int64_t)o_ca);   // whole words of the padded buffer
  const int pc = pack_to_host(PL, sol->pack, lay.bytes, stage, s);
  if (pc != RC_OK) return pc;
  RC_HIP(hipStreamSynchronize(s));
  stage.landed();
  const DevStatus hs = *stage.at<DevStatus>(o_st);
  if (hs.error || hs.k < 0 || hs.k > kmax) {
    set_last_error_msg("traceback: optarg walk did not end at (empty set, 0)");
    return RC_E_DEVICE;
  }
  if (k) *k = hs.k;
  if (chain_host) std::copy(stage.at<int32_t>(o_ch), stage.at<int32_t>(o_ch) + hs.k, chain_host);
  if (seg_host) std::copy(stage.at<int32_t>(o_sg), stage.at<int32_t>(o_sg) + n, seg_host);
  if (cached_host) std::copy(stage.at<uint8_t>(o_ca), stage.at<uint8_t>(o_ca) + n, cached_host);
  if (overhead) *overhead = hs.overhead;
  if (peak) *peak = hs.peak;
  if (cache_mem) *cache_mem = hs.cache_mem;
  return RC_OK;
}

int rc_export_table(rc_solution sol, int64_t first, int64_t count, int64_t* m_host,
                    int32_t* arg_host, void* stream) {
  if (!sol || first < 0 || count < 0 || first + count > sol->f->F) return RC_E_ARG;
  rc_family f = sol->f;
  hipStream_t s = as_stream(stream);
  const int64_t W = f->g->T_total + 1;
  if (arg_host && !sol->arg) {               // optarg of the whole table, derived once
    sol->arg = sol->arena.get_n<uint16_t>(f->cells_alloc);
    if (!sol->arg) return RC_E_NOMEM;
    RC_HIP(launch_arg_all(sol, s));
  }
  const int64_t c0 = f->row_off_host[first], c1 = f->row_off_host[first + count];
  std::vector<uint16_t> mm(sol->cell32 ? 0 : c1 - c0), aa(arg_host ? c1 - c0 : 0);
  std::vector<uint32_t> mm32(sol->cell32 ? c1 - c0 : 0);
  if (c1 > c0) {
    if (sol->cell32)
      RC_HIP(hipMemcpyAsync(mm32.data(), sol->m32 + c0, 4 * (c1 - c0), hipMemcpyDeviceToHost, s));
    else
      RC_HIP(hipMemcpyAsync(mm.data(), sol->m + c0, 2 * (c1 - c0), hipMemcpyDeviceToHost, s));
    if (arg_host)
      RC_HIP(hipMemcpyAsync(aa.data(), sol->arg + c0, 2 * (c1 - c0), hipMemcpyDeviceToHost, s));
  }
  RC_HIP(hipStreamSynchronize(s));
  const uint32_t inf = sol->cell32 ? 0xFFFFFFFFu : kInfM;
  for (int64_t r = 0; r < count; r++) {
    const int64_t set = first + r;
    const int64_t off = f->row_off_host[set] - c0;
    const int64_t w = f->w_host[set];
    for (int64_t t = 0; t < W; t++) {
      const bool in = t < w;
      const uint32_t mv = !in ? inf : sol->cell32 ? mm32[off + t] : mm[off + t];
      const uint32_t av = (in && arg_host) ? aa[off + t] : kNoArg;
      if (m_host) m_host[r * W + t] = mv == inf ? -1 : (int64_t)mv;
      if (arg_host) arg_host[r * W + t] = (mv == inf || av == kNoArg) ? -1 : (int32_t)av;
    }
  }
  return RC_OK;
}

void rc_solution_free(rc_solution sol) {
  if (!sol) return;
  (void)hipDeviceSynchronize();
  destroy_events(sol);
  sol->arena.release_all();
  delete sol;
}

}  // extern "C"
