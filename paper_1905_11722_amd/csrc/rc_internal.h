// Internal declarations of the MI355X recomputation-DP library.
// Every kernel and launcher shared between the .hip translation units is
// declared here; the C ABI lives in include/rc.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

#include "rc.h"

namespace rcdp {

constexpr int kMaxNodes = 4096;                 // words <= 64 = one lane per word
constexpr int kMaxWords = kMaxNodes / 64;
constexpr int kMaxSets = 65535;                 // family index fits 16 bits
constexpr uint32_t kInfM = 0xFFFFu;             // opt = infinity in a 16-bit cell
constexpr uint32_t kNoArg = 0xFFFFu;            // optarg = none
constexpr int64_t kRowAlign = 64;               // cells; rows end on 128-byte lines
constexpr int64_t kGuard = 256;                 // infinite cells before every row and after
                                                // the last one (a 256-cell window that
                                                // overlaps a row reads no other row)
constexpr int kJB = 8;                          // blocked fill: targets per block
constexpr int64_t kMaxRecords = (int64_t)1 << 21;  // blocked fill: cap on panel records
constexpr int kRecInts = 32;                    // blocked fill: int32 per compact record
constexpr int kRecDma = 24;                     // blocked fill: first record word of the
                                                // column-independent window DMA terms
constexpr int kSpan = 248;                      // blocked fill: shifts staged together
constexpr int kHalo = 512;                      // blocked fill: row pushes with shift <= kHalo
                                                // read the row's halo, larger ones a window
constexpr int kFarMax = 2 * kJB - 1;            // blocked fill: targets of one row's pushes
constexpr int kPushInts = 64;                   // blocked fill: int32 per (block, row) push list
constexpr int kMetaInts = 8;                    // blocked fill: int32 per block
constexpr int kLiveCap = 2048;                  // blocked fill: columns with their own live counts
constexpr uint32_t kPendM = 0xFFFE;             // blocked fill: cell not written yet
constexpr int64_t kMaxBudget = 0xFFFC;          // finite opt values stay below kPendM
constexpr int64_t kMaxBudget32 = (int64_t)1 << 30;   // uint32 cells: min(B, 2 M(V)) up to this
constexpr int kBlocksFixed = 1;                 // family blocks: kJB targets each (row pushes)
constexpr int kBlocksGhost = 2;                 // family blocks: cut to fit the ghost halo
constexpr int kGhostHalo = 64;                  // ghost-zone fill: cells recomputed to the right
constexpr int kGhostMaxSets = 4096;             // ghost-zone fill: largest family it takes
constexpr int kWideMinSets = 100;               // families this large take the split-panel fill
constexpr int kNear = kJB;                      // ghost cut: predecessors j-1 .. j-kNear examined
constexpr int kTriInts = 16;                    // ghost-zone fill: int32 per (block, row) list
constexpr int kWC = 256;                        // split-panel fill: cells per column
constexpr int kWH = 512;                        // split-panel fill: halo cells of a row push
constexpr int kWTd = 8;                         // split-panel fill: int32 budgets + additions
constexpr int kWPad = 64;                       // split-panel fill: records read past the end
constexpr int kWMeta = 8;                       // split-panel fill: int32 per block
constexpr int kWMaxRec = 4096;                  // split-panel fill: records of one block
constexpr int kWPush = 64;                      // split-panel fill: int32 per (block, row) list
// layout of a split-panel push list (one row of a block and its 16 target slots:
// the later rows of its block, then the rows of the next block)
constexpr int kWpE = 0;                         // [16] shift of each slot, -1 = no live pair
constexpr int kWpTau = 16;                      // [8] budgets of slots 2q, 2q+1 (uint16 pairs)
constexpr int kWpDm = 24;                       // [8] additions of slots 2q, 2q+1
constexpr int kWpP = 32;                        // P_j of the row
constexpr int kWpEnd = 33;                      // [2] index of the row's cell u = 0
constexpr int kWpEmax = 35;                     // largest live shift
constexpr int kWpMaxPt = 36;                    // largest P of a live target (-1 none)
constexpr int kWpHalo = 37;                     // halo cells to stage (multiple of 64)
constexpr int kWpFar = 38;                      // bit mask of slots with shift > kWH
constexpr int kWpNear = 39;                     // bit mask of slot pairs with a shift <= kWH

// Cells of row slot s: the row's w cells right-aligned on a kRowAlign
// boundary, preceded by at least kGuard padding cells (infinity).
__host__ __device__ inline int64_t row_slot(int64_t w) {
  return (w + kRowAlign - 1) / kRowAlign * kRowAlign + kGuard;
}

// Device allocator with ownership tracking.
struct Arena {
  rc_alloc_fn alloc = nullptr;
  rc_free_fn free_fn = nullptr;
  void* user = nullptr;
  std::vector<void*> ptrs;
  char* cur = nullptr;                         // free part of the current chunk
  char* end = nullptr;
  static constexpr size_t kChunk = (size_t)4 << 20;
  void* get(size_t bytes);                     // nullptr on failure; 256-byte aligned
  void* raw(size_t bytes);                     // one call of the allocator
  template <class T> T* get_n(int64_t count) {
    return static_cast<T*>(get(sizeof(T) * (size_t)(count > 0 ? count : 1)));
  }
  void release_all();
};

// Small device status block: error flags and scalar results.
struct DevStatus {
  int32_t error;         // nonzero: a kernel found an inconsistency
  int32_t overflow;      // family enumeration exceeded its cap
  int64_t count;         // enumeration counter / family size
  int32_t t_sel;         // selection result
  int32_t m_sel;
  int64_t walg;          // relaxations
  int32_t k;             // chain length
  int32_t pad0;
  int64_t overhead, peak, cache_mem;
  int64_t bmin;          // smallest feasible budget (rc_min_budget)
};

// One pair (L, L') of the level fill (fill.hip): the source row's first
// cell lo, the source cell of target cell t' of L' at base - row_off(L') + t'
// (base = lo - dt), the budget term, the addition, the source row's width
// and index.
struct LevelPair {
  int64_t lo;
  int64_t base;
  int32_t c;
  int32_t dm;
  int32_t w;
  int32_t src;
};

// Panel / triangle records of the blocked fill (blocks.hip).
struct BlockRecords {
  int32_t* src = nullptr;       // [R] source family index
  int32_t* e = nullptr;         // [R * kJB] shift of (src, j0 + slot), -1 = no pair
  uint32_t* kadd = nullptr;     // [R * kJB] (dm << 16) | src
  int32_t* c = nullptr;         // [R * kJB] budget term
  int32_t* tri_e = nullptr;     // [nblk * kJB * kJB] in-block pairs (row slot, target slot)
  uint32_t* tri_kadd = nullptr;
  int32_t* tri_c = nullptr;
};

}  // namespace rcdp

struct rc_graph_s {
  int32_t n = 0, words = 0;
  int64_t T_total = 0, M_total = 0;
  rcdp::Arena arena;
  // device
  int32_t* dT = nullptr;          // [n]
  int32_t* dM = nullptr;          // [n]
  uint64_t* dSucc = nullptr;      // [n][words] successor masks
  uint64_t* dPred = nullptr;      // [n][words] predecessor masks
  int32_t* dPredPtr = nullptr;    // [n+1] predecessor CSR
  int32_t* dPredIdx = nullptr;
  int32_t num_pred_edges = 0;
  int32_t* dByDepth = nullptr;    // nodes sorted by depth (longest path from a source)
  int32_t* dDepthPtr = nullptr;   // [num_depths+1]
  int32_t num_depths = 0;
  int32_t num_sinks = 0;          // nodes without successors
  uint64_t* dAnc = nullptr;       // [n][words] ancestors of each node (without the node),
                                  // the pruned family's generators, computed once per graph
};

struct rc_family_s {
  rc_graph g = nullptr;
  int32_t mode = 0;
  int64_t F = 0, P = 0, cells = 0, relax = 0, max_row = 0;
  int64_t cells_alloc = 0;        // cells + kGuard: the table with its trailing guard
  int64_t fstride = 0;            // stride of the word-major bitmask arrays
  rcdp::Arena arena;
  // device: family, word-major [words][fstride]
  uint64_t* bits = nullptr;
  uint64_t* bd = nullptr;
  // device: per set [F]
  int32_t *size = nullptr, *Tsum = nullptr, *Msum = nullptr, *Tbd = nullptr, *Mbd = nullptr;
  int32_t *A = nullptr, *w = nullptr;
  int64_t* row_off = nullptr;     // [F+1], rows padded to kRowAlign cells
  // device: predecessor pairs, CSR by target
  int64_t* pred_ptr = nullptr;    // [F+1]
  int32_t *pidx = nullptr, *pdt = nullptr, *pdm = nullptr, *pc = nullptr;
  rcdp::LevelPair* lpair = nullptr; // [P] the level fill's pair records (built on first use)
  // blocked fill: records per block of at most kJB targets (absent when too large)
  int32_t blk_kind = 0;           // kBlocksFixed or kBlocksGhost (0: no records)
  int64_t nblk = 0;
  int32_t* bstart = nullptr;      // [nblk+1] first target of each block
  std::vector<int32_t> bstart_host;
  int64_t rec_total = 0;
  bool has_records = false;
  int64_t* rec_ptr = nullptr;     // [nblk+1]
  int64_t* clu_ptr = nullptr;     // [nblk+1] compact records (shift clusters) per block
  int64_t clu_total = 0;
  int64_t* wrec_ptr = nullptr;    // [nblk+1] split-panel records per block (upper bound)
  int64_t wrec_total = 0;
  bool has_wide = false;          // the split-panel fill can take this family
  rcdp::BlockRecords rec;
  rcdp::DevStatus* status = nullptr;
  uint32_t* bmin_scratch = nullptr; // rc_min_budget: f values of large families
  // host copies used for launches
  std::vector<int64_t> level_ptr; // family index ranges of equal set size
  std::vector<int64_t> level_pairs; // the most pairs of a target in each level
  std::vector<int32_t> level_maxw;
  std::vector<int32_t> w_host;
  std::vector<int64_t> row_off_host;
};

struct rc_solution_s {
  // cells of 32 bits when min(B, 2 M(V)) exceeds kMaxBudget: m32 holds the
  // table (the level fill), m stays null
  bool cell32 = false;
  uint32_t* m32 = nullptr;
  rc_family f = nullptr;
  int64_t B = 0, Beff = 0;
  int32_t objective = 0;
  int32_t result = 0;             // RC_OK or RC_INFEASIBLE
  int64_t t_star = -1, m_star = -1;
  rcdp::Arena arena;
  uint16_t* m = nullptr;          // [cells] opt values, kInfM = infinity
  uint16_t* arg = nullptr;        // [cells] optarg, derived on demand by rc_export_table
  rcdp::DevStatus* status = nullptr;
  int32_t* chain = nullptr;       // [F]
  int32_t* seg = nullptr;         // [n]
  uint8_t* cached = nullptr;      // [n]
  void* pack = nullptr;           // the traceback's results gathered for one copy to the host
  uint32_t* nxt = nullptr;        // the traceback's optarg slice [F * (t* + 1)] (fill.hip)
  int64_t nxt_cells = 0;
  int32_t trace_path = -1;        // the last traceback: 0 predecessor scans, 1 optarg slice
  int32_t* progress = nullptr;    // blocked fill: rows finished per column
  int32_t* ticket = nullptr;      // blocked fill: next column to take
  int32_t* crec = nullptr;        // blocked fill: compact live records [clu_total * kRecInts]
  int32_t* crec_tmp = nullptr;    // blocked fill: the same records before sorting
  int32_t* live = nullptr;        // blocked fill: live records per (block, column, kind)
  int32_t live_cap = 0;           // blocked fill: columns of the live table (min(K, kLiveCap))
  int32_t* blk_meta = nullptr;    // blocked fill: per block metadata [nblk * kMetaInts]
  int32_t* push = nullptr;        // blocked fill: row push lists [nblk * kJB * kPushInts]
  int32_t* tri = nullptr;         // ghost-zone fill: in-block lists [nblk * kJB * kTriInts]
  int64_t* wkey = nullptr;        // split-panel fill: sort keys of the unsorted records
  int32_t* wbl_tmp = nullptr;     // split-panel fill: unsorted window base / limit
  int32_t* wtd_tmp = nullptr;     // split-panel fill: unsorted budgets / additions
  int32_t* wbl = nullptr;         // split-panel fill: [2 (R + kWPad)] sorted
  int32_t* wtd = nullptr;         // split-panel fill: [kWTd (R + kWPad)] sorted
  int32_t* wmeta = nullptr;       // split-panel fill: [nblk * kWMeta]
  int32_t* wlive = nullptr;       // split-panel fill: [nblk * K] records reaching each column
  int32_t* wpush = nullptr;       // split-panel fill: [nblk * kJB * kWPush]
  int32_t cpt = 1;                // blocked fill: cells per thread of a column
  uint16_t* sentinel = nullptr;   // 8 cells of infinity
  int32_t fill_path = 0;          // 0 level launches, 1 row-push wavefront, 2 ghost-zone
                                  // wavefront, 3 split-panel wavefront
  hipEvent_t ev0 = nullptr, ev1 = nullptr;    // around the whole fill
  hipEvent_t evk0 = nullptr, evk1 = nullptr;  // around the wavefront kernel alone
  float fill_ms = 0.f;
  float kernel_ms = 0.f;
};

namespace rcdp {

// Thread-local description of the last RC_E_DEVICE (rc_api.hip).
void set_last_error(const char* what, hipError_t e);
void set_last_error_msg(const char* msg);

// Seed of the wavefront fills' random delays (the race test), from the
// environment switch RCDP_JITTER; 0 (unset): no delays (rc_api.hip).
int32_t jitter_seed();

// Pinned host memory for the copies between host and device inside one
// call (rc_api.hip).  A copy to or from pinned memory is asynchronous, so
// the copies of a call cost one synchronisation of the stream; a copy to or
// from pageable memory waits for itself.  Buffers come from a process-wide
// pool (kept until the process ends), one caller at a time; data() is null
// when pinned memory could not be had.  Between in_flight() (copies are
// enqueued) and landed() (the stream was synchronised) the buffer is not
// returned to the pool: a call that leaves on an error in between gives it
// up rather than hand a buffer with copies still pending to another call.
class Staging {
 public:
  explicit Staging(size_t bytes);
  ~Staging();
  Staging(const Staging&) = delete;
  Staging& operator=(const Staging&) = delete;
  char* data() const { return p_; }
  template <class T> T* at(size_t byte_offset) const {
    return reinterpret_cast<T*>(p_ + byte_offset);
  }
  void in_flight() { pending_ = true; }
  void landed() { pending_ = false; }

 private:
  char* p_ = nullptr;
  size_t n_ = 0;
  bool pending_ = false;
};

// Byte offsets of consecutive parts of a staging buffer, each aligned to 64.
struct StageLayout {
  size_t bytes = 0;
  template <class T> size_t add(int64_t count) {
    const size_t off = bytes;
    bytes += (sizeof(T) * (size_t)(count > 0 ? count : 0) + 63) & ~size_t(63);
    return off;
  }
};

// ---- utilities (family.hip)
hipError_t launch_zero(void* p, size_t bytes, hipStream_t s);  // bytes % 8 == 0
// Device segments gathered into one device buffer (whole 32-bit words; the
// byte counts, offsets and pointers are multiples of 4).
struct PackSeg {
  const void* src;
  int64_t bytes;
  int64_t dst_off;
};
constexpr int kPackMax = 8;
struct PackList {
  PackSeg seg[kPackMax];
  int32_t n = 0;
  void add(const void* src, int64_t bytes, int64_t dst_off) {
    if (bytes > 0) seg[n++] = PackSeg{src, bytes, dst_off};
  }
};
hipError_t launch_pack(const PackList& L, void* dst, hipStream_t s);

// ---- graph kernels (family.hip)
hipError_t launch_graph_masks(rc_graph g, const int32_t* d_row_ptr, const int32_t* d_col_idx,
                              hipStream_t s);

// ---- family kernels (family.hip)
hipError_t launch_ancestors(rc_graph g, uint64_t* anc, hipStream_t s);
hipError_t launch_pruned_candidates(rc_graph g, const uint64_t* anc, uint64_t* cand,
                                    hipStream_t s);
hipError_t launch_enum_exact(rc_graph g, uint64_t* cand, int64_t cap, int32_t* lvl,
                             DevStatus* st, hipStream_t s);
hipError_t launch_rank(rc_graph g, int32_t mode, const uint64_t* cand, int64_t ncand_max,
                       const int32_t* lvl, uint64_t* bits, int64_t fstride, DevStatus* st,
                       hipStream_t s);
hipError_t launch_set_quantities(rc_family f, hipStream_t s);
hipError_t launch_pair_count(rc_family f, int64_t* counts, hipStream_t s);
hipError_t launch_scan(const int64_t* in, int64_t* out, int64_t count, int64_t align,
                       hipStream_t s);
hipError_t launch_pair_write(rc_family f, int64_t* walg_per_target, hipStream_t s);
hipError_t launch_row_widths(rc_family f, int64_t* padded, hipStream_t s);
hipError_t launch_sum(const int64_t* in, int64_t count, int64_t* out, hipStream_t s);

// ---- DP kernels (fill.hip)
hipError_t launch_solve_init(rc_solution sol, hipStream_t s);
hipError_t launch_fill(rc_solution sol, hipStream_t s);
hipError_t launch_select(rc_solution sol, hipStream_t s);
hipError_t launch_trace(rc_solution sol, hipStream_t s);
hipError_t launch_arg_all(rc_solution sol, hipStream_t s);

// ---- blocked fill (blocks.hip, blocked.hip)
hipError_t launch_row_align(rc_family f, hipStream_t s);
hipError_t launch_blk_count(rc_family f, int64_t nblk, int64_t* count, hipStream_t s);
hipError_t launch_blk_fill(rc_family f, int64_t nblk, hipStream_t s);
hipError_t launch_blk_clusters(rc_family f, int64_t* count, hipStream_t s);
hipError_t launch_rec_prepare(rc_solution sol, hipStream_t s);
hipError_t launch_push_prepare(rc_solution sol, int32_t C, hipStream_t s);
hipError_t launch_rec_sort(rc_solution sol, int32_t C, int32_t H, hipStream_t s);
hipError_t launch_fill_pending(rc_solution sol, hipStream_t s);
hipError_t launch_pad_init(rc_solution sol, hipStream_t s);
int blocked_cells_per_thread(rc_family f);
int num_cus();                          // compute units of the current device (cached)

// Kernel parameters of one table of the blocked fill (blocked.hip).
struct BParams {
  int32_t F;
  int32_t nblk;
  int32_t K;                             // columns
  const int32_t* w;
  const int64_t* row_off;
  const int64_t* clu_ptr;                // first compact panel record of each block
  const int32_t* crec;
  const int32_t* meta;                   // [nblk * kMetaInts]
  const int32_t* push;                   // [nblk * kJB * kPushInts]
  const int32_t* live;                   // [nblk * cap * 2] live panel records per column
  int32_t cap;
  int32_t jitter;                        // race test: seed of random delays (0: none)
  const uint16_t* sentinel;              // 8 cells of infinity
  uint16_t* m;
  int32_t* progress;
  int32_t* ticket;
  DevStatus* st;
  int64_t timeout_ticks;
};
hipError_t launch_fill_blocked_batch(rc_solution* sols, int32_t nb, BParams* host_prm,
                                     BParams* dev_prm, hipStream_t s);

// ---- ghost-zone wavefront fill (ghost.hip)
// Kernel parameters of one table.
struct GParams {
  int32_t F;
  int32_t nblk;
  int32_t K;                             // columns
  const int32_t* bstart;                 // [nblk + 1]
  const int64_t* clu_ptr;                // first compact panel record of each block
  const int32_t* crec;
  const int32_t* meta;                   // [nblk * kMetaInts]
  const int32_t* tri;                    // [nblk * kJB * kTriInts]
  const int32_t* live;                   // [nblk * cap * 2] live panel records per column
  int32_t cap;
  int32_t jitter;                        // race test: seed of random delays (0: none)
  const uint16_t* sentinel;              // 8 cells of infinity
  uint16_t* m;
  int32_t* progress;
  int32_t* ticket;
  DevStatus* st;
  int64_t timeout_ticks;
};
// near[j * kNear + d - 1] = right-aligned shift of the pair (L_{j-d}, L_j), -1 without one.
hipError_t launch_near_shifts(rc_family f, int32_t* near, hipStream_t s);
// Cut targets 1..F-1 into blocks of at most kJB whose in-block dependency
// cones fit kGhostHalo cells (host; near from launch_near_shifts).
std::vector<int32_t> ghost_cut(int64_t F, const std::vector<int32_t>& near);
int ghost_cells_per_thread(rc_family f);
int64_t ghost_columns(rc_family f);
hipError_t launch_fill_ghost(rc_solution sol, hipStream_t s);
hipError_t launch_fill_ghost_batch(rc_solution* sols, int32_t nb, GParams* host_prm,
                                   GParams* dev_prm, hipStream_t s);

// ---- smallest feasible budget (budget.hip)
size_t min_budget_scratch_bytes(rc_family f, int32_t hi0);
hipError_t launch_min_budget(rc_family f, int32_t hi0, uint32_t* scratch, hipStream_t s);
// Memory-indexed table of Algorithm 1's recursion (dual.hip): D[F * W]
// uint32, W = min(B, M(V)) + 1; t and the least m of the objective into
// st->t_sel / st->m_sel (-1 when no chain reaches V).  level_pairs[l]: the
// most pairs of a target of size level l.  e0/e1 (may be null) are recorded
// around the table's launches.
hipError_t launch_dual(rc_family f, const std::vector<int64_t>& level_pairs, int32_t B, int32_t W,
                       int objective, uint32_t* D, DevStatus* st, hipEvent_t e0, hipEvent_t e1,
                       hipStream_t s);
int64_t blocked_columns(rc_family f);

// One memory-indexed solve (rc_api.hip): the sizes it needs and the device
// buffers it runs in (the caller's arena, or the static scratch of the
// allocation-free entry point).
struct DualBuffers {
  int64_t Beff = 0, W = 0, cells = 0;
  uint32_t* D = nullptr;          // [cells]
  DevStatus* st = nullptr;
  int32_t* chain = nullptr;       // [F]
  int32_t* seg = nullptr;         // [n]
  uint8_t* cached = nullptr;      // [n]
};
int dual_buffers(rc_family f, int64_t B, int32_t objective, DualBuffers* out);
int dual_solve(rc_family f, int32_t objective, const DualBuffers& b, hipEvent_t e0,
               hipEvent_t e1, hipStream_t s, int64_t* t_opt, int64_t* m_opt, int32_t* k,
               int32_t* chain_host, int32_t* seg_host, uint8_t* cached_host, int64_t* overhead,
               int64_t* peak, int64_t* cache_mem);
hipError_t launch_fill_blocked(rc_solution sol, hipStream_t s);


// ---- split-panel wavefront fill (wide.hip)
// Kernel parameters of one table.
struct WParams {
  int32_t F;
  int32_t nblk;
  int32_t K;                             // columns of kWC cells
  int32_t rec_cap;                       // records of the family (upper bound)
  const int32_t* meta;                   // [nblk * kWMeta]
  const int64_t* rptr;                   // [nblk + 1] first record of each block
  const int32_t* live;                   // [nblk * K] records reaching each column
  const int32_t* bl;                     // [2 (R + kWPad)] window base / limit (bytes)
  const int32_t* td;                     // [kWTd (R + kWPad)] budgets / additions
  const int32_t* push;                   // [nblk * kJB * kWPush]
  uint16_t* m;
  int64_t m_bytes;                       // the table with its trailing guard
  int32_t null_off;                      // byte offset of the trailing guard
  int32_t jitter;                        // race test: seed of random delays (0: none)
  int32_t* progress;
  int32_t* ticket;
  DevStatus* st;
  int64_t timeout_ticks;
};
// Resident workgroups per compute unit of the split-panel fill with np
// panel waves: sixteen waves, four per SIMD.
__host__ __device__ constexpr int wide_slots_per_cu(int np) { return 16 / (np + 1); }
int64_t wide_columns(rc_family f);
hipError_t launch_wide_count(rc_family f, int64_t* count, hipStream_t s);
hipError_t launch_fill_wide(rc_solution sol, hipStream_t s);
hipError_t launch_fill_wide_batch(rc_solution* sols, int32_t nb, WParams* host_prm,
                                  WParams* dev_prm, hipStream_t s);

}  // namespace rcdp
