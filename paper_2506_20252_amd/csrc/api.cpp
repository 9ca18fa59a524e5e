// C-ABI of the PAT library: argument checks, plan cache, execution modes.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <memory>
#include <mutex>
#include <tuple>
#include <vector>

#include "../../include/pat.h"
#include "kernels.hpp"
#include "plan.hpp"

namespace {

constexpr size_t kDefaultBudget = size_t(8) << 20;
constexpr uint32_t kDefaultTimeoutUs = 10u * 1000u * 1000u;
constexpr int kMaxRanks = 1 << 16;

std::mutex g_mu;
size_t g_budget = 0;     // 0: default
int g_mode = -1;         // -1: environment / default
uint32_t g_timeout_us = 0;  // 0: default
int g_order = -1;           // -1: environment / default (far-first)
int g_fusion = -1;          // -1: environment / default (auto)
int g_aggregation = -1;     // -1: environment / default (power-of-two sub-trees)
std::atomic<int> g_last_hip{0};

size_t budget_now() {
  if (g_budget) return g_budget;
  if (const char* e = std::getenv("PAT_BUFFER_BYTES")) {
    const long long v = std::atoll(e);
    if (v > 0) return size_t(v);
  }
  return kDefaultBudget;
}

int mode_now() {
  if (g_mode >= 0) return g_mode;
  if (const char* e = std::getenv("PAT_EXEC_MODE")) {
    if (!std::strcmp(e, "persistent")) return PAT_EXEC_PERSISTENT;
    if (!std::strcmp(e, "graph")) return PAT_EXEC_GRAPH;
    if (!std::strcmp(e, "dataflow")) return PAT_EXEC_DATAFLOW;
  }
  return PAT_EXEC_STREAM;
}

int order_now() {
  if (g_order >= 0) return g_order;
  if (const char* e = std::getenv("PAT_LINEAR_ORDER"))
    if (!std::strcmp(e, "close")) return pat::kCloseFirst;
  return pat::kFarFirst;
}

int aggregation_now() {
  if (g_aggregation >= 0) return g_aggregation;
  if (const char* e = std::getenv("PAT_AGGREGATION"))
    if (!std::strcmp(e, "budget")) return PAT_AGGREGATION_BUDGET;
  return PAT_AGGREGATION_POW2;
}

// Pipelined pieces (tuning): PAT_PIECE_PIPELINE=1 when a plan is made cuts a
// chunk larger than the budget into pieces of half the budget, alternating
// between two halves of every slot, and runs two pieces' steps per launch.
bool pipeline_now() {
  const char* e = std::getenv("PAT_PIECE_PIPELINE");
  return e && e[0] == '1';
}

int fusion_now() {
  if (g_fusion >= 0) return g_fusion;
  if (const char* e = std::getenv("PAT_TOP_FUSION")) {
    if (!std::strcmp(e, "on")) return PAT_FUSION_ON;
    if (!std::strcmp(e, "off")) return PAT_FUSION_OFF;
  }
  return PAT_FUSION_AUTO;
}

// Tuning overrides come from the environment (positive integers only).
int64_t env_or(const char* name, int64_t dflt) {
  if (const char* e = std::getenv(name)) {
    const long long v = std::atoll(e);
    if (v > 0) return v;
  }
  return dflt;
}

// Vectors of a chunk per workgroup of a fused range, for N trees of V-vector
// chunk-pieces.  A fused launch is a chain of dependent steps that every
// workgroup runs for its (tree, tile): smaller tiles spread a step over more
// workgroups, but once the grid outgrows what the chip holds at once, a
// second round of workgroups runs the whole chain again.  So: the smallest
// power of two from 32 vectors up to 256 with N x tiles <= 1024 workgroups
// (every variant of the fused kernel keeps at least 5 workgroups of 256 lanes
// resident per CU, 1280 on 256 CUs), capped at V.  Measured on MI355X against
// a fixed 256: N=24 64 KiB bf16 all-gather 27.0 -> 21.0 us, N=128 4 KiB
// float32 reduce-scatter 51.3 -> 37.9 us.  PAT_TREE_TILE overrides.
int64_t tree_tile_vecs(int N, int64_t V) {
  int64_t t = 32;
  while (t < 256 && int64_t(N) * ((V + t - 1) / t) > 1024) t *= 2;
  return env_or("PAT_TREE_TILE", t);
}

// PAT_FUSION_AUTO fuses the far end of the fusable steps: those that move at
// most 128 MiB (short, latency-bound steps) and whose edges of one tree,
// times the vectors of one tile, fit a few load rounds per lane.  Larger
// steps keep a kernel each, which spreads their edges over the whole chip.
// Measured on MI355X against 64 MiB: reduce-scatters 1-3% faster; all-gathers
// of 4 KiB chunks 5-7% faster (N = 64 and 128), N = 1000 with 256 B chunks
// 0.5% faster, others within 0.4%; 256 MiB gains nothing more.
// PAT_TREE_FUSE_BYTES / PAT_TREE_FUSE_VECS override.
int64_t tree_fuse_vecs() { return env_or("PAT_TREE_FUSE_VECS", 2048); }
int64_t tree_fuse_bytes() { return env_or("PAT_TREE_FUSE_BYTES", int64_t(128) << 20); }

// Launch-level steps [*s0, *s1) that run as one fused launch, for a plan whose
// chunk-pieces hold V vectors; empty when nothing is fused.  The candidates
// are the steps whose slot entries each serve one tree: the top part (the
// first t steps of the all-gather order, the last t of the reduce-scatter's),
// and the whole schedule when the sub-trees span M <= 4.  There a linear-part
// node at position p keeps its chunk at index p / 4 of its distance's slot,
// which only p = 4 idx + 2 uses (distance 2), and leaves keep nothing; from
// M = 8 on, positions 8 idx + 2 and 8 idx + 6 share a distance-2 entry.  AUTO
// keeps the narrow far end (the reduce-scatter's last steps, the
// all-gather's first: chunks per rank grow toward the near end).
void fused_range(const pat::PlanDesc& d, int64_t V, int fusion, int* s0, int* s1, int64_t* tile_vecs) {
  *s0 = *s1 = 0;
  *tile_vecs = std::max<int64_t>(1, std::min<int64_t>(V, tree_tile_vecs(d.N, V)));
  if (fusion == PAT_FUSION_OFF || d.pieces != 1 || d.sched.list) return;  // list schedules share slots across trees
  const int ns = (int)d.exec.size(), t = d.sched.t;
  const bool whole = d.sched.M <= 4;
  int lo = whole || d.coll == 0 ? 0 : ns - t, hi = whole || d.coll == 1 ? ns : t;
  if (fusion == PAT_FUSION_AUTO) {
    const int64_t cap = tree_fuse_vecs(), cap_bytes = tree_fuse_bytes();
    // bytes a step moves: about three chunk transfers per edge
    auto narrow = [&](int s) {
      const int64_t k = d.exec[s].k;
      return k * *tile_vecs <= cap && 3 * int64_t(d.N) * k * d.count * d.esize_in <= cap_bytes;
    };
    if (d.coll == 1)
      while (lo < hi && !narrow(lo)) ++lo;
    else
      while (hi > lo && !narrow(hi - 1)) --hi;
  }
  if (hi - lo >= 2) {
    *s0 = lo;
    *s1 = hi;
  }
}

uint32_t timeout_us_now() { return g_timeout_us ? g_timeout_us : kDefaultTimeoutUs; }

// Persistent grid: at most this many workgroups per compute unit (0: as many
// as the occupancy calculator allows).  The work-queue kernel needs no
// co-residency, so this is a tuning knob, not a safety margin.  Each
// workgroup pays a device-scope release and acquire per step, so small steps
// run best on few workgroups and large ones on a full chip (measured on
// MI355X: 2 per CU below 128 MiB per step, 4 below 2 GiB, then all).
// PAT_PERSISTENT_BLOCKS_PER_CU overrides.
int blocks_per_cu_cap(double bytes_per_step) {
  if (const char* e = std::getenv("PAT_PERSISTENT_BLOCKS_PER_CU")) return std::max(0, std::atoi(e));
  if (bytes_per_step < 128.0 * (1 << 20)) return 2;
  if (bytes_per_step < 2048.0 * (1 << 20)) return 4;
  return 0;
}

// Loads and stores stream (nontemporal) when an operation moves at least this
// many bytes; smaller operations keep their data in the 256 MB Infinity Cache
// between steps (measured on MI355X: plain accesses are 6-17% faster below,
// streaming ones 8-12% faster far above).  PAT_STREAMING=0/1 overrides.
constexpr double kStreamingBytes = 1e9;

// Work-item order of the step kernels: each XCD takes runs of this many
// consecutive work items (0: a contiguous eighth of the step).  Measured on
// MI355X against the plain order (runs of 1): all-gather steps, which write
// up to two bytes per byte read, run up to 24% faster with a contiguous
// eighth per XCD; reduce-scatter steps 1-7% faster with runs of 32 (16-32
// are alike).  PAT_XCD_GRAIN overrides (a count of items; tuning).
int64_t xcd_run_for(int coll) {
  if (const char* e = std::getenv("PAT_XCD_GRAIN")) return std::max(0LL, std::atoll(e));
  return coll == 0 ? 0 : 32;
}

int64_t xcd_grain(int64_t run) { return run > 0 ? run : (int64_t(1) << 40); }

bool streaming_for(double alg_bytes) {
  if (const char* e = std::getenv("PAT_STREAMING")) return e[0] == '1';
  return alg_bytes >= kStreamingBytes;
}

int elem_size(pat_dtype_t t) { return t == PAT_BFLOAT16 ? 2 : 4; }

size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// Bytes between consecutive slot entries (and root accumulators) of a rank.
// Entries of 256 bytes or more start on 256-byte boundaries.  Smaller ones are
// packed at their own size: a multiple of 16 whenever the 128-bit path can
// run, of the element size otherwise.  Padding them to 256 bytes would make
// the intermediate memory of tiny chunks up to 64 times the data it holds.
size_t entry_stride(size_t bytes) { return bytes >= 256 ? round_up(bytes, 256) : bytes; }

#define HIP_TRY(expr)                                 \
  do {                                                \
    hipError_t e_ = (expr);                           \
    if (e_ != hipSuccess) {                           \
      g_last_hip.store((int)e_);                      \
      return PAT_ERR_HIP;                             \
    }                                                 \
  } while (0)

// The host-side part of a plan: schedule tables per path and the constants
// derived from them.  Building it allocates only ordinary host memory.
struct HostPlan {
  pat::PlanDesc desc;
  // Launch-level steps per path: [0] element-wide, [1] 128-bit vectors at
  // 16-byte-aligned addresses, [2] relaxed 128-bit vectors (element-aligned
  // addresses, a partial last vector per piece).  A path is empty where the
  // plan's sizes rule it out.
  bool has_path[3] = {true, false, false};
  std::vector<pat::DevStep> steps[3];
  bool streaming = true;
  int64_t xcd_run = 1;     // step kernels: work items per XCD run (0: a contiguous eighth)
  double alg_bytes = 0.0;  // algorithmic bytes of one operation
  int64_t slot_chunk_stride = 0, slot_rank_stride = 0, rootacc_stride = 0;
  int64_t slot_half_bytes = 0, root_half_bytes = 0;  // pipelined pieces: offsets of the second halves
};

struct Plan {
  HostPlan h;
  int device = 0;
  pat::DevEntry* d_entries = nullptr;
  pat::DevStep* d_steps[3] = {nullptr, nullptr, nullptr};
  const void** d_send = nullptr;
  void** d_recv = nullptr;
  char* d_slots = nullptr;
  char* d_rootacc = nullptr;
  unsigned* d_sync = nullptr;  // persistent-kernel counters: [2] status, work queue from [4]
  size_t sync_words = 0;
  std::vector<const void*> h_send;
  std::vector<void*> h_recv;
  void** pinned = nullptr;  // 2N pointers staged for upload
  hipEvent_t upload_done = nullptr;
  bool upload_pending = false;
  // Captured graphs by [vec][own_copy] and fused step range (s0, s1): a
  // change of the fusion setting selects or captures its own graph.
  std::map<std::tuple<int, int, int, int>, hipGraphExec_t> graphs;
  int capacity[pat::kNumVariants][2] = {};
  int cus = 0;
  int64_t clock_khz = 0;
  size_t bytes = 0;          // device memory held (slots, accumulators, tables)
  hipEvent_t done = nullptr;  // recorded after the plan's last operation
  bool used = false;
  uint64_t last_use = 0;     // LRU stamp
  // Step clock of fused launches (PAT_STEP_CLOCK=1 when the plan was made;
  // stream mode): the last fused launch's per-workgroup stamps.
  bool step_clock = false;
  uint64_t* d_stamps = nullptr;
  size_t stamps_cap = 0;      // entries
  int stamp_wgs = 0, stamps_per_wg = 0;
  // Dataflow execution (made on first use): every step tiled, per path; the
  // dependency table; per (rank, buffer) counters of completed tiles.
  bool df_ready = false;
  std::vector<pat::DevStep> df_steps[3];
  pat::DevStep* d_df_steps[3] = {nullptr, nullptr, nullptr};
  pat::DevDep* d_deps = nullptr;
  unsigned* d_counters = nullptr;

  ~Plan() {
    for (auto& kv : graphs)
      if (kv.second) (void)hipGraphExecDestroy(kv.second);
    if (done) (void)hipEventDestroy(done);
    if (upload_done) (void)hipEventDestroy(upload_done);
    if (pinned) (void)hipHostFree(pinned);
    (void)hipFree(d_entries);
    for (auto* p : d_steps) (void)hipFree(p);
    (void)hipFree(d_send);
    (void)hipFree(d_recv);
    (void)hipFree(d_slots);
    (void)hipFree(d_rootacc);
    (void)hipFree(d_sync);
    (void)hipFree(d_stamps);
    for (auto* p : d_df_steps) (void)hipFree(p);
    (void)hipFree(d_deps);
    (void)hipFree(d_counters);
  }
};

// coll, N, count, dtype, budget, linear order, device, aggregation
using PlanKey = std::tuple<int, int, int64_t, int, size_t, int, int, int>;
std::map<PlanKey, std::unique_ptr<Plan>> g_plans;
uint64_t g_tick = 0;

// Device memory the cached plans of one device may hold before the least
// recently used ones are released (PAT_PLAN_CACHE_BYTES; default 32 GiB).  A
// single plan larger than this is still allowed.
size_t cache_cap() {
  if (const char* e = std::getenv("PAT_PLAN_CACHE_BYTES")) {
    const long long v = std::atoll(e);
    if (v > 0) return size_t(v);
  }
  return size_t(32) << 30;
}

// Release least recently used plans of `device` until `need` more bytes fit
// under the cap (need == SIZE_MAX: release them all).  A plan's buffers are
// freed only after its last operation has finished on its stream.
void make_room(int device, size_t need) {
  for (;;) {
    size_t held = 0;
    auto victim = g_plans.end();
    for (auto it = g_plans.begin(); it != g_plans.end(); ++it) {
      if (it->second->device != device) continue;
      held += it->second->bytes;
      if (victim == g_plans.end() || it->second->last_use < victim->second->last_use) victim = it;
    }
    if (victim == g_plans.end()) return;
    if (need != SIZE_MAX && held + need <= cache_cap()) return;
    if (victim->second->used) (void)hipEventSynchronize(victim->second->done);
    g_plans.erase(victim);
  }
}

// Launch-level steps for one vector width: every schedule step of every piece.
// Chunk-pieces of at least `pack_tile` vectors are split into tiled work items
// of `tile` vectors (the last one ragged), smaller ones packed `pack_tile`
// vectors per work item.  `partial` (relaxed variants): a piece may end in a
// partial vector, but must hold one whole vector; the partial vector is the
// piece's last vector, or, with `items`, each edge's takes one lane of work
// items appended to the step.  Otherwise every piece must be whole vectors.
// False when the sizes rule the width out.  With out == nullptr, only that
// check (in O(1)).
bool build_steps(const pat::PlanDesc& d, int in_bytes, int tile, int pack_tile, bool partial, bool items,
                 std::vector<pat::DevStep>* out) {
  const int64_t per_vec = in_bytes / d.esize_in;  // elements per vector
  if (per_vec < 1) return false;
  if (!out) {
    // Only whether the width is possible: every piece but the last has the
    // first one's length, so those two decide.
    for (int piece : {0, d.pieces - 1}) {
      const int64_t len = std::min<int64_t>(d.piece_elems, d.count - int64_t(piece) * d.piece_elems);
      if (partial ? len < per_vec : (len * d.esize_in) % in_bytes != 0) return false;
    }
    return true;
  }
  out->clear();
  for (int piece = 0; piece < d.pieces; ++piece) {
    const int64_t e0 = int64_t(piece) * d.piece_elems;
    const int64_t len = std::min<int64_t>(d.piece_elems, d.count - e0);
    int64_t V = 0, back = 0;
    if (partial) {
      if (len < per_vec) return false;
      V = (len + per_vec - 1) / per_vec;
      back = V * per_vec - len;
      if (items && back) --V;
    } else {
      const int64_t bytes = len * d.esize_in;
      if (bytes % in_bytes) return false;
      V = bytes / in_bytes;
    }
    for (size_t j = 0; j < d.exec.size(); ++j) {
      const auto& st = d.exec[j];
      pat::DevStep ds{};
      ds.d = st.d;
      ds.k = st.k;
      ds.entry0 = st.first;
      ds.first = j == 0 ? 1 : 0;
      ds.half = d.pipelined ? piece % 2 : 0;
      ds.back = (int16_t)back;
      ds.e0 = e0;
      ds.V = V;
      const int64_t edges = int64_t(d.N) * st.k;
      if (V >= pack_tile) {
        ds.tiles_per_edge = (V + tile - 1) / tile;
        ds.items = edges * ds.tiles_per_edge;
      } else {
        ds.tiles_per_edge = 0;
        ds.items = (edges * V + pack_tile - 1) / pack_tile;
      }
      if (items && back) ds.items += (edges + pat::kThreads - 1) / pat::kThreads;  // partial vectors, one per lane
      out->push_back(ds);
    }
  }
  return true;
}

// Kernel variant of a path (0 element-wide, 1 aligned vectors, 2 relaxed vectors).
pat::Variant variant_for(int coll, pat_dtype_t dt, int path) {
  static const pat::Variant ag[3][3] = {{pat::kAgS4, pat::kAgVec, pat::kAgVecU},   // int32
                                        {pat::kAgS4, pat::kAgVec, pat::kAgVecU},   // float32
                                        {pat::kAgS2, pat::kAgVec, pat::kAgVecU}};  // bfloat16
  static const pat::Variant rs[3][3] = {{pat::kRsI32S, pat::kRsI32Vec, pat::kRsI32VecU},
                                        {pat::kRsF32S, pat::kRsF32Vec, pat::kRsF32VecU},
                                        {pat::kRsB16S, pat::kRsB16Vec, pat::kRsB16VecU}};
  const int t = dt == PAT_INT32 ? 0 : dt == PAT_FLOAT32 ? 1 : 2;
  return coll == 0 ? ag[t][path] : rs[t][path];
}

// The path a plan's 16-byte-aligned buffers take: aligned vectors when every
// piece is whole vectors, else relaxed vectors when every piece holds one,
// else element-wide.
int aligned_path(const bool (&has)[3]) { return has[1] ? 1 : has[2] ? 2 : 0; }

// Schedule tables and slot layout of a plan (host memory only).
pat_status_t make_host_plan(int coll, int N, int64_t count, pat_dtype_t dt, size_t budget, int order, int agg,
                            HostPlan* h) {
  if (!pat::make_plan_desc(coll, N, count, (int)dt, budget, order, &h->desc, agg, pipeline_now()))
    return PAT_ERR_INVALID_ARGUMENT;
  const pat::PlanDesc& d = h->desc;
  for (int path = 0; path < 3; ++path) {
    const pat::Variant v = variant_for(coll, dt, path);
    h->has_path[path] = build_steps(d, pat::variant_in_bytes(v), pat::variant_tile(v), pat::variant_pack_tile(v),
                                    path == 2 && pat::variant_partial(v), pat::variant_partial_items(v),
                                    &h->steps[path]);
  }
  if (!h->has_path[0]) return PAT_ERR_INTERNAL;
  h->streaming = streaming_for(d.alg_bytes);
  h->xcd_run = xcd_run_for(coll);
  h->alg_bytes = d.alg_bytes;
  h->slot_chunk_stride = (int64_t)entry_stride(size_t(d.piece_elems) * d.esize_slot);
  h->slot_rank_stride = h->slot_chunk_stride * d.slots.entries;
  h->rootacc_stride = (coll == 1 && dt == PAT_BFLOAT16) ? (int64_t)entry_stride(size_t(d.piece_elems) * 4) : 0;
  if (d.pipelined) {  // two halves per rank: [half 0 | half 1]
    h->slot_half_bytes = h->slot_rank_stride;
    h->slot_rank_stride *= 2;
    h->root_half_bytes = h->rootacc_stride;
    h->rootacc_stride *= 2;
  }
  return PAT_OK;
}

pat_status_t create_plan(int coll, int N, int64_t count, pat_dtype_t dt, size_t budget, int order, int agg,
                         int device, Plan** out) {
  auto p = std::make_unique<Plan>();
  const pat_status_t hs = make_host_plan(coll, N, count, dt, budget, order, agg, &p->h);
  if (hs != PAT_OK) return hs;
  const HostPlan& h = p->h;
  const pat::PlanDesc& d = h.desc;
  p->device = device;
  p->bytes = size_t(h.slot_rank_stride + h.rootacc_stride) * N + d.entries.size() * sizeof(pat::DevEntry) +
             (h.steps[0].size() + h.steps[1].size() + h.steps[2].size()) * sizeof(pat::DevStep) +
             2 * N * sizeof(void*) + pat::queue_words(h.steps[0].size()) * sizeof(unsigned);
  make_room(device, p->bytes);

  // On an allocation failure, release every other cached plan of this device
  // and try once more.
  auto alloc = [device](void** ptr, size_t bytes) -> pat_status_t {
    if (bytes == 0) return PAT_OK;
    hipError_t e = hipMalloc(ptr, bytes);
    if (e == hipErrorOutOfMemory) {
      (void)hipGetLastError();
      make_room(device, SIZE_MAX);
      e = hipMalloc(ptr, bytes);
    }
    if (e == hipErrorOutOfMemory) {
      (void)hipGetLastError();
      return PAT_ERR_OUT_OF_MEMORY;
    }
    if (e != hipSuccess) {
      g_last_hip.store((int)e);
      return PAT_ERR_HIP;
    }
    return PAT_OK;
  };
  pat_status_t s;
  if ((s = alloc((void**)&p->d_entries, d.entries.size() * sizeof(pat::DevEntry))) != PAT_OK) return s;
  for (int v = 0; v < 3; ++v)
    if ((s = alloc((void**)&p->d_steps[v], h.steps[v].size() * sizeof(pat::DevStep))) != PAT_OK) return s;
  if ((s = alloc((void**)&p->d_send, N * sizeof(void*))) != PAT_OK) return s;
  if ((s = alloc((void**)&p->d_recv, N * sizeof(void*))) != PAT_OK) return s;
  if ((s = alloc((void**)&p->d_slots, size_t(h.slot_rank_stride) * N)) != PAT_OK) return s;
  if ((s = alloc((void**)&p->d_rootacc, size_t(h.rootacc_stride) * N)) != PAT_OK) return s;
  p->sync_words = pat::queue_words(h.steps[0].size());  // every path has the same steps
  if ((s = alloc((void**)&p->d_sync, p->sync_words * sizeof(unsigned))) != PAT_OK) return s;
  HIP_TRY(hipMemset(p->d_sync, 0, p->sync_words * sizeof(unsigned)));
  if (const char* e = std::getenv("PAT_POISON_SLOTS")) {
    if (e[0] == '1') {
      if (p->d_slots) HIP_TRY(hipMemset(p->d_slots, 0xFF, size_t(h.slot_rank_stride) * N));
      if (p->d_rootacc) HIP_TRY(hipMemset(p->d_rootacc, 0xFF, size_t(h.rootacc_stride) * N));
    }
  }
  if (!d.entries.empty())
    HIP_TRY(hipMemcpy(p->d_entries, d.entries.data(), d.entries.size() * sizeof(pat::DevEntry),
                      hipMemcpyHostToDevice));
  for (int v = 0; v < 3; ++v)
    if (!h.steps[v].empty())
      HIP_TRY(hipMemcpy(p->d_steps[v], h.steps[v].data(), h.steps[v].size() * sizeof(pat::DevStep),
                        hipMemcpyHostToDevice));
  HIP_TRY(hipHostMalloc((void**)&p->pinned, 2 * size_t(N) * sizeof(void*), hipHostMallocDefault));
  HIP_TRY(hipEventCreateWithFlags(&p->upload_done, hipEventDisableTiming));
  HIP_TRY(hipEventCreateWithFlags(&p->done, hipEventDisableTiming));
  if (const char* e = std::getenv("PAT_STEP_CLOCK")) p->step_clock = e[0] == '1';
  if (const char* e = std::getenv("PAT_DEBUG")) {
    if (e[0] == '1') {
      std::fprintf(stderr,
                   "[pat] plan coll=%d N=%d count=%lld dtype=%d L=%d t=%d T=%d steps=%zu pieces=%d "
                   "max_k=%d slot_entries/rank=%d slot_bytes=%lld alg_bytes=%.0f paths=%d%d%d streaming=%d\n",
                   coll, N, (long long)count, (int)dt, d.sched.L, d.sched.t, d.sched.T, d.exec.size(),
                   d.pieces, d.max_k, d.slots.entries, (long long)(h.slot_rank_stride * N), d.alg_bytes,
                   (int)h.has_path[0], (int)h.has_path[1], (int)h.has_path[2], (int)h.streaming);
    }
  }
  *out = p.get();
  g_plans[PlanKey(coll, N, count, (int)dt, budget, order, device, agg)] = std::move(p);
  return PAT_OK;
}

// Receive buffers may not overlap anything except the in-place alias of the
// same rank (all-gather: send inside recv at chunk r; reduce-scatter: recv
// inside send at chunk r).  Send buffers may overlap each other (read-only).
bool overlaps_ok(int coll, const void* const* send, void* const* recv, int N, size_t send_bytes,
                 size_t recv_bytes, size_t chunk_bytes) {
  struct Iv {
    uintptr_t lo, hi;
    int rank;
  };
  std::vector<Iv> rv(N);
  for (int r = 0; r < N; ++r) {
    const uintptr_t lo = (uintptr_t)recv[r];
    rv[r] = {lo, lo + recv_bytes, r};
  }
  std::sort(rv.begin(), rv.end(), [](const Iv& a, const Iv& b) { return a.lo < b.lo; });
  for (int i = 1; i < N; ++i)
    if (rv[i].lo < rv[i - 1].hi) return false;  // equal lengths: adjacent check suffices
  for (int r = 0; r < N; ++r) {
    const uintptr_t lo = (uintptr_t)send[r], hi = lo + send_bytes;
    auto it = std::upper_bound(rv.begin(), rv.end(), lo, [](uintptr_t v, const Iv& a) { return v < a.hi; });
    for (; it != rv.end() && it->lo < hi; ++it) {
      if (it->rank != r) return false;
      const uintptr_t q = (uintptr_t)recv[r];
      const bool alias = coll == 0 ? (lo == q + uintptr_t(r) * chunk_bytes)
                                   : (q == lo + uintptr_t(r) * chunk_bytes);
      if (!alias) return false;
    }
  }
  return true;
}

// The pointer set a thread last passed the per-pointer checks with, and what
// they found.  A caller that reuses its buffers passes the same set call after
// call; comparing it costs O(N) instead of the checks' O(N log N).
struct CheckedPointers {
  int coll = -1, N = 0, dt = -1;
  size_t count = 0;
  std::vector<const void*> send;
  std::vector<void*> recv;
  bool vec = false;
};
thread_local CheckedPointers t_checked;

// Dataflow execution: work items per step for chunks of one tile or more.
constexpr int64_t kDataflowItems = 4096;

// Largest counter array dataflow execution allocates (N x (slot entries + 1)
// words); beyond it the mode is refused with PAT_ERR_UNSUPPORTED.
constexpr size_t kMaxDataflowCounters = size_t(256) << 20;

// The dataflow tables of a plan, made on its first dataflow operation.
pat_status_t ensure_dataflow(Plan* p, int coll, pat_dtype_t dt) {
  if (p->df_ready) return PAT_OK;
  const HostPlan& h = p->h;
  const pat::PlanDesc& d = h.desc;
  const size_t stride = size_t(d.slots.entries) + 1;
  if (stride * d.N * sizeof(unsigned) > kMaxDataflowCounters) return PAT_ERR_UNSUPPORTED;
  std::vector<pat::DevDep> deps;
  if (!pat::dataflow_deps(d, &deps)) return PAT_ERR_INTERNAL;
  for (int path = 0; path < 3; ++path) {
    if (!h.has_path[path]) continue;
    const pat::Variant v = variant_for(coll, dt, path);
    const int pack = pat::variant_pack_tile(v);
    if (!build_steps(d, pat::variant_in_bytes(v), pat::variant_tile(v), pack, path == 2 && pat::variant_partial(v),
                     pat::variant_partial_items(v), &p->df_steps[path]))
      return PAT_ERR_INTERNAL;
    // Work items: whole edges, about four packed work items' worth of vectors
    // and at most one edge per lane, for chunks under one tile; else runs of
    // tiles of one edge, about kDataflowItems items per step.
    for (auto& st : p->df_steps[path]) {
      const int64_t edges = int64_t(d.N) * st.k;
      if (st.tiles_per_edge == 0) {
        st.df_edges = (int32_t)std::max<int64_t>(1, std::min<int64_t>(pat::kThreads, 4 * pack / std::max<int64_t>(1, st.V)));
        st.df_tiles = 1;
        st.items = (edges + st.df_edges - 1) / st.df_edges;
      } else {
        st.df_edges = 0;
        st.df_tiles = (int32_t)std::max<int64_t>(
            1, std::min<int64_t>(st.tiles_per_edge, (edges * st.tiles_per_edge + kDataflowItems - 1) / kDataflowItems));
        st.items = edges * ((st.tiles_per_edge + st.df_tiles - 1) / st.df_tiles);
      }
    }
  }
  HIP_TRY(hipMalloc((void**)&p->d_deps, std::max<size_t>(1, deps.size()) * sizeof(pat::DevDep)));
  if (!deps.empty())
    HIP_TRY(hipMemcpy(p->d_deps, deps.data(), deps.size() * sizeof(pat::DevDep), hipMemcpyHostToDevice));
  HIP_TRY(hipMalloc((void**)&p->d_counters, stride * d.N * sizeof(unsigned)));
  HIP_TRY(hipMemset(p->d_counters, 0, stride * d.N * sizeof(unsigned)));
  for (int path = 0; path < 3; ++path) {
    if (p->df_steps[path].empty()) continue;
    HIP_TRY(hipMalloc((void**)&p->d_df_steps[path], p->df_steps[path].size() * sizeof(pat::DevStep)));
    HIP_TRY(hipMemcpy(p->d_df_steps[path], p->df_steps[path].data(),
                      p->df_steps[path].size() * sizeof(pat::DevStep), hipMemcpyHostToDevice));
  }
  p->bytes += std::max<size_t>(1, deps.size()) * sizeof(pat::DevDep) + stride * d.N * sizeof(unsigned);
  p->df_ready = true;
  return PAT_OK;
}

// Argument checks shared by every entry point.  PAT_OK with *nothing set
// when count == 0 (no pointer is examined then); *vec tells whether every
// pointer is 16-byte aligned.
pat_status_t check_args(int coll, const void* const* send, void* const* recv, size_t count, pat_dtype_t dt,
                        int N, bool* vec, bool* nothing) {
  *nothing = false;
  if (N < 1 || N > kMaxRanks || send == nullptr || recv == nullptr) return PAT_ERR_INVALID_ARGUMENT;
  if (dt != PAT_INT32 && dt != PAT_FLOAT32 && dt != PAT_BFLOAT16) return PAT_ERR_UNSUPPORTED;
  const size_t es = (size_t)elem_size(dt);
  if (count > (size_t(1) << 40) / es || (unsigned __int128)count * es * N > ((unsigned __int128)1 << 62))
    return PAT_ERR_INVALID_ARGUMENT;
  if (count == 0) {
    *nothing = true;
    return PAT_OK;
  }
  const size_t chunk = count * es;
  CheckedPointers& ck = t_checked;
  const bool checked = ck.coll == coll && ck.N == N && ck.dt == (int)dt && ck.count == count &&
                       !std::memcmp(ck.send.data(), send, N * sizeof(void*)) &&
                       !std::memcmp(ck.recv.data(), recv, N * sizeof(void*));
  if (checked) {
    *vec = ck.vec;
    return PAT_OK;
  }
  ck.coll = -1;  // invalid until this set passes
  bool v = true;
  for (int r = 0; r < N; ++r) {
    if (!send[r] || !recv[r]) return PAT_ERR_INVALID_ARGUMENT;
    if (((uintptr_t)send[r] | (uintptr_t)recv[r]) % es) return PAT_ERR_INVALID_ARGUMENT;
    if (((uintptr_t)send[r] | (uintptr_t)recv[r]) % 16) v = false;
  }
  const size_t send_bytes = coll == 0 ? chunk : chunk * N;
  const size_t recv_bytes = coll == 0 ? chunk * N : chunk;
  if (!overlaps_ok(coll, send, recv, N, send_bytes, recv_bytes, chunk)) return PAT_ERR_INVALID_ARGUMENT;
  ck.send.assign(send, send + N);
  ck.recv.assign(recv, recv + N);
  ck.N = N;
  ck.dt = (int)dt;
  ck.count = count;
  ck.vec = v;
  ck.coll = coll;
  *vec = v;
  return PAT_OK;
}

// The path a call takes: 16-byte-aligned buffers take the plan's best path;
// others the relaxed vectors where the sizes allow, else element-wide kernels.
int path_for(const HostPlan& h, bool vec) { return vec ? aligned_path(h.has_path) : h.has_path[2] ? 2 : 0; }

// Whether an all-gather copies each rank's own chunk (not in place).
bool needs_own_copy(int coll, const void* const* send, void* const* recv, int N, size_t chunk) {
  if (coll != 0) return false;
  for (int r = 0; r < N; ++r)
    if ((const char*)send[r] != (const char*)recv[r] + size_t(r) * chunk) return true;
  return false;
}

// Kernel context of a call whose tables and buffers sit at the given device
// addresses.
pat::KCtx make_ctx(const HostPlan& h, int vi, const void* const* d_send, void* const* d_recv, char* slots,
                   char* rootacc, const pat::DevEntry* entries, const pat::DevStep* steps, size_t count, int N,
                   bool own_copy) {
  pat::KCtx cx{};
  cx.send = d_send;
  cx.recv = d_recv;
  cx.slots = slots;
  cx.rootacc = rootacc;
  cx.entries = entries;
  cx.steps = steps;
  cx.count = (int64_t)count;
  cx.slot_chunk_stride = h.slot_chunk_stride;
  cx.slot_rank_stride = h.slot_rank_stride;
  cx.rootacc_stride = h.rootacc_stride;
  cx.slot_half_bytes = h.slot_half_bytes;
  cx.root_half_bytes = h.root_half_bytes;
  cx.esize = (int64_t)h.desc.esize_in;
  cx.N = N;
  cx.nsteps = (int32_t)h.steps[vi].size();
  cx.own_copy = own_copy ? 1 : 0;
  return cx;
}

// The fused range of a call (stream and graph modes).
// The fused launch of a plan, with the steps whose edges it caches: the
// longest run of its narrow end (the all-gather's first steps, the
// reduce-scatter's last) holding at most pat::kTreeCacheEdges entries in
// pat::kTreeCacheSteps steps, whose entries follow each other in the table.
// PAT_TREE_EDGE_CACHE=0 turns the cache off.  (Leaving the all-gather's first
// step out, to fill during it, measured 0.3 us slower on MI355X.)
pat::TreeRange tree_range(const HostPlan& h, int vi) {
  pat::TreeRange tr{};
  const auto& steps = h.steps[vi];
  fused_range(h.desc, steps.empty() ? 0 : steps[0].V, fusion_now(), &tr.s0, &tr.s1, &tr.tile_vecs);
  if (tr.s1 <= tr.s0) return tr;
  tr.tiles = (steps[0].V + tr.tile_vecs - 1) / tr.tile_vecs;
  const char* e = std::getenv("PAT_TREE_EDGE_CACHE");
  if (e && std::atoi(e) == 0) return tr;
  auto fits = [&](int s) { return tr.c1 - tr.c0 < pat::kTreeCacheSteps && tr.cn + steps[s].k <= pat::kTreeCacheEdges; };
  tr.c0 = tr.c1 = h.desc.coll == 0 ? tr.s0 : tr.s1;
  if (h.desc.coll == 0)
    while (tr.c1 < tr.s1 && fits(tr.c1)) tr.cn += steps[tr.c1++].k;
  else
    while (tr.c0 > tr.s0 && fits(tr.c0 - 1)) tr.cn += steps[--tr.c0].k;
  if (tr.cn == 0) {
    tr.c0 = tr.c1 = 0;
    return tr;
  }
  tr.ce0 = steps[tr.c0].entry0;
  for (int s = tr.c0, end = 0; s < tr.c1; ++s) {
    if (steps[s].entry0 != tr.ce0 + end) {  // not one run of the table: no cache
      tr.c0 = tr.c1 = tr.cn = tr.ce0 = 0;
      return tr;
    }
    end += steps[s].k;
    tr.cend[s - tr.c0] = (int16_t)end;
  }
  return tr;
}

// Launch tracing (pat_trace_start / pat_trace_read): a HIP event pair around
// each kernel launch of stream-mode operations, with the launch's algorithmic
// bytes, until `max` launches are recorded.  Guarded by g_mu.
struct Trace {
  bool armed = false;
  int max = 0, used = 0;
  std::vector<hipEvent_t> ev;  // [2 * max]: before / after launch j
  std::vector<double> bytes;   // [max]
  std::vector<int32_t> kind;   // [max]: 0 step kernel, 1 fused range
  std::vector<int32_t> step;   // [max]: launch-level step (the first of a fused range)

  void clear() {
    for (hipEvent_t e : ev)
      if (e) (void)hipEventDestroy(e);
    ev.clear();
    bytes.clear();
    kind.clear();
    step.clear();
    armed = false;
    max = used = 0;
  }
};
Trace g_trace;

// Algorithmic bytes of launch-level step s (a schedule step of one piece).
double launch_bytes(const HostPlan& h, int vi, int s) {
  const pat::PlanDesc& d = h.desc;
  const int nexec = (int)d.exec.size();
  const int64_t e0 = h.steps[vi][s].e0;
  return pat::step_bytes(d, s % nexec, std::min<int64_t>(d.piece_elems, d.count - e0));
}

// Stream-mode launch sequence: one kernel per step, except that the fused
// range (steps whose slot entries each serve one tree) runs as one launch.
// With a trace, each launch is bracketed by its event pair on `q`.
hipError_t enqueue_stream(const HostPlan& h, int coll, pat_dtype_t dt, int vi, const pat::KCtx& cx,
                          const pat::TreeRange& tr, hipStream_t q, Trace* trace = nullptr) {
  const pat::Variant var = variant_for(coll, dt, vi);
  const auto& steps = h.steps[vi];
  if (h.desc.pipelined) {
    // Piece p starts at launch (p / 2) * S + p % 2 (S steps per piece): two
    // pieces in flight, one step apart, in the two slot halves; a piece
    // starts its half only once the piece two before it has finished.
    const int S = (int)h.desc.exec.size(), P = h.desc.pieces;
    const int launches = ((P - 1) / 2) * S + (P - 1) % 2 + S;
    for (int j = 0; j < launches; ++j) {
      int idx[2], n = 0;
      for (int p = 0; p < P && n < 2; ++p) {
        const int start = (p / 2) * S + p % 2;
        if (j >= start && j < start + S) idx[n++] = p * S + (j - start);
      }
      const bool traced = trace && trace->used < trace->max;
      if (traced) {
        const hipError_t e = hipEventRecord(trace->ev[2 * trace->used], q);
        if (e != hipSuccess) return e;
      }
      const hipError_t e =
          n == 2 ? pat::launch_step2(var, h.streaming, xcd_grain(h.xcd_run), cx, idx[0], steps[idx[0]], idx[1],
                                     steps[idx[1]], q)
                 : pat::launch_step(var, h.streaming, xcd_grain(h.xcd_run), cx, steps[idx[0]], q);
      if (e != hipSuccess) return e;
      if (traced) {
        const int t = trace->used;
        const hipError_t e2 = hipEventRecord(trace->ev[2 * t + 1], q);
        if (e2 != hipSuccess) return e2;
        trace->bytes[t] = launch_bytes(h, vi, idx[0]) + (n == 2 ? launch_bytes(h, vi, idx[1]) : 0.0);
        trace->kind[t] = 0;
        trace->step[t] = idx[0];
        trace->used = t + 1;
      }
    }
    return hipSuccess;
  }
  const bool fuse = tr.s1 > tr.s0;
  for (int s = 0; s < (int)steps.size(); ++s) {
    const bool traced = trace && trace->used < trace->max;
    if (traced) {
      const hipError_t e = hipEventRecord(trace->ev[2 * trace->used], q);
      if (e != hipSuccess) return e;
    }
    const int first = s;
    hipError_t e;
    if (fuse && s == tr.s0) {
      e = pat::launch_tree(var, h.streaming, cx, tr, q);
      s = tr.s1 - 1;
    } else {
      e = pat::launch_step(var, h.streaming, xcd_grain(h.xcd_run), cx, steps[s], q);
    }
    if (e != hipSuccess) return e;
    if (traced) {
      const int j = trace->used;
      e = hipEventRecord(trace->ev[2 * j + 1], q);
      if (e != hipSuccess) return e;
      double bytes = 0.0;
      for (int k = first; k <= s; ++k) bytes += launch_bytes(h, vi, k);
      trace->bytes[j] = bytes;
      trace->kind[j] = fuse && first == tr.s0 ? 1 : 0;
      trace->step[j] = first;
      trace->used = j + 1;
    }
  }
  return hipSuccess;
}

pat_status_t run(int coll, const void* const* send, void* const* recv, size_t count, pat_dtype_t dt, int N,
                 hipStream_t stream) {
  bool vec = false, nothing = false;
  const pat_status_t cs = check_args(coll, send, recv, count, dt, N, &vec, &nothing);
  if (cs != PAT_OK || nothing) return cs;
  const size_t chunk = count * (size_t)elem_size(dt);

  if (N == 1) {
    if (send[0] != recv[0])
      HIP_TRY(hipMemcpyAsync(recv[0], send[0], chunk, hipMemcpyDeviceToDevice, stream));
    return PAT_OK;
  }

  std::lock_guard<std::mutex> lock(g_mu);
  int device = 0;
  HIP_TRY(hipGetDevice(&device));
  const size_t budget = budget_now();
  const int order = order_now();
  const int agg = aggregation_now();
  Plan* plan = nullptr;
  auto it = g_plans.find(PlanKey(coll, N, (int64_t)count, (int)dt, budget, order, device, agg));
  if (it != g_plans.end()) {
    plan = it->second.get();
  } else {
    const pat_status_t s = create_plan(coll, N, (int64_t)count, dt, budget, order, agg, device, &plan);
    if (s != PAT_OK) return s;
  }
  const HostPlan& h = plan->h;
  const int vi = path_for(h, vec);
  const bool own_copy = needs_own_copy(coll, send, recv, N, chunk);

  // Pointer tables: upload only when they changed since the last call.  The
  // remembered set is replaced only once its upload is queued.
  const bool same = plan->h_send.size() == size_t(N) &&
                    !std::memcmp(plan->h_send.data(), send, N * sizeof(void*)) &&
                    !std::memcmp(plan->h_recv.data(), recv, N * sizeof(void*));
  if (!same) {
    if (plan->upload_pending) HIP_TRY(hipEventSynchronize(plan->upload_done));
    plan->h_send.clear();
    plan->h_recv.clear();
    std::memcpy(plan->pinned, send, N * sizeof(void*));
    std::memcpy(plan->pinned + N, recv, N * sizeof(void*));
    HIP_TRY(hipMemcpyAsync(plan->d_send, plan->pinned, N * sizeof(void*), hipMemcpyHostToDevice, stream));
    HIP_TRY(hipMemcpyAsync(plan->d_recv, plan->pinned + N, N * sizeof(void*), hipMemcpyHostToDevice, stream));
    HIP_TRY(hipEventRecord(plan->upload_done, stream));
    plan->upload_pending = true;
    plan->h_send.assign(send, send + N);
    plan->h_recv.assign(recv, recv + N);
  }

  pat::KCtx cx = make_ctx(h, vi, plan->d_send, plan->d_recv, plan->d_slots, plan->d_rootacc, plan->d_entries,
                          plan->d_steps[vi], count, N, own_copy);
  if (plan->clock_khz == 0) {
    int khz = 0, cus = 0;
    HIP_TRY(hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, device));
    HIP_TRY(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device));
    plan->clock_khz = khz > 0 ? khz : 100000;
    plan->cus = cus;
  }
  cx.timeout_ticks = (int64_t)timeout_us_now() * plan->clock_khz / 1000;
  cx.queue = plan->d_sync;
  cx.status = plan->d_sync + 2;

  const pat::Variant var = variant_for(coll, dt, vi);
  const auto& steps = h.steps[vi];
  const int mode = mode_now();
  if (mode == PAT_EXEC_DATAFLOW) {
    // The relaxed bf16 reduce-scatter gives partial vectors work items of
    // their own, spanning many edges: dataflow runs its element-wide twin.
    const int dvi = pat::variant_partial_items(var) ? 0 : vi;
    const pat::Variant dvar = variant_for(coll, dt, dvi);
    const pat_status_t ds = ensure_dataflow(plan, coll, dt);
    if (ds != PAT_OK) return ds;
    const bool nt = h.streaming;
    int& capacity = plan->capacity[dvar][nt ? 1 : 0];
    if (capacity == 0) HIP_TRY(pat::persistent_capacity(dvar, nt, &capacity));
    const auto& dsteps = plan->df_steps[dvi];
    const int nexec = (int)h.desc.exec.size();
    int64_t most = 1;
    for (const auto& st : dsteps) most = std::max(most, st.items);
    int64_t cap = capacity;
    const double per_step = h.alg_bytes / double(std::max<size_t>(1, dsteps.size()));
    if (const int per_cu = blocks_per_cu_cap(per_step)) cap = std::min<int64_t>(cap, int64_t(per_cu) * plan->cus);
    const int grid = (int)std::max<int64_t>(1, std::min<int64_t>(cap, most));  // any size is safe
    pat::KCtx dx = make_ctx(h, dvi, plan->d_send, plan->d_recv, plan->d_slots, plan->d_rootacc, plan->d_entries,
                            plan->d_df_steps[dvi], count, N, own_copy);
    dx.timeout_ticks = cx.timeout_ticks;
    dx.queue = cx.queue;
    dx.status = cx.status;
    dx.deps = plan->d_deps;
    dx.counters = plan->d_counters;
    dx.counter_stride = int64_t(h.desc.slots.entries) + 1;
    dx.nsteps = nexec;
    for (int piece = 0; piece < h.desc.pieces; ++piece) {
      dx.steps = plan->d_df_steps[dvi] + size_t(piece) * nexec;
      const bool small = dsteps[size_t(piece) * nexec].tiles_per_edge == 0;  // a piece's steps share V
      HIP_TRY(pat::launch_dataflow(dvar, nt, dx, small, grid, stream));
    }
  } else if (mode == PAT_EXEC_PERSISTENT) {
    const bool nt = h.streaming;
    int& capacity = plan->capacity[var][nt ? 1 : 0];
    if (capacity == 0) HIP_TRY(pat::persistent_capacity(var, nt, &capacity));
    int64_t most = 1;
    for (const auto& st : steps) most = std::max(most, st.items);
    int64_t cap = capacity;
    const double per_step = h.alg_bytes / double(std::max<size_t>(1, steps.size()));
    if (const int per_cu = blocks_per_cu_cap(per_step)) cap = std::min<int64_t>(cap, int64_t(per_cu) * plan->cus);
    const int grid = (int)std::max<int64_t>(1, std::min<int64_t>(cap, most));  // any size is safe
    if (const char* e = std::getenv("PAT_DEBUG"))
      if (e[0] == '1')
        std::fprintf(stderr, "[pat] persistent launch: capacity=%d cus=%d grid=%d steps=%d\n",
                     capacity, plan->cus, grid, cx.nsteps);
    HIP_TRY(pat::launch_persistent(var, nt, cx, grid, stream));
  } else {
    const pat::TreeRange tr = tree_range(h, vi);
    if (mode == PAT_EXEC_STREAM && plan->step_clock && tr.s1 > tr.s0) {
      const int wgs = N * (int)tr.tiles, per = tr.s1 - tr.s0 + 1;
      const size_t need = size_t(wgs) * per;
      if (plan->stamps_cap < need) {
        HIP_TRY(hipStreamSynchronize(stream));
        HIP_TRY(hipFree(plan->d_stamps));
        plan->d_stamps = nullptr;
        plan->stamps_cap = 0;
        HIP_TRY(hipMalloc((void**)&plan->d_stamps, need * sizeof(uint64_t)));
        plan->stamps_cap = need;
      }
      plan->stamp_wgs = wgs;
      plan->stamps_per_wg = per;
      cx.stamps = plan->d_stamps;
    }
    if (mode == PAT_EXEC_STREAM) {
      HIP_TRY(enqueue_stream(h, coll, dt, vi, cx, tr, stream, g_trace.armed ? &g_trace : nullptr));
    } else {
      hipGraphExec_t& exec = plan->graphs[std::make_tuple(vi, cx.own_copy, tr.s0, tr.s1)];
      if (!exec) {
        hipStream_t cs = nullptr;
        HIP_TRY(hipStreamCreateWithFlags(&cs, hipStreamNonBlocking));
        hipGraph_t g = nullptr;
        hipError_t e = hipStreamBeginCapture(cs, hipStreamCaptureModeThreadLocal);
        if (e == hipSuccess) e = enqueue_stream(h, coll, dt, vi, cx, tr, cs);
        const hipError_t e2 = hipStreamEndCapture(cs, &g);
        if (e == hipSuccess) e = e2;
        if (e == hipSuccess) e = hipGraphInstantiate(&exec, g, nullptr, nullptr, 0);
        if (g) (void)hipGraphDestroy(g);
        (void)hipStreamDestroy(cs);
        if (e != hipSuccess) {
          exec = nullptr;
          g_last_hip.store((int)e);
          return PAT_ERR_HIP;
        }
      }
      HIP_TRY(hipGraphLaunch(exec, stream));
    }
  }
  HIP_TRY(hipEventRecord(plan->done, stream));
  plan->used = true;
  plan->last_use = ++g_tick;
  return PAT_OK;
}

// ---------------------------------------------------------------------------
// The entry point that allocates nothing: everything the kernels need beyond
// the caller's buffers lives in the library's fixed per-device scratch array
// (noalloc.hip).  Per device, the host remembers which plan's tables and which
// pointer set the scratch holds, so that repeated calls only launch kernels.
// ---------------------------------------------------------------------------

struct ScratchState {
  bool have_plan = false;
  PlanKey key;
  HostPlan plan;
  int vi = -1;                     // path whose step table is in the scratch (-1: none)
  std::vector<const void*> send;   // pointer set in the scratch's tables
  std::vector<void*> recv;
  size_t off_entries = 0, off_steps = 0, off_send = 0, off_recv = 0, off_slots = 0, off_rootacc = 0, end = 0;
};
std::map<int, ScratchState> g_scratch;  // by device

size_t align256(size_t v) { return (v + 255) / 256 * 256; }

// Scratch layout of a plan: a reserved line, the entry table, one path's step
// table (sized for the longest path), the two pointer tables, the slots and
// the float32 root accumulators.  Returns the bytes it needs.
size_t scratch_layout(const HostPlan& h, int N, ScratchState* ss) {
  size_t o = 256;
  ss->off_entries = o;
  o = align256(o + h.desc.entries.size() * sizeof(pat::DevEntry));
  size_t most = 0;
  for (const auto& v : h.steps) most = std::max(most, v.size());
  ss->off_steps = o;
  o = align256(o + most * sizeof(pat::DevStep));
  ss->off_send = o;
  o = align256(o + size_t(N) * sizeof(void*));
  ss->off_recv = o;
  o = align256(o + size_t(N) * sizeof(void*));
  ss->off_slots = o;
  o = align256(o + size_t(h.slot_rank_stride) * N);
  ss->off_rootacc = o;
  o = align256(o + size_t(h.rootacc_stride) * N);
  ss->end = o;
  return o;
}

pat_status_t run_noalloc(int coll, const void* const* send, void* const* recv, size_t count, pat_dtype_t dt,
                         int N, hipStream_t stream) {
  bool vec = false, nothing = false;
  const pat_status_t cs = check_args(coll, send, recv, count, dt, N, &vec, &nothing);
  if (cs != PAT_OK || nothing) return cs;
  const size_t chunk = count * (size_t)elem_size(dt);
  if (N == 1) {
    if (send[0] != recv[0])
      HIP_TRY(hipMemcpyAsync(recv[0], send[0], chunk, hipMemcpyDeviceToDevice, stream));
    return PAT_OK;
  }

  std::lock_guard<std::mutex> lock(g_mu);
  int device = 0;
  HIP_TRY(hipGetDevice(&device));
  char* base = nullptr;
  HIP_TRY(pat::scratch_base(device, &base));  // this device's array (looked up once per device)
  ScratchState& ss = g_scratch[device];
  const PlanKey key(coll, N, (int64_t)count, (int)dt, budget_now(), order_now(), device, aggregation_now());
  if (!ss.have_plan || ss.key != key) {
    // A new plan: its tables must be uploaded before use.
    ss.have_plan = false;
    ss.vi = -1;
    ss.send.clear();
    ss.recv.clear();
    ss.plan = HostPlan();
    const pat_status_t s =
        make_host_plan(coll, N, (int64_t)count, dt, std::get<4>(key), std::get<5>(key), std::get<7>(key), &ss.plan);
    if (s != PAT_OK) return s;
    if (scratch_layout(ss.plan, N, &ss) > pat::scratch_bytes()) return PAT_ERR_TOO_LARGE;
    ss.key = key;
    ss.have_plan = true;
  }
  const HostPlan& h = ss.plan;
  const int vi = path_for(h, vec);
  if (ss.vi != vi) {
    ss.vi = -1;
    const auto& entries = h.desc.entries;
    if (!entries.empty())
      HIP_TRY(hipMemcpyAsync(base + ss.off_entries, entries.data(), entries.size() * sizeof(pat::DevEntry),
                             hipMemcpyHostToDevice, stream));
    HIP_TRY(hipMemcpyAsync(base + ss.off_steps, h.steps[vi].data(), h.steps[vi].size() * sizeof(pat::DevStep),
                           hipMemcpyHostToDevice, stream));
    ss.vi = vi;
  }
  const bool same = ss.send.size() == size_t(N) && !std::memcmp(ss.send.data(), send, N * sizeof(void*)) &&
                    !std::memcmp(ss.recv.data(), recv, N * sizeof(void*));
  if (!same) {
    ss.send.assign(send, send + N);
    ss.recv.assign(recv, recv + N);
    HIP_TRY(hipMemcpyAsync(base + ss.off_send, ss.send.data(), N * sizeof(void*), hipMemcpyHostToDevice, stream));
    HIP_TRY(hipMemcpyAsync(base + ss.off_recv, ss.recv.data(), N * sizeof(void*), hipMemcpyHostToDevice, stream));
  }
  const pat::KCtx cx = make_ctx(h, vi, (const void* const*)(base + ss.off_send), (void* const*)(base + ss.off_recv),
                                base + ss.off_slots, base + ss.off_rootacc,
                                (const pat::DevEntry*)(base + ss.off_entries),
                                (const pat::DevStep*)(base + ss.off_steps), count, N,
                                needs_own_copy(coll, send, recv, N, chunk));
  HIP_TRY(enqueue_stream(h, coll, dt, vi, cx, tree_range(h, vi), stream));
  return PAT_OK;
}

pat_status_t describe(int coll, int N, size_t count, pat_dtype_t dt, pat::PlanDesc* d) {
  if (coll != 0 && coll != 1) return PAT_ERR_INVALID_ARGUMENT;
  if (N < 1 || N > kMaxRanks) return PAT_ERR_INVALID_ARGUMENT;
  if (dt != PAT_INT32 && dt != PAT_FLOAT32 && dt != PAT_BFLOAT16) return PAT_ERR_UNSUPPORTED;
  if (count > (size_t(1) << 40)) return PAT_ERR_INVALID_ARGUMENT;
  size_t budget;
  int order, agg;
  {
    std::lock_guard<std::mutex> lock(g_mu);
    budget = budget_now();
    order = order_now();
    agg = aggregation_now();
  }
  if (!pat::make_plan_desc(coll, N, (int64_t)count, (int)dt, budget, order, d, agg, pipeline_now()))
    return PAT_ERR_INVALID_ARGUMENT;
  return PAT_OK;
}

}  // namespace

extern "C" {

pat_status_t pat_allgather(const void* const* sendbufs, void* const* recvbufs, size_t count, pat_dtype_t dtype,
                           int nranks, hipStream_t stream) {
  return run(0, sendbufs, recvbufs, count, dtype, nranks, stream);
}

pat_status_t pat_reducescatter(const void* const* sendbufs, void* const* recvbufs, size_t count,
                               pat_dtype_t dtype, pat_op_t op, int nranks, hipStream_t stream) {
  if (op != PAT_SUM) return PAT_ERR_UNSUPPORTED;
  return run(1, sendbufs, recvbufs, count, dtype, nranks, stream);
}

pat_status_t pat_reducescatter_noalloc(const void* const* sendbufs, void* const* recvbufs, size_t count,
                                       pat_dtype_t dtype, pat_op_t op, int nranks, hipStream_t stream) {
  if (op != PAT_SUM) return PAT_ERR_UNSUPPORTED;
  return run_noalloc(1, sendbufs, recvbufs, count, dtype, nranks, stream);
}

pat_status_t pat_set_buffer_bytes(size_t bytes_per_slot) {
  std::lock_guard<std::mutex> lock(g_mu);
  g_budget = bytes_per_slot;
  return PAT_OK;
}

size_t pat_get_buffer_bytes(void) {
  std::lock_guard<std::mutex> lock(g_mu);
  return budget_now();
}

pat_status_t pat_set_exec_mode(int mode) {
  if (mode < PAT_EXEC_PERSISTENT || mode > PAT_EXEC_DATAFLOW) return PAT_ERR_INVALID_ARGUMENT;
  std::lock_guard<std::mutex> lock(g_mu);
  g_mode = mode;
  return PAT_OK;
}

int pat_get_exec_mode(void) {
  std::lock_guard<std::mutex> lock(g_mu);
  return mode_now();
}

pat_status_t pat_set_top_fusion(int mode) {
  if (mode < PAT_FUSION_AUTO || mode > PAT_FUSION_ON) return PAT_ERR_INVALID_ARGUMENT;
  std::lock_guard<std::mutex> lock(g_mu);
  g_fusion = mode;
  return PAT_OK;
}

int pat_get_top_fusion(void) {
  std::lock_guard<std::mutex> lock(g_mu);
  return fusion_now();
}

pat_status_t pat_set_aggregation(int mode) {
  if (mode != PAT_AGGREGATION_POW2 && mode != PAT_AGGREGATION_BUDGET) return PAT_ERR_INVALID_ARGUMENT;
  std::lock_guard<std::mutex> lock(g_mu);
  g_aggregation = mode;
  return PAT_OK;
}

int pat_get_aggregation(void) {
  std::lock_guard<std::mutex> lock(g_mu);
  return aggregation_now();
}

pat_status_t pat_set_linear_order(int order) {
  if (order != PAT_LINEAR_FAR_FIRST && order != PAT_LINEAR_CLOSE_FIRST) return PAT_ERR_INVALID_ARGUMENT;
  std::lock_guard<std::mutex> lock(g_mu);
  g_order = order;
  return PAT_OK;
}

int pat_get_linear_order(void) {
  std::lock_guard<std::mutex> lock(g_mu);
  return order_now();
}

pat_status_t pat_set_barrier_timeout_us(uint32_t microseconds) {
  std::lock_guard<std::mutex> lock(g_mu);
  g_timeout_us = microseconds;
  return PAT_OK;
}

pat_status_t pat_plan_info(pat_collective_t coll, int nranks, size_t count, pat_dtype_t dtype,
                           pat_plan_info_t* out) {
  if (!out) return PAT_ERR_INVALID_ARGUMENT;
  pat::PlanDesc d;
  const pat_status_t s = describe((int)coll, nranks, count, dtype, &d);
  if (s != PAT_OK) return s;
  pat_plan_info_t info{};
  info.nranks = nranks;
  info.L = d.sched.L;
  info.t = d.sched.t;
  info.T = d.sched.T;
  info.steps = (int)d.exec.size();
  info.pieces = d.pieces;
  info.max_chunks_per_step = d.max_k;
  bool has[3] = {true, false, false};
  for (int path = 1; path < 3; ++path) {
    const pat::Variant v = variant_for((int)coll, dtype, path);
    has[path] = build_steps(d, pat::variant_in_bytes(v), pat::variant_tile(v), pat::variant_pack_tile(v),
                            path == 2 && pat::variant_partial(v), pat::variant_partial_items(v), nullptr);
  }
  info.vector_path = aligned_path(has);
  info.count = count;
  info.piece_elems = (size_t)d.piece_elems;
  info.slot_elem_bytes = (size_t)d.esize_slot;
  info.slot_dims = d.slots.dims;
  info.slot_chunks_per_rank = d.slots.entries;
  const size_t chunk_stride = entry_stride(size_t(d.piece_elems) * d.esize_slot);
  info.slot_bytes_per_rank = chunk_stride * d.slots.entries;
  const bool bf16_rs = coll == PAT_REDUCESCATTER && dtype == PAT_BFLOAT16;
  const size_t root = bf16_rs ? entry_stride(size_t(d.piece_elems) * 4) : 0;
  info.slot_bytes_total = (info.slot_bytes_per_rank + root) * size_t(nranks);
  info.alg_bytes = d.alg_bytes;
  info.bus_bytes_per_rank = double(nranks - 1) * double(count) * d.esize_in;
  {
    const pat::Variant var = variant_for((int)coll, dtype, info.vector_path);
    const int64_t per_vec = pat::variant_in_bytes(var) / d.esize_in;
    const int64_t V = pat::variant_partial_items(var) ? int64_t(d.piece_elems) / per_vec  // as build_steps counts
                                                      : (int64_t(d.piece_elems) + per_vec - 1) / per_vec;
    int s0, s1;
    int64_t tile;
    std::lock_guard<std::mutex> lock(g_mu);
    fused_range(d, V, fusion_now(), &s0, &s1, &tile);
    info.fused_steps = s1 - s0;
    info.launches_per_op = int(d.exec.size()) * d.pieces - (s1 > s0 ? s1 - s0 - 1 : 0);
    if (d.pipelined) info.launches_per_op = ((d.pieces - 1) / 2) * int(d.exec.size()) + (d.pieces - 1) % 2 + int(d.exec.size());
  }
  info.streaming = streaming_for(d.alg_bytes) ? 1 : 0;
  info.xcd_run = (int)std::min<int64_t>(xcd_run_for((int)coll), INT32_MAX);
  info.list_schedule = d.sched.list ? 1 : 0;
  *out = info;
  return PAT_OK;
}

pat_status_t pat_plan_steps(pat_collective_t coll, int nranks, size_t count, pat_dtype_t dtype, int32_t* step_d,
                            int32_t* step_k, int max_steps, int32_t* pos, int32_t* a, int32_t* b, int32_t* c,
                            int max_entries, int* nsteps, int* nentries) {
  if (!nsteps || !nentries) return PAT_ERR_INVALID_ARGUMENT;
  pat::PlanDesc d;
  const pat_status_t s = describe((int)coll, nranks, count, dtype, &d);
  if (s != PAT_OK) return s;
  *nsteps = (int)d.exec.size();
  *nentries = (int)d.entries.size();
  if (*nsteps > max_steps || *nentries > max_entries) return PAT_ERR_INVALID_ARGUMENT;
  for (size_t i = 0; i < d.exec.size(); ++i) {
    if (step_d) step_d[i] = d.exec[i].d;
    if (step_k) step_k[i] = d.exec[i].k;
  }
  for (size_t j = 0; j < d.entries.size(); ++j) {
    if (pos) pos[j] = d.entries[j].p;
    if (a) a[j] = d.entries[j].a;
    if (b) b[j] = d.entries[j].b;
    if (c) c[j] = d.entries[j].c;
  }
  return PAT_OK;
}

pat_status_t pat_trace_start(int max_launches) {
  if (max_launches < 1 || max_launches > (1 << 20)) return PAT_ERR_INVALID_ARGUMENT;
  std::lock_guard<std::mutex> lock(g_mu);
  g_trace.clear();
  g_trace.ev.assign(2 * size_t(max_launches), nullptr);
  // Timing-only events: without the system-scope fence an event record costs
  // no cache writeback, which would otherwise sit between the traced kernels.
  for (auto& e : g_trace.ev) {
    const hipError_t err = hipEventCreateWithFlags(&e, hipEventDisableSystemFence);
    if (err != hipSuccess) {
      g_last_hip.store((int)err);
      g_trace.clear();
      return PAT_ERR_HIP;
    }
  }
  g_trace.bytes.assign(max_launches, 0.0);
  g_trace.kind.assign(max_launches, 0);
  g_trace.step.assign(max_launches, 0);
  g_trace.max = max_launches;
  g_trace.armed = true;
  return PAT_OK;
}

pat_status_t pat_trace_read(float* ms, double* bytes, int32_t* kind, int32_t* step, int max, int* n) {
  if (!n) return PAT_ERR_INVALID_ARGUMENT;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_trace.armed) {
    *n = 0;
    return PAT_ERR_INVALID_ARGUMENT;
  }
  const int used = g_trace.used;
  *n = used;
  if (used > max) return PAT_ERR_INVALID_ARGUMENT;  // still armed: call again with room for n
  for (int j = 0; j < used; ++j) {
    float t = 0.0f;
    hipError_t e = hipEventSynchronize(g_trace.ev[2 * j + 1]);
    if (e == hipSuccess) e = hipEventElapsedTime(&t, g_trace.ev[2 * j], g_trace.ev[2 * j + 1]);
    if (e != hipSuccess) {
      g_last_hip.store((int)e);
      g_trace.clear();
      return PAT_ERR_HIP;
    }
    if (ms) ms[j] = t;
    if (bytes) bytes[j] = g_trace.bytes[j];
    if (kind) kind[j] = g_trace.kind[j];
    if (step) step[j] = g_trace.step[j];
  }
  g_trace.clear();
  return PAT_OK;
}

pat_status_t pat_step_clock(pat_collective_t coll, int nranks, size_t count, pat_dtype_t dtype, uint64_t* stamps,
                            size_t max, int* workgroups, int* per_workgroup, double* ticks_per_us) {
  if (!workgroups || !per_workgroup) return PAT_ERR_INVALID_ARGUMENT;
  *workgroups = *per_workgroup = 0;
  std::lock_guard<std::mutex> lock(g_mu);
  int device = 0;
  HIP_TRY(hipGetDevice(&device));
  auto it = g_plans.find(
      PlanKey((int)coll, nranks, (int64_t)count, (int)dtype, budget_now(), order_now(), device, aggregation_now()));
  if (it == g_plans.end() || !it->second->step_clock || it->second->stamp_wgs == 0) return PAT_ERR_INVALID_ARGUMENT;
  Plan* p = it->second.get();
  *workgroups = p->stamp_wgs;
  *per_workgroup = p->stamps_per_wg;
  if (ticks_per_us) *ticks_per_us = double(p->clock_khz) / 1000.0;
  const size_t need = size_t(p->stamp_wgs) * p->stamps_per_wg;
  if (!stamps || max < need) return PAT_ERR_INVALID_ARGUMENT;
  if (p->used) HIP_TRY(hipEventSynchronize(p->done));
  HIP_TRY(hipMemcpy(stamps, p->d_stamps, need * sizeof(uint64_t), hipMemcpyDeviceToHost));
  return PAT_OK;
}

pat_status_t pat_cache_stats(int* plans, size_t* bytes) {
  if (!plans || !bytes) return PAT_ERR_INVALID_ARGUMENT;
  std::lock_guard<std::mutex> lock(g_mu);
  *plans = (int)g_plans.size();
  size_t b = 0;
  for (const auto& kv : g_plans) b += kv.second->bytes;
  *bytes = b;
  return PAT_OK;
}

pat_status_t pat_check_device_status(hipStream_t stream) {
  HIP_TRY(hipStreamSynchronize(stream));
  std::lock_guard<std::mutex> lock(g_mu);
  int device = 0;
  HIP_TRY(hipGetDevice(&device));
  pat_status_t result = PAT_OK;
  for (auto& kv : g_plans) {
    Plan* p = kv.second.get();
    if (p->device != device) continue;
    unsigned st = 0;
    HIP_TRY(hipMemcpy(&st, p->d_sync + 2, sizeof(st), hipMemcpyDeviceToHost));
    if (st) {
      result = PAT_ERR_TIMEOUT;
      HIP_TRY(hipMemset(p->d_sync, 0, p->sync_words * sizeof(unsigned)));
    }
  }
  return result;
}

int pat_last_hip_error(void) { return g_last_hip.load(); }

const char* pat_status_string(pat_status_t status) {
  switch (status) {
    case PAT_OK: return "PAT_OK";
    case PAT_ERR_INVALID_ARGUMENT: return "PAT_ERR_INVALID_ARGUMENT";
    case PAT_ERR_UNSUPPORTED: return "PAT_ERR_UNSUPPORTED";
    case PAT_ERR_OUT_OF_MEMORY: return "PAT_ERR_OUT_OF_MEMORY";
    case PAT_ERR_HIP: return "PAT_ERR_HIP";
    case PAT_ERR_TIMEOUT: return "PAT_ERR_TIMEOUT";
    case PAT_ERR_INTERNAL: return "PAT_ERR_INTERNAL";
    case PAT_ERR_TOO_LARGE: return "PAT_ERR_TOO_LARGE";
    default: return "PAT_ERR_UNKNOWN";
  }
}

pat_status_t pat_finalize(void) {
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_plans.empty()) return PAT_OK;
  int cur = 0;
  HIP_TRY(hipGetDevice(&cur));
  std::vector<int> devices;
  for (auto& kv : g_plans) devices.push_back(kv.second->device);
  std::sort(devices.begin(), devices.end());
  devices.erase(std::unique(devices.begin(), devices.end()), devices.end());
  for (int dev : devices) {
    HIP_TRY(hipSetDevice(dev));
    HIP_TRY(hipDeviceSynchronize());
  }
  HIP_TRY(hipSetDevice(cur));
  g_plans.clear();
  return PAT_OK;
}

}  // extern "C"
