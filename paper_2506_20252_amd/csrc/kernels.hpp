// Step kernels: host-side launch interface.
#pragma once

#include <hip/hip_runtime_api.h>

#include <cstdint>

#include "device_types.hpp"

namespace pat {

#ifndef PAT_THREADS
#define PAT_THREADS 256
#endif
constexpr int kThreads = PAT_THREADS;  // workgroup size, a multiple of the 64-lane wavefront

// Everything a step kernel needs, passed by value (device pointers only).
struct KCtx {
  const void* const* send;    // [N] device pointers (library-owned device table)
  void* const* recv;          // [N]
  char* slots;                // slot area: rank r's entries start at r * slot_rank_stride
  char* rootacc;              // bf16 reduce-scatter: float32 root accumulators, [N][piece]
  const DevEntry* entries;
  const DevStep* steps;
  int64_t count;              // elements per chunk
  int64_t slot_chunk_stride;  // bytes per slot entry
  int64_t slot_rank_stride;   // bytes per rank's slot area
  int64_t rootacc_stride;     // bytes per rank's root accumulator
  int64_t esize;              // bytes per user element
  int32_t N;
  int32_t nsteps;             // launch-level steps (schedule steps x pieces)
  int32_t own_copy;           // all-gather: copy the own chunk (0 when in place)
  uint32_t pad0;
  int64_t timeout_ticks;      // persistent kernel: wall-clock ticks one wait may take before giving up
  unsigned* queue;            // persistent kernel: [1] workgroups finished, then per step 32 sharded
                              // "ids taken", 32 "ids done" and one "shards done" counter, 128 B apart
                              // (zero between launches)
  unsigned* status;           // bit 0: a persistent kernel's wait timed out
  uint64_t* stamps;           // fused launches, measurement only (null: off): per workgroup, the device
                              // wall clock before its first step and after each step, (s1 - s0 + 1) apiece
  const DevDep* deps;         // dataflow execution: per entry of the step table, the counters it waits on
  unsigned* counters;         // dataflow execution: [N][counter_stride] completed tiles per buffer (zero
                              // between launches)
  int64_t counter_stride;     // slot entries per rank + 1 (the own chunk's accumulator)
  int64_t slot_half_bytes;    // pipelined pieces: offset of a slot area's second half (0 otherwise)
  int64_t root_half_bytes;    // pipelined pieces: offset of a root accumulator's second half
};

// Words of the persistent kernel's counter area for `nsteps` launch-level steps.
inline size_t queue_words(size_t nsteps) { return 4 + (2 * 32 + 1) * nsteps * 32; }

enum Variant : int {
  kAgVec = 0,   // all-gather, 16-byte units
  kAgS4,        // all-gather, 4-byte elements
  kAgS2,        // all-gather, 2-byte elements
  kRsI32Vec,
  kRsF32Vec,
  kRsB16Vec,    // bf16 in (4 per vector), float32 partials
  kRsI32S,
  kRsF32S,
  kRsB16S,
  // Relaxed vectors: 16-byte vectors (bf16 reduce-scatter inputs: 8-byte) at
  // element-aligned addresses; a chunk-piece may end in a partial vector.
  kAgVecU,
  kRsI32VecU,
  kRsF32VecU,
  kRsB16VecU,
  kNumVariants
};

// Bytes of user data per vector; vectors of one tiled work item (one tile of
// one edge) and of one packed work item (consecutive vectors of consecutive
// edges).  The element-wide variants give a tiled item twice the vectors.
int variant_in_bytes(Variant v);
int variant_tile(Variant v);
int variant_pack_tile(Variant v);
// A chunk-piece may end in a partial vector (the relaxed variants).
bool variant_partial(Variant v);
// Its partial vector is not among the V the vector loops take: the step's
// last work items take every edge's, one per lane (the relaxed bf16
// reduce-scatter).  Otherwise the vector loops take it as vector V - 1.
bool variant_partial_items(Variant v);

// streaming: nontemporal loads and stores, for operations much larger than
// the 256 MB Infinity Cache; plain accesses let a small operation's steps
// hit in it (each step reads the slots the previous one wrote).
// grain: each XCD takes runs of this many consecutive work items (1: every
// eighth item; large: a contiguous eighth of the step; see step_kernel).
hipError_t launch_step(Variant v, bool streaming, int64_t grain, const KCtx& cx, const DevStep& st,
                       hipStream_t stream);
// Pipelined pieces: two launch-level steps of the device step table (indices
// ia, ib; different pieces and slot halves, hence independent) in one launch,
// the items of step ia first.
hipError_t launch_step2(Variant v, bool streaming, int64_t grain, const KCtx& cx, int ia, const DevStep& a, int ib,
                        const DevStep& b, hipStream_t stream);
// Fused range: launch-level steps [s0, s1) of one piece, run by one
// workgroup per (tree, tile of tile_vecs vectors); tiles = ceil(V / tile_vecs).
// Most slot entries, and steps, whose edges a fused launch resolves into LDS.
constexpr int kTreeCacheEdges = 128;
constexpr int kTreeCacheSteps = 16;

struct TreeRange {
  int32_t s0, s1;
  int64_t tile_vecs;
  int64_t tiles;
  // Steps [c0, c1) within [s0, s1) whose edges each workgroup resolves into
  // LDS once: their cn entries (at most kTreeCacheEdges; 0: none) are
  // entries [ce0, ce0 + cn) of the plan, and entry ce0 + t belongs to step
  // c0 + (the number of cend[] values <= t), cend[i] being the end of step
  // c0 + i relative to ce0.
  int32_t c0, c1;
  int32_t cn, ce0;
  int16_t cend[kTreeCacheSteps];
};
hipError_t launch_tree(Variant v, bool streaming, const KCtx& cx, const TreeRange& tr, hipStream_t stream);
// Persistent execution: one launch of `grid` workgroups that take per-step
// worker ids from device counters in step order.  Any grid size is safe (a
// workgroup only waits on work that running workgroups already hold).
hipError_t launch_persistent(Variant v, bool streaming, const KCtx& cx, int grid, hipStream_t stream);
// Dataflow execution: one launch per piece (cx.steps: that piece's steps,
// cx.nsteps of them), workgroups taking per-step worker ids like the
// persistent kernel, every work item waiting only for the counters of the
// buffers its edges touch.  small: every step packs whole edges into items
// (DevStep::df_edges, chunks under one tile); else items are DevStep::df_tiles
// tiles of one edge.  Any grid size is safe.
hipError_t launch_dataflow(Variant v, bool streaming, const KCtx& cx, bool small, int grid, hipStream_t stream);
// Workgroups of the persistent kernel that fit on the current device at once.
hipError_t persistent_capacity(Variant v, bool streaming, int* blocks);

// The no-allocation entry point's fixed scratch array (noalloc.hip): its size,
// and its device address on `device`, which must be the current device.
size_t scratch_bytes();
hipError_t scratch_base(int device, char** base);

}  // namespace pat
