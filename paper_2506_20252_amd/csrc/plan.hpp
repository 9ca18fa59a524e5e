// Host-side PAT plan: schedule generation, slot layout and the byte model.
//
// Pure C++ (no HIP): the library builds every table here once per
// (collective, ranks, count, dtype, budget) and uploads it; the device never
// computes the schedule.  The paper notes that computing the steps is itself
// linear work (section "Performance"), so it is hoisted out of the hot path.
#pragma once

#include <cstddef>
#include <cstdint>
#include <vector>

#include "device_types.hpp"

namespace pat {

int ceil_log2(int64_t n);

// One step of the relative all-gather schedule: every rank r sends, for each
// tree position p in pos[first .. first + k), chunk (r - p) mod N to rank
// (r + d) mod N.  The table is the same for every rank up to the shift r.
struct StepSpec {
  int32_t d;
  int32_t k;
  int32_t first;
};

struct Schedule {
  int N = 0, L = 0, t = 0, T = 1, M = 1;
  bool list = false;            // a list schedule (make_list_schedule): K chunks per step, T = K, t and M unused
  std::vector<StepSpec> steps;  // all-gather order
  std::vector<int32_t> pos;     // sender positions, step after step
};

// Linear order inside the parallel sub-trees (section "The PAT algorithm"):
// far-first (the paper's main schedule) or close-first (the alternative it
// allows).  Both are pre-order walks, so each slot is drained before its
// distance is used again.
enum LinearOrder : int { kFarFirst = 0, kCloseFirst = 1 };

// Steps for N ranks and T = 2^t parallel sub-trees (section "The PAT
// algorithm"): the top t distances fully aggregated, farthest first; then a
// pre-order walk of a span-M sub-tree (M = 2^(L - t)) in the given linear
// order, every walk edge taken in all T sub-trees at once.  Edges a truncated
// tree lacks are dropped, and so is a step left empty.
Schedule make_schedule(int N, int t, int order = kFarFirst);

int max_chunks_per_step(const Schedule& s);

struct SlotMap;

// List schedule for K chunks per step (any K >= 1), one distance per step, as
// the paper's steps are: every rank sends to one peer r + d per step.  Each
// step takes the distance whose ready edges carry the largest sub-trees (ties:
// the farther distance), then up to K of its ready edges, largest sub-trees
// first; a node forwards its children farthest first, so the reduce-scatter
// adds them nearest first, the same association as the power-of-two
// schedule's.  An edge into a node that forwards needs room in the slot of
// its distance: at most K chunks per slot, a slot entry freed after the step
// of its chunk's last forward.  Entries are assigned lowest-free-first, and
// `slots` gets the resulting per-position table.  Returns an empty schedule
// with N > 1 if no step can be formed (cannot happen for K >= 1).
Schedule make_list_schedule(int N, int K, SlotMap* slots);

// Intermediate-buffer layout of one rank.  A node of a tree that forwards
// (all-gather) or accumulates (reduce-scatter) keeps the chunk in the slot of
// the distance D it arrived on / will leave on, D = lowest set bit of its
// position p, at index p / max(2D, M): the top distances use each slot once,
// and a linear-part slot holds one chunk per sub-tree because the far-first
// walk drains it before the same distance is used again.
struct SlotMap {
  int N = 0, L = 0, M = 1;
  std::vector<int32_t> base;  // by log2 D: first entry of that distance's slot
  std::vector<int32_t> cap;   // by log2 D: entries of that slot
  int32_t entries = 0;        // chunk-sized entries per rank
  int dims = 0;               // distances that need a slot
  std::vector<int32_t> table; // list schedules: entry of each position (-1: none); empty: the formula
  // Entry index of position p, or -1 if that node neither forwards nor accumulates.
  int32_t index(int p) const;
};

SlotMap make_slot_map(int N, int L, int M);

struct PlanDesc {
  int coll = 0;        // 0 all-gather, 1 reduce-scatter
  int order = kFarFirst;
  int N = 0;
  int dtype = 0;
  int64_t count = 0;
  int esize_in = 0;    // bytes per user element
  int esize_slot = 0;  // bytes per slot element (float32 partials for bf16 sums)
  Schedule sched;
  SlotMap slots;
  std::vector<DevEntry> entries;   // execution order
  std::vector<StepSpec> exec;      // execution order (reduce-scatter: reversed)
  int pieces = 1;
  int64_t piece_elems = 0;
  bool pipelined = false;  // pieces of half the budget, alternating between two halves of every slot
  int max_k = 0;
  double alg_bytes = 0.0;
};

// Aggregation rule: the paper's power-of-two number of parallel sub-trees,
// or any number of chunks per step the budget holds (the list schedule where
// it takes fewer steps than the power-of-two one).
enum Aggregation : int { kAggPow2 = 0, kAggBudget = 1 };

// Budget in bytes per slot.  Returns false for unsupported arguments.
// pipeline: a chunk larger than the budget is cut into pieces of half the
// budget, piece p using half p % 2 of every slot, so that two pieces can be
// in flight at once (their steps one apart); no effect when the chunk fits.
bool make_plan_desc(int coll, int N, int64_t count, int dtype, size_t budget, int order, PlanDesc* out,
                    int aggregation = kAggPow2, bool pipeline = false);

// Dependencies of every entry of d.entries for dataflow execution (one piece
// in execution order): for each of the two buffers an edge touches, the
// number of accesses to that buffer in earlier steps (see DevDep).  The
// schedule is the same for every rank up to a shift, so these counts hold at
// every rank.  Returns false if two edges of one step would touch one buffer
// (the schedules never do).
bool dataflow_deps(const PlanDesc& d, std::vector<DevDep>* deps);

// Algorithmic memory bytes of one operation (read + written by the steps):
// all-gather: per chunk-edge, read C, write C to the receiver's buffer, write
// C again to its slot when it forwards (plus each rank's own chunk, C);
// reduce-scatter: per chunk-edge, read the child's partial, read the
// receiver's own input or accumulator, write the accumulator.
double algorithmic_bytes(const PlanDesc& d);

// The same byte model for one step of one piece: step s of d.exec over a
// piece of `elems` elements per chunk, all N ranks (all-gather: the own
// chunk's copy counts in the first step).  Summed over every step and piece
// it gives algorithmic_bytes(d).
double step_bytes(const PlanDesc& d, int s, int64_t elems);

}  // namespace pat
