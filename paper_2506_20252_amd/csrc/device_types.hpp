// Tables the host uploads and the step kernels read.  Plain structs, no HIP.
#pragma once

#include <cstdint>

namespace pat {

// Markers in DevEntry slot fields.
enum : int32_t {
  kUser = -1,       // the rank's own send buffer (raw input)
  kRoot = -2,       // the rank's own chunk: receive buffer (int32/fp32) or float32 root accumulator (bf16)
  kRootFinal = -3,  // the root's last receive: write the receive buffer (bf16: rounded)
};

// One chunk-edge of a step, relative to the acting rank r (16 bytes).
//   all-gather:     p = sender position;   a = source slot | kUser;   b = receiver slot | kUser (none);
//                   c = kUser (unused)
//   reduce-scatter: p = receiver position; a = child slot | kUser (child's input);
//                   b = own accumulator slot | kUser (own input) | kRoot;
//                   c = destination slot | kRoot | kRootFinal
struct DevEntry {
  int32_t p, a, b, c;
};

// Dataflow execution: the two rank-relative counters one chunk-edge touches
// (entry j of the step table).  Every rank's slot entry e (and, as entry
// `entries`, its own chunk's accumulator) counts the completed tiles of the
// edges that accessed it.  Access 1 is at rank r + o1, access 2 at r + o2
// (all-gather: o1 = 0, the sender's source slot; o2 = d, the receiver's slot;
// reduce-scatter: o1 = d, the child's partial; o2 = 0, the receiver's
// accumulator).  e = -1: no counter.  Counters count completed tiles (1 per
// whole edge for chunks under one tile); an edge may run once counter e has
// reached need * (tiles per edge): every earlier access to that buffer, in
// step order, is complete.
struct DevDep {
  int32_t e1, need1, e2, need2;
};

// One launch-level step (a schedule step of one piece), as the kernels see it.
struct DevStep {
  int32_t d;               // distance: peer = r + d (all-gather) / child = r + d (reduce-scatter)
  int32_t k;               // entries per rank
  int32_t entry0;          // first entry in the entry table
  int16_t first;           // 1: first step of a piece (all-gather fuses the own-chunk copy here)
  int16_t back;            // relaxed variants: the piece ends in a partial vector, made of its
                           // last 4 or 8 elements, which begin this many elements inside the
                           // last whole vector; 0: no partial vector
  int64_t e0;              // first element of the piece within a chunk
  int64_t V;               // vectors per chunk-piece: a partial one counts as vector V - 1, or,
                           // where the step's last work items take it, not at all
  int64_t tiles_per_edge;  // > 0: each work item is one tile of one edge; 0: items pack edges
  int64_t items;           // work items (workgroups) of this step; where they take the partial
                           // vectors, the last ceil(N * k / 256) give each edge's to a lane
  int32_t df_edges;        // dataflow execution: whole edges per work item (chunks under one tile;
                           // 0: the item is df_tiles tiles of one edge)
  int32_t df_tiles;        // dataflow execution: tiles of one edge per work item
  int32_t half;            // pipelined pieces: the half of every slot (and root accumulator) this
                           // piece uses (0 otherwise)
  int32_t pad;
};

}  // namespace pat
