// PAT step kernels for gfx950 (CDNA4).
//
// One step of the schedule is N * k independent chunk-edges (k entries of the
// step table, for every acting rank r).  A workgroup processes one work item:
//   tiled:  one tile of kThreads * kUnroll vectors of one edge, the edge's
//           addresses computed once per workgroup (wavefront-uniform);
//   packed: chunks smaller than a tile; consecutive vectors of consecutive
//           edges, addresses computed per lane.
// Every lane issues all of its loads before it uses any (U vectors per
// stream, 16 bytes each; bf16 reduce-scatter: 8-byte inputs beside 16-byte
// float32 partials, at twice the unroll) and stores only after every value of
// its tile is computed, so that neither a conversion nor a store in a branch
// makes the compiler wait for one access before the next.  Accesses use
// explicit global pointers; loads and stores are nontemporal for operations
// far larger than the Infinity Cache, and plain (cached) otherwise, so that a
// small operation's next step finds the slots just written still in cache.
// The data path has no matrix work and no reuse, so there is no LDS staging:
// a load lands in VGPRs and is stored from there.
//
// Variants: aligned vectors (16-byte-aligned buffers, whole vectors), relaxed
// vectors (element-aligned buffers; a chunk-piece may end in a partial
// vector, which ends where the piece ends and stores only the elements past
// the vector before it) and single elements (pieces under one vector).
//
// All-gather step (section "The PAT algorithm"): the sender at tree position
// p copies chunk (r - p) mod N from its send buffer (p = 0) or from the slot
// it arrived in, to the receiver r + d: into its receive buffer, and into its
// slot when the receiver forwards the chunk later.  The first step also
// copies each rank's own chunk into its receive buffer (a local copy).
//
// Reduce-scatter step (section "Conversion to reduce-scatter operations"):
// the receiver at position p of tree c = (r - p) mod N loads the partial of
// the child at p + d (its raw input if it is a leaf, else its accumulator
// slot) and its own value (raw input at the first receive, else its
// accumulator), adds, and stores the accumulator -- or, at the root, the
// receive buffer.  int32 adds wrap; float32 adds round to nearest even;
// bf16 data is widened exactly to float32 and rounded once, at the root's
// last receive.
//
// Step order: steps depend on each other (a slot written at step s is read
// at step s + 1).  Per-step launches get the ordering from the kernel
// boundary; the persistent kernel orders its work queue by per-step
// completion counters whose fences make every workgroup's writes visible
// across the XCDs' separate L2 caches; a fused range of steps (tree_kernel)
// needs only workgroup barriers, since there each tree's data is its
// workgroup's.

#include <hip/hip_runtime.h>

#include <type_traits>

#include "kernels.hpp"

// Tuning knobs (compile time): vectors in flight per lane.  Whether loads and
// stores stream (nontemporal) and the work-item order are launch arguments,
// chosen per plan.
//
// The all-gather's whole-vector stores into receive buffers stream
// (nontemporal) even where the plan keeps its accesses cached: the operation
// never reads them again, and caching them only evicts the slots the next
// steps read (measured on MI355X: all-gathers of N=1000 ranks with 256 B
// chunks and of N=24 with 64 KiB chunks run 9-10% faster).  A chunk's partial
// last vector, a few element stores into a line shared with the next chunk,
// keeps the plan's policy: streamed, it made an odd count 38% slower.  The
// reduce-scatter's raw inputs, also read once, measured no different
// streamed and keep the plan's policy.
#ifndef PAT_UNROLL
#define PAT_UNROLL 2
#endif
// bf16 reduce-scatter: 8-byte input vectors beside 16-byte float32 partials.
#ifndef PAT_B16_UNROLL
#define PAT_B16_UNROLL (2 * PAT_UNROLL)
#endif
// Element-wide kernels (pointers or sizes that rule out 128-bit vectors): 4
// elements per lane on the packed and fused paths, 8 on the tiled path, where
// a lane's few bytes in flight otherwise limit a bandwidth-bound step.
#ifndef PAT_SCALAR_UNROLL
#define PAT_SCALAR_UNROLL 4
#endif
#ifndef PAT_SCALAR_TILED_UNROLL
#define PAT_SCALAR_TILED_UNROLL 8
#endif

namespace pat {
namespace {

// Native clang vectors (not HIP's wrapper structs), so that the nontemporal
// builtins apply directly to the 128-bit loads and stores.
typedef unsigned int v2u __attribute__((ext_vector_type(2)));
typedef unsigned int v4u __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int kSU = PAT_SCALAR_UNROLL;         // element-wide kernels: packed and fused paths
constexpr int kSTU = PAT_SCALAR_TILED_UNROLL;  // element-wide kernels: tiled path

// Buffer addresses come from pointer tables, so the compiler cannot tell they
// are global memory and would emit flat accesses; every data access goes
// through an explicit global (address space 1) pointer instead.
#define PAT_GLOBAL __attribute__((address_space(1)))

// Access alignment A: 0 keeps the type's own; A > 0 lets a 16-byte vector
// sit at any A-byte-aligned address (the relaxed variants, for buffers that
// are only element-aligned).  Code objects for gfx950 run in unaligned-access
// mode, where such a vector is still one 128-bit load or store.
template <typename T, int A>
struct Access {
  typedef T type __attribute__((aligned(A)));
};
template <typename T>
struct Access<T, 0> {
  typedef T type;
};

template <typename T, bool NT, int A = 0>
__device__ __forceinline__ T ldg(const char* p) {
  using AT = typename Access<T, A>::type;
  const PAT_GLOBAL AT* q = (const PAT_GLOBAL AT*)(p);
  if constexpr (NT) return __builtin_nontemporal_load(q);
  return *q;
}

template <bool NT, int A = 0, typename T>
__device__ __forceinline__ void stg(char* p, const T& v) {
  using AT = typename Access<T, A>::type;
  PAT_GLOBAL AT* q = (PAT_GLOBAL AT*)(p);
  if constexpr (NT)
    __builtin_nontemporal_store(v, q);
  else
    *q = v;
}

// Word q of a vector, as raw bits.
__device__ __forceinline__ uint32_t word(v4u x, int q) { return x[q]; }
__device__ __forceinline__ uint32_t word(v2u x, int q) { return x[q]; }
__device__ __forceinline__ uint32_t word(v4f x, int q) { return __float_as_uint(x[q]); }

// Stores elements [from, n) of the vector x, taken as n elements of EB bytes
// each (EB = 2 or 4; 2-byte element 2j is the low half of word j).  Used for
// a chunk-piece's partial last vector, which is moved back to end at the
// piece's end: its first `from` elements belong to the vector before it.
template <bool NT, int EB, typename T>
__device__ __forceinline__ void stg_from(char* p, T x, int from) {
  static_assert(EB == 2 || EB == 4, "2- or 4-byte elements");
  constexpr int W = sizeof(T) / 4;
  if constexpr (EB == 4) {
#pragma unroll
    for (int q = 0; q < W; ++q)
      if (q >= from) stg<NT>(p + 4 * q, word(x, q));
  } else {
#pragma unroll
    for (int q = 0; q < 2 * W; ++q)
      if (q >= from) stg<NT>(p + 2 * q, (uint16_t)(word(x, q / 2) >> (16 * (q & 1))));
  }
}

__device__ __forceinline__ int wrap_add(int a, int b, int n) {
  const int s = a + b;
  return s >= n ? s - n : s;
}

__device__ __forceinline__ int wrap_sub(int a, int b, int n) {
  const int s = a - b;
  return s < 0 ? s + n : s;
}

// Split a flat vector index of a packed step into (rank, entry, vector).
__device__ __forceinline__ void split_flat(int64_t g, const DevStep& st, int* r, int* i, int64_t* v,
                                           bool small) {
  if (small) {
    const uint32_t gg = (uint32_t)g, V = (uint32_t)st.V, k = (uint32_t)st.k;
    const uint32_t e = gg / V;
    *v = gg - e * V;
    *r = (int)(e / k);
    *i = (int)(e - (uint32_t)(*r) * k);
  } else {
    const int64_t e = g / st.V;
    *v = g - e * st.V;
    *r = (int)(e / st.k);
    *i = (int)(e - (int64_t)(*r) * st.k);
  }
}

// Waits for every outstanding memory access of this wave.  Used between a
// load phase and stores that sit in per-lane branches: there the compiler
// cannot count which loads a store still needs and waits before each store
// for all earlier ones, stores included; one wait up front avoids that.
__device__ __forceinline__ void wait_loads() { __builtin_amdgcn_s_waitcnt(0); }

// Work items of a step that cover whole vectors: with a partial vector per
// edge (st.back > 0), the step's last items give each edge's one to a lane.
__device__ __forceinline__ int64_t main_items(const KCtx& cx, const DevStep& st) {
  return st.back ? st.items - ((int64_t)cx.N * st.k + kThreads - 1) / kThreads : st.items;
}

// Split a tiled work item into (rank, entry, tile).
__device__ __forceinline__ void split_tile(int64_t item, const DevStep& st, int* r, int* i, int64_t* tile) {
  const int64_t e = item / st.tiles_per_edge;
  *tile = item - e * st.tiles_per_edge;
  *r = (int)(e / st.k);
  *i = (int)(e - (int64_t)(*r) * st.k);
}

// Workgroup size of a fused range of steps.  A tree's steps run one after
// another inside its workgroup, so a wide workgroup covers a whole step in
// fewer load rounds (a shorter chain of dependent accesses per step).  The
// host's tile choice assumes 256 lanes.
#ifndef PAT_TREE_THREADS
#define PAT_TREE_THREADS 256
#endif
constexpr int kTreeThreads = PAT_TREE_THREADS;
static_assert(kTreeThreads % 64 == 0 && kTreeThreads <= 1024, "tree workgroup: whole wavefronts, at most 1024 lanes");

// One step of one tree in a fused range: the pairs (entry i, vector v)
// with i < k and v in [t0, t0 + TV), flattened vector-fastest so that lanes
// sweep each edge's tile contiguously, U pairs per lane at a time.  CACHED:
// the step's edges were resolved for this tree at the start of the launch and
// sit in LDS at `cached`, so a lane reads its edges there instead of loading
// the entries and pointer tables, and a narrow step is one data round trip.
template <class Op, bool CACHED>
__device__ __forceinline__ void tree_step_impl(const KCtx& cx, const DevStep& st, int c, int64_t t0, int64_t TV,
                                               const typename Op::Edge* cached) {
  constexpr int U = Op::U;
  const int64_t n = (int64_t)st.k * TV;
  for (int64_t base = 0; base < n; base += (int64_t)kTreeThreads * U) {
    int rr[U], ii[U];
    int64_t vv[U];
#pragma unroll
    for (int j = 0; j < U; ++j) {
      const int64_t f = base + j * kTreeThreads + threadIdx.x;
      vv[j] = -1;
      rr[j] = c;
      ii[j] = 0;
      if (f < n) {
        const int64_t i = f / TV;
        ii[j] = (int)i;
        vv[j] = t0 + (f - i * TV);
      }
    }
    Op::template batch<true, CACHED>(cx, st, rr, ii, vv, cached);
  }
}

// ---------------------------------------------------------------------------
// All-gather
// ---------------------------------------------------------------------------

// U vectors per lane on the packed and fused paths, TU on the tiled path.
// kA > 0: the relaxed variant (A-byte-aligned 16-byte vectors; a chunk-piece
// may end in a partial vector, st.back elements short).
template <typename Unit, int kU, bool NT, int kTU = kU, int kA = 0>
struct AgOp {
  static constexpr bool kGather = true;
  static constexpr int U = kU;
  static constexpr int TU = kTU;
  static constexpr int kTile = kThreads * TU;      // vectors of one tiled work item
  static constexpr int kPackTile = kThreads * U;   // vectors of one packed work item
  static constexpr bool kTail = kA > 0;
  static constexpr bool RNT = true;  // whole-vector stores into receive buffers: always streaming
  static_assert(!kTail || sizeof(Unit) == 16, "relaxed all-gather moves 16-byte vectors");

  struct Edge {
    const char* src;
    char* dst;   // receiver's receive buffer
    char* dst2;  // receiver's slot (null: the receiver does not forward)
    char* dst3;  // own chunk into the sender's receive buffer (first step only)
  };

  __device__ static Edge edge(const KCtx& cx, const DevStep& st, int r, int i) {
    return edge_of(cx, st, r, cx.entries[st.entry0 + i]);
  }

  __device__ static Edge edge_of(const KCtx& cx, const DevStep& st, int r, const DevEntry& en) {
    const int c = wrap_sub(r, en.p, cx.N);
    const int peer = wrap_add(r, st.d, cx.N);
    const int64_t piece = st.e0 * cx.esize;
    const int64_t chunk = cx.count * cx.esize;
    // Pointer-table reads happen whether or not the edge uses them, so that
    // none of them sits in a branch of its own (and waits there).
    const char* send_r = (const char*)cx.send[r];
    char* recv_peer = (char*)cx.recv[peer];
    char* recv_r = (char*)cx.recv[r];
    char* const slots = cx.slots + st.half * cx.slot_half_bytes;
    Edge e;
    e.src = en.a == kUser ? send_r + piece : slots + r * cx.slot_rank_stride + en.a * cx.slot_chunk_stride;
    e.dst = recv_peer + c * chunk + piece;
    e.dst2 = en.b >= 0 ? slots + peer * cx.slot_rank_stride + en.b * cx.slot_chunk_stride : nullptr;
    e.dst3 = (st.first && en.p == 0 && cx.own_copy) ? recv_r + r * chunk + piece : nullptr;
    return e;
  }

  // Byte offset of vector v in the chunk-piece.  A partial last vector is
  // moved back by st.back elements so that it ends where the piece ends: it
  // loads the tail of the vector before it too, and stores only its own
  // elements.
  __device__ static int64_t off(const KCtx& cx, const DevStep& st, int64_t v) {
    int64_t o = v * (int64_t)sizeof(Unit);
    if constexpr (kTail)
      if (v == st.V - 1) o -= st.back * cx.esize;
    return o;
  }

  __device__ static void put(const KCtx& cx, const DevStep& st, const Edge& e, int64_t v, const Unit& x) {
    const int64_t o = off(cx, st, v);
    if constexpr (kTail) {
      if (st.back && v == st.V - 1) {
        if (cx.esize == 4) {
          stg_from<NT, 4>(e.dst + o, x, st.back);
          if (e.dst2) stg_from<NT, 4>(e.dst2 + o, x, st.back);
          if (e.dst3) stg_from<NT, 4>(e.dst3 + o, x, st.back);
        } else {
          stg_from<NT, 2>(e.dst + o, x, st.back);
          if (e.dst2) stg_from<NT, 2>(e.dst2 + o, x, st.back);
          if (e.dst3) stg_from<NT, 2>(e.dst3 + o, x, st.back);
        }
        return;
      }
    }
    stg<RNT, kA>(e.dst + o, x);
    if (e.dst2) stg<NT, kA>(e.dst2 + o, x);
    if (e.dst3) stg<RNT, kA>(e.dst3 + o, x);
  }

  // Vectors of the chunk-piece that the straight-line full-tile code may take
  // (all but a partial last one).
  __device__ static int64_t whole_vecs(const DevStep& st) {
    if constexpr (kTail) return st.V - (st.back ? 1 : 0);
    return st.V;
  }

  __device__ static void run(const KCtx& cx, const DevStep& st, int64_t item) {
    if (st.tiles_per_edge > 0) {
      Unit x[TU];
      int r, i;
      int64_t tile;
      split_tile(item, st, &r, &i, &tile);
      const Edge e = edge(cx, st, r, i);
      const int64_t v0 = tile * kTile + threadIdx.x;
      if ((tile + 1) * kTile <= whole_vecs(st)) {
        // Full tile (uniform): straight-line loads, then one store loop per
        // destination, so no store waits for another store.
#pragma unroll
        for (int j = 0; j < TU; ++j)
          x[j] = ldg<Unit, NT, kA>(e.src + (v0 + j * kThreads) * (int64_t)sizeof(Unit));
#pragma unroll
        for (int j = 0; j < TU; ++j) stg<RNT, kA>(e.dst + (v0 + j * kThreads) * (int64_t)sizeof(Unit), x[j]);
        if (e.dst2) {
#pragma unroll
          for (int j = 0; j < TU; ++j) stg<NT, kA>(e.dst2 + (v0 + j * kThreads) * (int64_t)sizeof(Unit), x[j]);
        }
        if (e.dst3) {
#pragma unroll
          for (int j = 0; j < TU; ++j) stg<RNT, kA>(e.dst3 + (v0 + j * kThreads) * (int64_t)sizeof(Unit), x[j]);
        }
        return;
      }
#pragma unroll
      for (int j = 0; j < TU; ++j) {
        const int64_t v = v0 + j * kThreads;
        if (v < st.V) x[j] = ldg<Unit, NT, kA>(e.src + off(cx, st, v));
      }
      wait_loads();
#pragma unroll
      for (int j = 0; j < TU; ++j) {
        const int64_t v = v0 + j * kThreads;
        if (v < st.V) put(cx, st, e, v, x[j]);
      }
    } else {
      const int64_t units = (int64_t)cx.N * st.k * st.V;
      const bool small = units < (int64_t(1) << 31);
      int rr[U], ii[U];
      int64_t vv[U];
#pragma unroll
      for (int j = 0; j < U; ++j) {
        const int64_t g = item * kPackTile + j * kThreads + threadIdx.x;
        vv[j] = -1;
        if (g < units) split_flat(g, st, &rr[j], &ii[j], &vv[j], small);
      }
      batch<false>(cx, st, rr, ii, vv);
    }
  }

  // U vectors per lane, each given as (rank, entry, vector), or (tree, entry,
  // vector) when TREE (the acting rank is then tree + the entry's position);
  // vv[j] < 0 marks an unused slot.  In phases (entries, then pointer tables,
  // then data), so that each level of dependent loads is in flight for all U
  // vectors at once.
  // CACHED: the edges of entries ii[] are at cached[ii[j]] (LDS).
  template <bool TREE, bool CACHED = false>
  __device__ static void batch(const KCtx& cx, const DevStep& st, const int (&rr)[U], const int (&ii)[U],
                               const int64_t (&vv)[U], const Edge* cached = nullptr) {
    Unit x[U];
    Edge e[U];
    if constexpr (CACHED) {
#pragma unroll
      for (int j = 0; j < U; ++j)
        if (vv[j] >= 0) e[j] = cached[ii[j]];
    } else {
      DevEntry en[U];
#pragma unroll
      for (int j = 0; j < U; ++j)
        if (vv[j] >= 0) en[j] = cx.entries[st.entry0 + ii[j]];
#pragma unroll
      for (int j = 0; j < U; ++j)
        if (vv[j] >= 0) e[j] = edge_of(cx, st, TREE ? wrap_add(rr[j], en[j].p, cx.N) : rr[j], en[j]);
    }
#pragma unroll
    for (int j = 0; j < U; ++j)
      if (vv[j] >= 0) x[j] = ldg<Unit, NT, kA>(e[j].src + off(cx, st, vv[j]));
    wait_loads();
#pragma unroll
    for (int j = 0; j < U; ++j)
      if (vv[j] >= 0) put(cx, st, e[j], vv[j], x[j]);
  }

  // Every edge of step st in tree c, over vectors [t0, t0 + TV) of the chunk
  // (a partial last vector among them); `cached`: the step's resolved edges.
  template <bool CACHED>
  __device__ static void tree_step(const KCtx& cx, const DevStep& st, int c, int64_t t0, int64_t TV, bool,
                                   const Edge* cached) {
    tree_step_impl<AgOp, CACHED>(cx, st, c, t0, TV, cached);
  }
};

// ---------------------------------------------------------------------------
// Reduce-scatter
// ---------------------------------------------------------------------------

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// float32 -> bf16, round to nearest, ties to even (NaN stays a quiet NaN).
__device__ __forceinline__ uint32_t bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (u >> 16) | 0x40u;
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

struct TI32V {
  using in_t = v4u;
  using acc_t = v4u;
  static constexpr int kInElem = 4;
  static constexpr int kAlign = 0;  // natural alignment
  static constexpr bool kPartial = false;
  static constexpr bool kPartialItems = false;
  static constexpr bool kSeparateRoot = false;
  static constexpr int kUnroll = PAT_UNROLL;
  static constexpr int kTiledUnroll = kUnroll;
  __device__ static acc_t widen(const in_t& x) { return x; }
  __device__ static in_t narrow(const acc_t& x) { return x; }
  __device__ static acc_t add(const acc_t& a, const acc_t& b) { return a + b; }  // wraps
};

struct TF32V {
  using in_t = v4f;
  using acc_t = v4f;
  static constexpr int kInElem = 4;
  static constexpr int kAlign = 0;  // natural alignment
  static constexpr bool kPartial = false;
  static constexpr bool kPartialItems = false;
  static constexpr bool kSeparateRoot = false;
  static constexpr int kUnroll = PAT_UNROLL;
  static constexpr int kTiledUnroll = kUnroll;
  __device__ static acc_t widen(const in_t& x) { return x; }
  __device__ static in_t narrow(const acc_t& x) { return x; }
  __device__ static acc_t add(const acc_t& a, const acc_t& b) { return a + b; }
};

struct TB16V {
  using in_t = v2u;  // 4 bf16, element 2j in the low half of word j
  using acc_t = v4f;
  static constexpr int kInElem = 2;
  static constexpr int kAlign = 0;  // natural alignment
  static constexpr bool kPartial = false;
  static constexpr bool kPartialItems = false;
  static constexpr bool kSeparateRoot = true;
  static constexpr int kUnroll = PAT_B16_UNROLL;
  static constexpr int kTiledUnroll = kUnroll;
  __device__ static acc_t widen(const in_t& x) {
    return v4f{bf16_lo(x.x), bf16_hi(x.x), bf16_lo(x.y), bf16_hi(x.y)};
  }
  __device__ static in_t narrow(const acc_t& a) {
    return v2u{bf16_rne(a.x) | (bf16_rne(a.y) << 16), bf16_rne(a.z) | (bf16_rne(a.w) << 16)};
  }
  __device__ static acc_t add(const acc_t& a, const acc_t& b) { return a + b; }
};

struct TI32S {
  using in_t = uint32_t;
  using acc_t = uint32_t;
  static constexpr int kInElem = 4;
  static constexpr int kAlign = 0;  // natural alignment
  static constexpr bool kPartial = false;
  static constexpr bool kPartialItems = false;
  static constexpr bool kSeparateRoot = false;
  static constexpr int kUnroll = PAT_SCALAR_UNROLL;
  static constexpr int kTiledUnroll = PAT_SCALAR_TILED_UNROLL;
  __device__ static acc_t widen(in_t x) { return x; }
  __device__ static in_t narrow(acc_t x) { return x; }
  __device__ static acc_t add(acc_t a, acc_t b) { return a + b; }
};

struct TF32S {
  using in_t = float;
  using acc_t = float;
  static constexpr int kInElem = 4;
  static constexpr int kAlign = 0;  // natural alignment
  static constexpr bool kPartial = false;
  static constexpr bool kPartialItems = false;
  static constexpr bool kSeparateRoot = false;
  static constexpr int kUnroll = PAT_SCALAR_UNROLL;
  static constexpr int kTiledUnroll = PAT_SCALAR_TILED_UNROLL;
  __device__ static acc_t widen(in_t x) { return x; }
  __device__ static in_t narrow(acc_t x) { return x; }
  __device__ static acc_t add(acc_t a, acc_t b) { return a + b; }
};

struct TB16S {
  using in_t = uint16_t;
  using acc_t = float;
  static constexpr int kInElem = 2;
  static constexpr int kAlign = 0;  // natural alignment
  static constexpr bool kPartial = false;
  static constexpr bool kPartialItems = false;
  static constexpr bool kSeparateRoot = true;
  static constexpr int kUnroll = PAT_SCALAR_UNROLL;
  static constexpr int kTiledUnroll = PAT_SCALAR_TILED_UNROLL;
  __device__ static acc_t widen(in_t x) { return __uint_as_float((uint32_t)x << 16); }
  __device__ static in_t narrow(acc_t x) { return (uint16_t)bf16_rne(x); }
  __device__ static acc_t add(acc_t a, acc_t b) { return a + b; }
};

// Relaxed variants: the vector traits at element alignment, for buffers that
// are not 16-byte aligned and chunk-pieces that end in a partial vector.
struct TI32U : TI32V {
  static constexpr int kAlign = 4;
  static constexpr bool kPartial = true;
};
struct TF32U : TF32V {
  static constexpr int kAlign = 4;
  static constexpr bool kPartial = true;
};
struct TB16U : TB16V {
  static constexpr int kAlign = 2;
  static constexpr bool kPartial = true;
  static constexpr bool kPartialItems = true;  // partial vectors in work items of their own
};

template <class R, bool NT>
struct RsOp {
  static constexpr bool kGather = false;
  using in_t = typename R::in_t;
  using acc_t = typename R::acc_t;
  static constexpr int U = R::kUnroll;         // packed and fused paths
  static constexpr int TU = R::kTiledUnroll;   // tiled path
  static constexpr int kTile = kThreads * TU;
  static constexpr int kPackTile = kThreads * U;
  static constexpr int kA = R::kAlign;
  // A chunk-piece may end in a partial vector, which either the vector loops
  // take (kTail) or work items of its own (kItems; the bf16 op, which the
  // in-loop form grows past what the compiler keeps in registers).
  static constexpr bool kTail = R::kPartial && !R::kPartialItems;
  static constexpr bool kItems = R::kPartial && R::kPartialItems;
  static_assert(!R::kPartial || sizeof(acc_t) == 16, "relaxed reduce-scatter vectors hold 4 elements");

  struct Edge {
    const char* child;
    const char* own;
    char* dst;
    bool child_in;   // child is a leaf: its raw input
    bool own_in;     // first receive: the own raw input
    bool dst_final;  // root's last receive (bf16): store rounded to the receive buffer
  };

  __device__ static Edge edge(const KCtx& cx, const DevStep& st, int r, int i) {
    return edge_of(cx, st, r, cx.entries[st.entry0 + i]);
  }

  __device__ static Edge edge_of(const KCtx& cx, const DevStep& st, int r, const DevEntry& en) {
    const int c = wrap_sub(r, en.p, cx.N);
    const int child = wrap_add(r, st.d, cx.N);
    const int64_t uoff = (c * cx.count + st.e0) * R::kInElem;
    // Pointer-table reads happen whether or not the edge uses them, so that
    // none of them sits in a branch of its own (and waits there).
    const char* send_child = (const char*)cx.send[child];
    const char* send_r = (const char*)cx.send[r];
    char* const recv_r = (char*)cx.recv[r] + st.e0 * R::kInElem;
    char* const root_acc =
        R::kSeparateRoot ? cx.rootacc + st.half * cx.root_half_bytes + r * cx.rootacc_stride : recv_r;
    char* const slots = cx.slots + st.half * cx.slot_half_bytes;
    char* const slots_r = slots + r * cx.slot_rank_stride;
    Edge e;
    e.child_in = en.a == kUser;
    e.child = e.child_in ? send_child + uoff : slots + child * cx.slot_rank_stride + en.a * cx.slot_chunk_stride;
    e.own_in = en.b == kUser;
    e.own = e.own_in ? send_r + uoff : en.b == kRoot ? root_acc : slots_r + en.b * cx.slot_chunk_stride;
    e.dst_final = R::kSeparateRoot && en.c == kRootFinal;
    e.dst = en.c >= 0 ? slots_r + en.c * cx.slot_chunk_stride : e.dst_final ? recv_r : root_acc;
    return e;
  }

  // int32 and float32: a raw input vector and an accumulator vector are alike.
  static constexpr bool kSameVec = std::is_same<in_t, acc_t>::value;

  template <bool RAW>
  using vec_t = typename std::conditional<RAW, in_t, acc_t>::type;

  template <bool RAW>
  __device__ static acc_t to_acc(const vec_t<RAW>& x) {
    if constexpr (RAW)
      return R::widen(x);
    else
      return x;
  }

  // Byte offset of vector v (of type X, 4 elements) in a chunk-piece of V
  // vectors: a partial last vector is moved back by `back` elements so that
  // it ends where the piece ends.  Its loads then cover the tail of the
  // vector before it (values it does not store), its stores only its own
  // elements.
  template <typename X>
  __device__ static int64_t off(int64_t v, int64_t V, int back) {
    int64_t o = v * (int64_t)sizeof(X);
    if constexpr (kTail)
      if (v == V - 1) o -= back * (int64_t)(sizeof(X) / 4);
    return o;
  }

  __device__ static void store(const Edge& e, int64_t v, int64_t V, int back, const acc_t& x) {
    if constexpr (kTail) {
      if (back && v == V - 1) {
        if (e.dst_final)
          stg_from<NT, sizeof(in_t) / 4>(e.dst + off<in_t>(v, V, back), R::narrow(x), back);
        else
          stg_from<NT, 4>(e.dst + off<acc_t>(v, V, back), x, back);
        return;
      }
    }
    if (e.dst_final)
      stg<NT, kA>(e.dst + v * (int64_t)sizeof(in_t), R::narrow(x));
    else
      stg<NT, kA>(e.dst + v * (int64_t)sizeof(acc_t), x);
  }

  // One edge's partial last vector as a work item of its own (kItems): the
  // piece's last 4 elements, which begin st.back elements inside its last
  // whole vector (st.V counts whole vectors only); only the elements past
  // that vector are stored.
  __device__ static void part(const DevStep& st, const Edge& e) {
    const int64_t in_off = st.V * (int64_t)sizeof(in_t) - st.back * (int64_t)(sizeof(in_t) / 4);
    const int64_t acc_off = st.V * (int64_t)sizeof(acc_t) - st.back * (int64_t)(sizeof(acc_t) / 4);
    acc_t a, b;
    if constexpr (kSameVec) {
      a = ldg<acc_t, NT, kA>(e.own + acc_off);
      b = ldg<acc_t, NT, kA>(e.child + acc_off);
    } else {
      if (e.own_in)
        a = R::widen(ldg<in_t, NT, kA>(e.own + in_off));
      else
        a = ldg<acc_t, NT, kA>(e.own + acc_off);
      if (e.child_in)
        b = R::widen(ldg<in_t, NT, kA>(e.child + in_off));
      else
        b = ldg<acc_t, NT, kA>(e.child + acc_off);
    }
    const acc_t sum = R::add(a, b);
    if (e.dst_final)
      stg_from<NT, sizeof(in_t) / 4>(e.dst + in_off, R::narrow(sum), st.back);
    else
      stg_from<NT, 4>(e.dst + acc_off, sum, st.back);
  }

  // One tile of one edge whose operand kinds are known: every load is issued
  // before any value is used, so a lane keeps 2U loads in flight (a raw bf16
  // input widened right after its load would wait for each load in turn).
  template <bool OWN_RAW, bool CHILD_RAW>
  __device__ static void tile(const Edge& e, int64_t tile_idx, int64_t V, int back) {
    vec_t<OWN_RAW> a[TU];
    vec_t<CHILD_RAW> b[TU];
    const int64_t v0 = tile_idx * kTile + threadIdx.x;
    const int64_t whole = kTail && back ? V - 1 : V;  // vectors the straight-line code may take
    if ((tile_idx + 1) * kTile <= whole) {
      // Full tile (uniform): straight-line code, no per-lane guards.
#pragma unroll
      for (int j = 0; j < TU; ++j) {
        const int64_t v = v0 + j * kThreads;
        a[j] = ldg<vec_t<OWN_RAW>, NT, kA>(e.own + v * (int64_t)sizeof(vec_t<OWN_RAW>));
        b[j] = ldg<vec_t<CHILD_RAW>, NT, kA>(e.child + v * (int64_t)sizeof(vec_t<CHILD_RAW>));
      }
      acc_t sum[TU];
#pragma unroll
      for (int j = 0; j < TU; ++j) sum[j] = R::add(to_acc<OWN_RAW>(a[j]), to_acc<CHILD_RAW>(b[j]));
      if (R::kSeparateRoot && e.dst_final) {
#pragma unroll
        for (int j = 0; j < TU; ++j)
          stg<NT, kA>(e.dst + (v0 + j * kThreads) * (int64_t)sizeof(in_t), R::narrow(sum[j]));
      } else {
#pragma unroll
        for (int j = 0; j < TU; ++j) stg<NT, kA>(e.dst + (v0 + j * kThreads) * (int64_t)sizeof(acc_t), sum[j]);
      }
      return;
    }
#pragma unroll
    for (int j = 0; j < TU; ++j) {
      const int64_t v = v0 + j * kThreads;
      if (v < V) {
        a[j] = ldg<vec_t<OWN_RAW>, NT, kA>(e.own + off<vec_t<OWN_RAW>>(v, V, back));
        b[j] = ldg<vec_t<CHILD_RAW>, NT, kA>(e.child + off<vec_t<CHILD_RAW>>(v, V, back));
      }
    }
    acc_t sum[TU];
#pragma unroll
    for (int j = 0; j < TU; ++j)
      if (v0 + j * kThreads < V) sum[j] = R::add(to_acc<OWN_RAW>(a[j]), to_acc<CHILD_RAW>(b[j]));
#pragma unroll
    for (int j = 0; j < TU; ++j) {
      const int64_t v = v0 + j * kThreads;
      if (v < V) store(e, v, V, back, sum[j]);
    }
  }

  __device__ static void run(const KCtx& cx, const DevStep& st, int64_t item) {
    if constexpr (kItems) {
      const int64_t main = main_items(cx, st);
      if (item >= main) {  // one lane per edge: its partial last vector
        const int64_t g = (item - main) * kThreads + threadIdx.x;
        if (g < (int64_t)cx.N * st.k) {
          const int r = (int)(g / st.k);
          part(st, edge(cx, st, r, (int)(g - (int64_t)r * st.k)));
        }
        return;
      }
    }
    if (st.tiles_per_edge > 0) {
      int r, i;
      int64_t tile_idx;
      split_tile(item, st, &r, &i, &tile_idx);
      const Edge e = edge(cx, st, r, i);
      if constexpr (kSameVec) {
        tile<false, false>(e, tile_idx, st.V, st.back);
      } else if (e.own_in) {
        if (e.child_in)
          tile<true, true>(e, tile_idx, st.V, st.back);
        else
          tile<true, false>(e, tile_idx, st.V, st.back);
      } else {
        if (e.child_in)
          tile<false, true>(e, tile_idx, st.V, st.back);
        else
          tile<false, false>(e, tile_idx, st.V, st.back);
      }
    } else {
      const int64_t units = (int64_t)cx.N * st.k * st.V;
      const bool small = units < (int64_t(1) << 31);
      int rr[U], ii[U];
      int64_t vv[U];
#pragma unroll
      for (int j = 0; j < U; ++j) {
        const int64_t g = item * kPackTile + j * kThreads + threadIdx.x;
        vv[j] = -1;
        if (g < units) split_flat(g, st, &rr[j], &ii[j], &vv[j], small);
      }
      batch<false>(cx, st, rr, ii, vv);
    }
  }

  // U vectors per lane, each given as (rank, entry, vector), or (tree, entry,
  // vector) when TREE (the acting rank is then tree + the entry's position);
  // vv[j] < 0 marks an unused slot.  Each lane's vectors may belong to
  // different edges, so both kinds of load are predicated per lane.  In phases
  // (entries, then pointer tables, then data), so that each level of
  // dependent loads is in flight for all U vectors at once; conversions come
  // after every load has been issued.
  // CACHED: the edges of entries ii[] are at cached[ii[j]] (LDS).
  template <bool TREE, bool CACHED = false>
  __device__ static void batch(const KCtx& cx, const DevStep& st, const int (&rr)[U], const int (&ii)[U],
                               const int64_t (&vv)[U], const Edge* cached = nullptr) {
    Edge e[U];
    in_t ra[U], rb[U];
    acc_t xa[U], xb[U];
    if constexpr (CACHED) {
#pragma unroll
      for (int j = 0; j < U; ++j)
        if (vv[j] >= 0) e[j] = cached[ii[j]];
    } else {
      DevEntry en[U];
#pragma unroll
      for (int j = 0; j < U; ++j)
        if (vv[j] >= 0) en[j] = cx.entries[st.entry0 + ii[j]];
#pragma unroll
      for (int j = 0; j < U; ++j)
        if (vv[j] >= 0) e[j] = edge_of(cx, st, TREE ? wrap_add(rr[j], en[j].p, cx.N) : rr[j], en[j]);
    }
#pragma unroll
    for (int j = 0; j < U; ++j) {
      if (vv[j] >= 0) {
        if constexpr (kSameVec) {
          xa[j] = ldg<acc_t, NT, kA>(e[j].own + off<acc_t>(vv[j], st.V, st.back));
          xb[j] = ldg<acc_t, NT, kA>(e[j].child + off<acc_t>(vv[j], st.V, st.back));
        } else {
          if (e[j].own_in)
            ra[j] = ldg<in_t, NT, kA>(e[j].own + off<in_t>(vv[j], st.V, st.back));
          else
            xa[j] = ldg<acc_t, NT, kA>(e[j].own + off<acc_t>(vv[j], st.V, st.back));
          if (e[j].child_in)
            rb[j] = ldg<in_t, NT, kA>(e[j].child + off<in_t>(vv[j], st.V, st.back));
          else
            xb[j] = ldg<acc_t, NT, kA>(e[j].child + off<acc_t>(vv[j], st.V, st.back));
        }
      }
    }
    acc_t sum[U];
#pragma unroll
    for (int j = 0; j < U; ++j)
      if (vv[j] >= 0) {
        acc_t a = xa[j], b = xb[j];
        if constexpr (!kSameVec) {
          if (e[j].own_in) a = R::widen(ra[j]);
          if (e[j].child_in) b = R::widen(rb[j]);
        }
        sum[j] = R::add(a, b);
      }
    wait_loads();
#pragma unroll
    for (int j = 0; j < U; ++j)
      if (vv[j] >= 0) store(e[j], vv[j], st.V, st.back, sum[j]);
  }

  // Every edge of step st in tree c, over vectors [t0, t0 + TV) of the chunk;
  // with kItems the workgroup of the last tile also takes the edges' partial
  // vectors.
  template <bool CACHED>
  __device__ static void tree_step(const KCtx& cx, const DevStep& st, int c, int64_t t0, int64_t TV, bool last,
                                   const Edge* cached) {
    tree_step_impl<RsOp, CACHED>(cx, st, c, t0, TV, cached);
    if constexpr (kItems) {
      if (last && st.back) {
        for (int i = threadIdx.x; i < st.k; i += kTreeThreads) {
          if constexpr (CACHED) {
            part(st, cached[i]);
          } else {
            const DevEntry en = cx.entries[st.entry0 + i];
            part(st, edge_of(cx, st, wrap_add(c, en.p, cx.N), en));
          }
        }
      }
    }
  }
};

// ---------------------------------------------------------------------------
// Drivers
// ---------------------------------------------------------------------------

// One launch per step; the step descriptor comes by value with the launch.
// Work-item order: workgroups are dispatched to the 8 XCDs round-robin, and
// with grain g each XCD takes runs of g consecutive work items (consecutive
// tiles of an edge): workgroup b, on XCD x = b % 8 as its j-th = b / 8,
// takes item (j / g) * 8g + x * g + j % g.  g = 1 is the plain order (all
// XCDs sweep the same few edges together); g = ceil(items / 8) gives each XCD
// a contiguous eighth of the step.  The grid is a multiple of 8g.
template <class Op>
__global__ __launch_bounds__(kThreads) void step_kernel(KCtx cx, DevStep st, int64_t grain) {
  int64_t item = blockIdx.x, stride = gridDim.x;
  if (grain > 1) {
    const int64_t x = blockIdx.x % 8, j = blockIdx.x / 8;
    item = (j / grain) * 8 * grain + x * grain + j % grain;
    stride = st.items;  // at most one item per workgroup
  }
  // One call site for Op::run: a second inlined copy of the bf16 op pushed
  // the compiler into scratch memory.
  for (; item < st.items; item += stride) Op::run(cx, st, item);
}

// Two independent launch-level steps in one launch (pipelined pieces): the
// items of step ia, then those of step ib, read from the device step table
// (one call site for Op::run).  Work-item order as in step_kernel, over the
// launch's items.
template <class Op>
__global__ __launch_bounds__(kThreads) void step2_kernel(KCtx cx, int ia, int ib, int64_t na, int64_t total,
                                                         int64_t grain) {
  int64_t item = blockIdx.x, stride = gridDim.x;
  if (grain > 1) {
    const int64_t x = blockIdx.x % 8, j = blockIdx.x / 8;
    item = (j / grain) * 8 * grain + x * grain + j % grain;
    stride = total;  // at most one item per workgroup
  }
  for (; item < total; item += stride) {
    const bool first = item < na;
    const DevStep st = cx.steps[first ? ia : ib];
    Op::run(cx, st, first ? item : item - na);
  }
}

// Fused range of steps: one workgroup per (tree, tile of its chunk) runs the
// launch-level steps s0 .. s1 - 1 in order.  The range holds only steps whose
// slot entries each serve one tree (the top part; every step when the
// sub-trees span at most 4), so the data a step of tree c reads was written by an earlier step of
// tree c, over the same tile: by this workgroup.
// A workgroup barrier between steps then replaces the kernel boundary; each
// wave first waits for its own stores.
//
// With cx.stamps set (measurement only), lane 0 records the device wall clock
// before the first step and after each step's barrier (the last step gets a
// barrier of its own then), so that step k of this workgroup took
// stamps[k + 1] - stamps[k] ticks.
//
// The edges of the launch-level steps [tr.c0, tr.c1) (tr.cn of them, at most
// kTreeCacheEdges: the narrow end of the range) are resolved for this tree
// once into LDS: their entries and pointer tables do not change during the
// operation, so those steps then wait for one data round trip each instead
// of a chain of three.  Lane t resolves entry t, its step found from the
// kernel arguments, so the fill costs one chain of two loads; it runs at the
// start when the cached steps come first (all-gather), else during the last
// step before them (reduce-scatter), whose barrier then also covers it.
template <class Op>
__device__ __forceinline__ void fill_edge_cache(const KCtx& cx, const TreeRange& tr, int c,
                                                typename Op::Edge* cache) {
  for (int t = threadIdx.x; t < tr.cn; t += kTreeThreads) {
    int s = tr.c0;
#pragma unroll
    for (int i = 0; i < kTreeCacheSteps - 1; ++i)
      if (i < tr.c1 - tr.c0 - 1 && t >= tr.cend[i]) s = tr.c0 + i + 1;
    const DevStep st = cx.steps[s];
    const DevEntry en = cx.entries[tr.ce0 + t];
    cache[t] = Op::edge_of(cx, st, wrap_add(c, en.p, cx.N), en);
  }
}

template <class Op>
__global__ __launch_bounds__(kTreeThreads) void tree_kernel(KCtx cx, TreeRange tr) {
  __shared__ typename Op::Edge cache[kTreeCacheEdges];
  const int c = (int)(blockIdx.x / tr.tiles);
  const int64_t tile = (int64_t)blockIdx.x - (int64_t)c * tr.tiles;
  const int64_t t0 = tile * tr.tile_vecs;
  uint64_t* const stamp = cx.stamps ? cx.stamps + (int64_t)blockIdx.x * (tr.s1 - tr.s0 + 1) : nullptr;
  if (stamp && threadIdx.x == 0) stamp[0] = wall_clock64();
  const bool cached = tr.cn > 0 && tr.cn <= kTreeCacheEdges && tr.c1 - tr.c0 <= kTreeCacheSteps &&
                      tr.c0 >= tr.s0 && tr.c1 <= tr.s1 && tr.c0 < tr.c1;
  if (cached && tr.c0 == tr.s0) {
    fill_edge_cache<Op>(cx, tr, c, cache);
    __syncthreads();
  }
  int coff = 0;  // first cached edge of the current step
  for (int s = tr.s0; s < tr.s1; ++s) {
    const DevStep st = cx.steps[s];
    const int64_t left = st.V - t0;
    const bool hit = cached && s >= tr.c0 && s < tr.c1;
    const int64_t TV = left < tr.tile_vecs ? left : tr.tile_vecs;
    if (hit) {
      Op::template tree_step<true>(cx, st, c, t0, TV, tile == tr.tiles - 1, cache + coff);
      coff += st.k;
    } else {
      Op::template tree_step<false>(cx, st, c, t0, TV, tile == tr.tiles - 1, nullptr);
    }
    if (cached && s + 1 == tr.c0) fill_edge_cache<Op>(cx, tr, c, cache);  // c0 > s0: the barrier follows
    if (s + 1 < tr.s1 || stamp) {
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
      if (stamp && threadIdx.x == 0) stamp[s - tr.s0 + 1] = wall_clock64();
    }
  }
}

// Persistent execution: one launch per operation.  Step s has
// G_s = min(grid, items_s) worker ids; a workgroup takes the next id of its
// current step and processes items id, id + G_s, ...  Once every id of the
// step has been taken it moves to the next step.  Before working on step s it
// waits until all G_{s-1} ids of step s - 1 are done; step s - 1 done implies
// every earlier step done, so each step sees exactly what a kernel boundary
// would give it.
//
// No co-residency is needed: a workgroup enters step s only after every id of
// step s - 1 was taken by a running workgroup, and those depend only on
// earlier steps, so by induction over the steps all work completes whatever
// the grid size.  The launch is a plain one; the host sizes its grid.
//
// Counters are spread over kShards cache lines per step: atomics on a single
// address serialise (about 11 ns each on MI355X, 20 us for one round of 1792
// workgroups), spread ones do not.  Id j*kShards + h lives in shard h; a
// workgroup takes ids from shard blockIdx % kShards and, when that shard is
// empty, looks at all shards before declaring the step fully taken.  An id
// done counts in its shard's done counter; whoever completes a shard counts
// it in the step's counter, so a step is done when that single word reaches
// the number of non-empty shards, and waiters poll one word.
//
// Memory ordering across the XCDs' separate L2 caches:
//  - finishing an id: every wave waits for its own stores (a workgroup
//    barrier does not), then one thread counts the id done with an
//    agent-scope release (one write-back of this XCD's L2); the shard's
//    completer reads its counter with acquire, so its release on the step
//    counter covers every id of the shard;
//  - entering a step: one thread polls the previous step's counter, then
//    takes an agent-scope acquire (invalidates this CU's L1 and stale L2
//    lines) before a workgroup barrier lets the other waves load.
// Every wait has a wall-clock limit; past it the status bit is set and the
// workgroup stops (the operation's result is then undefined).  The last
// workgroup out returns every counter to zero for the next launch.
constexpr int kShards = 32;
constexpr int kLineWords = 32;  // one 128-byte line per counter

// Counter lines: [0, S*kShards) ids taken, [S*kShards, 2*S*kShards) ids done,
// [2*S*kShards, 2*S*kShards + S) shards done per step, S = nsteps.
__device__ __forceinline__ unsigned* queue_line(const KCtx& cx, int64_t line) {
  return cx.queue + 4 + line * kLineWords;
}
__device__ __forceinline__ unsigned* taken_ctr(const KCtx& cx, int s, int h) {
  return queue_line(cx, (int64_t)s * kShards + h);
}
__device__ __forceinline__ unsigned* done_ctr(const KCtx& cx, int s, int h) {
  return queue_line(cx, ((int64_t)cx.nsteps + s) * kShards + h);
}
__device__ __forceinline__ unsigned* step_ctr(const KCtx& cx, int s) {
  return queue_line(cx, 2 * (int64_t)cx.nsteps * kShards + s);
}
__device__ __forceinline__ int64_t shard_ids(int64_t G, int h) {
  return G > h ? (G - h + kShards - 1) / kShards : 0;
}
__device__ __forceinline__ int64_t step_ids(const KCtx& cx, int s) {
  const int64_t items = cx.steps[s].items;
  return items < (int64_t)gridDim.x ? items : (int64_t)gridDim.x;
}

struct QueueShared {
  int64_t id;
  int flag;
  unsigned vals[kShards];
};

// Next worker id of step s for this workgroup, or -1 once every id of the
// step has been taken.  Called by all threads; the result is uniform.
__device__ int64_t take_id(const KCtx& cx, int s, int64_t G, QueueShared* q) {
  if (threadIdx.x == 0) {
    const int h = blockIdx.x % kShards;
    const unsigned j = __hip_atomic_fetch_add(taken_ctr(cx, s, h), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    q->id = (int64_t)j < shard_ids(G, h) ? (int64_t)j * kShards + h : -1;
  }
  __syncthreads();
  int64_t id = q->id;
  __syncthreads();
  while (id == -1) {
    if (threadIdx.x < kShards)
      q->vals[threadIdx.x] = __hip_atomic_load(taken_ctr(cx, s, threadIdx.x), __ATOMIC_RELAXED,
                                               __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    if (threadIdx.x == 0) {
      int64_t got = -2;  // every shard empty
      for (int h = 0; h < kShards; ++h) {
        if ((int64_t)q->vals[h] >= shard_ids(G, h)) continue;
        const unsigned j = __hip_atomic_fetch_add(taken_ctr(cx, s, h), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if ((int64_t)j < shard_ids(G, h)) {
          got = (int64_t)j * kShards + h;
          break;
        }
        got = -1;  // lost a race for that shard: look again
      }
      q->id = got;
    }
    __syncthreads();
    id = q->id;
    __syncthreads();
  }
  return id < 0 ? -1 : id;
}

// Thread 0 counts worker id `id` of step s done.
__device__ __forceinline__ void finish_id(const KCtx& cx, int s, int64_t G, int64_t id) {
  const int h = (int)(id % kShards);
  const unsigned before = __hip_atomic_fetch_add(done_ctr(cx, s, h), 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
  if ((int64_t)before + 1 == shard_ids(G, h))
    __hip_atomic_fetch_add(step_ctr(cx, s), 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}

// Waits until every id of step s is done.  Returns false on timeout.
__device__ bool wait_step(const KCtx& cx, int s, QueueShared* q) {
  if (threadIdx.x == 0) {
    const int64_t G = step_ids(cx, s);
    const unsigned need = (unsigned)(G < kShards ? G : kShards);
    const long long t0 = wall_clock64();
    int f = 0;
    for (;;) {
      if (__hip_atomic_load(step_ctr(cx, s), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= need) {
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        f = 1;
        break;
      }
      if (wall_clock64() - t0 > cx.timeout_ticks) {
        __hip_atomic_fetch_or(cx.status, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        f = -1;
        break;
      }
      __builtin_amdgcn_s_sleep(2);
    }
    q->flag = f;
  }
  __syncthreads();
  const int f = q->flag;
  __syncthreads();
  return f > 0;
}

template <class Op>
__global__ __launch_bounds__(kThreads) void persistent_kernel(KCtx cx) {
  __shared__ QueueShared q;
  int ready = 0;  // steps before `ready` are known done
  for (int s = 0; s < cx.nsteps;) {
    const DevStep st = cx.steps[s];
    const int64_t G = step_ids(cx, s);
    const int64_t w = take_id(cx, s, G, &q);
    if (w < 0) {
      ++s;  // every id of this step is taken
      continue;
    }
    if (s > ready) {
      if (!wait_step(cx, s - 1, &q)) break;
      ready = s;
    }
    for (int64_t item = w; item < st.items; item += G) Op::run(cx, st, item);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0) finish_id(cx, s, G, w);
  }
  // Leave the counters at zero: the last workgroup out (every other one has
  // finished all of its work by then) resets them.
  __syncthreads();
  if (threadIdx.x == 0)
    q.flag = (__hip_atomic_fetch_add(&cx.queue[1], 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT) + 1u == gridDim.x);
  __syncthreads();
  if (q.flag) {
    const int64_t n = (2 * (int64_t)kShards + 1) * cx.nsteps;
    for (int64_t k = threadIdx.x; k < n; k += blockDim.x)
      __hip_atomic_store(queue_line(cx, k), 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0) __hip_atomic_store(&cx.queue[1], 0u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// Dataflow execution (one launch per piece).  The work queue is the
// persistent kernel's: per step, worker ids taken in step order from sharded
// counters, each id running items id, id + G, ...  A work item is either a
// group of up to kThreads whole edges (chunks under one tile: lanes sweep
// their vectors as the packed path does) or a run of tiles of one edge.
// Instead of waiting for the whole previous step, an item waits until the
// two buffers each of its edges touches have seen every earlier access of the
// schedule complete: a per-(rank, buffer) counter must reach need * (the
// count one edge adds): every edge adds its tiles (1 for whole edges) to both
// of its counters as its items complete, so the unit is the same for every
// step of a launch, however the steps split their edges into items.  Items wait only on items of earlier steps, which
// running workgroups hold because ids are taken in step order, so the work
// always completes whatever the grid size.
//
// Ordering across the XCDs' separate L2 caches: each wave waits for its own
// stores, a workgroup barrier, then the lanes of one wave -- lane t for edge t
// of the item -- add with agent-scope release (one cache write-back per
// wave); waiting lanes poll with relaxed agent-scope loads and take an
// agent-scope acquire before the barrier that lets the other waves load.
// Every wait is bounded by the wall-clock limit (then the status bit is set
// and the workgroup stops; the result is undefined).  The last workgroup out
// zeroes the queue and the buffer counters.

// Ranks of an edge's two counters (DevDep).
template <class Op>
__device__ __forceinline__ void dep_ranks(const KCtx& cx, const DevStep& st, int r, int* x1, int* x2) {
  *x1 = Op::kGather ? r : wrap_add(r, st.d, cx.N);
  *x2 = Op::kGather ? wrap_add(r, st.d, cx.N) : r;
}

// Lane t < nedges waits for the counters of edge e0 + t to reach `unit`
// times their need (unit: the counts one edge adds when it completes, the
// same for every step of a launch).  Returns false (uniformly) on a timeout.
template <class Op>
__device__ bool wait_edges(const KCtx& cx, const DevStep& st, int nedges, int64_t e0, int64_t unit,
                           QueueShared* q) {
  if (threadIdx.x == 0) q->flag = 1;
  __syncthreads();
  if (threadIdx.x < nedges) {
    const int64_t e = e0 + threadIdx.x;
    const int r = (int)(e / st.k), i = (int)(e - (int64_t)r * st.k);
    const DevDep g = cx.deps[st.entry0 + i];
    int x1, x2;
    dep_ranks<Op>(cx, st, r, &x1, &x2);
    const unsigned t1 = (unsigned)(g.need1 * unit), t2 = (unsigned)(g.need2 * unit);
    unsigned* c1 = g.e1 >= 0 && t1 ? cx.counters + x1 * cx.counter_stride + g.e1 : nullptr;
    unsigned* c2 = g.e2 >= 0 && t2 ? cx.counters + x2 * cx.counter_stride + g.e2 : nullptr;
    if (c1 || c2) {
      const long long t0 = wall_clock64();
      for (;;) {
        const bool ok1 = !c1 || __hip_atomic_load(c1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= t1;
        const bool ok2 = !c2 || __hip_atomic_load(c2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= t2;
        if (ok1 && ok2) break;
        if (wall_clock64() - t0 > cx.timeout_ticks) {
          __hip_atomic_fetch_or(cx.status, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          q->flag = 0;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    }
  }
  __syncthreads();
  const int f = q->flag;
  __syncthreads();
  return f != 0;
}

// After the item's stores: lane t < nedges adds `amount` (the tiles of edge
// e0 + t the item completed) to both of that edge's counters.
template <class Op>
__device__ __forceinline__ void signal_edges(const KCtx& cx, const DevStep& st, int nedges, int64_t e0,
                                             unsigned amount) {
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x < nedges) {
    const int64_t e = e0 + threadIdx.x;
    const int r = (int)(e / st.k), i = (int)(e - (int64_t)r * st.k);
    const DevDep g = cx.deps[st.entry0 + i];
    int x1, x2;
    dep_ranks<Op>(cx, st, r, &x1, &x2);
    if (g.e1 >= 0)
      __hip_atomic_fetch_add(cx.counters + x1 * cx.counter_stride + g.e1, amount, __ATOMIC_RELEASE,
                             __HIP_MEMORY_SCOPE_AGENT);
    if (g.e2 >= 0)
      __hip_atomic_fetch_add(cx.counters + x2 * cx.counter_stride + g.e2, amount, __ATOMIC_RELEASE,
                             __HIP_MEMORY_SCOPE_AGENT);
  }
}

// SMALL: every step of the launch is packed (chunks under one tile) and an
// item is df_edges whole edges; otherwise every step is tiled and an item is
// df_tiles tiles of one edge.
template <class Op, bool SMALL>
__global__ __launch_bounds__(kThreads) void dataflow_kernel(KCtx cx) {
  __shared__ QueueShared q;
  bool ok = true;
  for (int s = 0; s < cx.nsteps && ok;) {
    const DevStep st = cx.steps[s];
    const int64_t G = step_ids(cx, s);
    const int64_t w = take_id(cx, s, G, &q);
    if (w < 0) {
      ++s;  // every id of this step is taken
      continue;
    }
    const int64_t edges = (int64_t)cx.N * st.k;
    for (int64_t item = w; item < st.items; item += G) {
      if constexpr (SMALL) {
        const int64_t e0 = item * st.df_edges;
        const int ne = (int)(edges - e0 < st.df_edges ? edges - e0 : st.df_edges);
        if (!wait_edges<Op>(cx, st, ne, e0, 1, &q)) {
          ok = false;
          break;
        }
        constexpr int U = Op::U;
        const int64_t nv = (int64_t)ne * st.V;
        for (int64_t base = 0; base < nv; base += (int64_t)kThreads * U) {
          int rr[U], ii[U];
          int64_t vv[U];
#pragma unroll
          for (int j = 0; j < U; ++j) {
            const int64_t f = base + j * kThreads + threadIdx.x;
            vv[j] = -1;
            rr[j] = 0;
            ii[j] = 0;
            if (f < nv) {
              const int64_t e = e0 + f / st.V;
              rr[j] = (int)(e / st.k);
              ii[j] = (int)(e - (int64_t)rr[j] * st.k);
              vv[j] = f - (f / st.V) * st.V;
            }
          }
          Op::template batch<false>(cx, st, rr, ii, vv);
        }
        signal_edges<Op>(cx, st, ne, e0, 1u);
      } else {
        const int64_t per_edge = (st.tiles_per_edge + st.df_tiles - 1) / st.df_tiles;
        const int64_t e = item / per_edge;
        const int64_t t0 = (item - e * per_edge) * st.df_tiles;
        const int64_t t1 = t0 + st.df_tiles < st.tiles_per_edge ? t0 + st.df_tiles : st.tiles_per_edge;
        if (!wait_edges<Op>(cx, st, 1, e, st.tiles_per_edge, &q)) {
          ok = false;
          break;
        }
        for (int64_t t = t0; t < t1; ++t) Op::run(cx, st, e * st.tiles_per_edge + t);
        signal_edges<Op>(cx, st, 1, e, (unsigned)(t1 - t0));
      }
    }
  }
  // Leave the queue and the counters at zero: the last workgroup out (every
  // other one has finished all of its work by then) resets them.
  __syncthreads();
  if (threadIdx.x == 0)
    q.flag = (__hip_atomic_fetch_add(&cx.queue[1], 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT) + 1u == gridDim.x);
  __syncthreads();
  if (q.flag) {
    const int64_t n = (2 * (int64_t)kShards + 1) * cx.nsteps;
    for (int64_t k = threadIdx.x; k < n; k += blockDim.x)
      __hip_atomic_store(queue_line(cx, k), 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int64_t nc = (int64_t)cx.N * cx.counter_stride;
    for (int64_t k = threadIdx.x; k < nc; k += blockDim.x)
      __hip_atomic_store(cx.counters + k, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0) __hip_atomic_store(&cx.queue[1], 0u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
  }
}

template <class Op>
hipError_t launch_dataflow_t(const KCtx& cx, bool small, int grid, hipStream_t stream) {
  if (small)
    hipLaunchKernelGGL((dataflow_kernel<Op, true>), dim3(grid), dim3(kThreads), 0, stream, cx);
  else
    hipLaunchKernelGGL((dataflow_kernel<Op, false>), dim3(grid), dim3(kThreads), 0, stream, cx);
  return hipGetLastError();
}

template <class Op>
hipError_t launch_step_t(const KCtx& cx, const DevStep& st, int64_t grain, hipStream_t stream) {
  const int64_t items = st.items;
  if (items <= 0) return hipSuccess;
  const int64_t cap = int64_t(1) << 30;
  unsigned grid = (unsigned)(items < cap ? items : cap);
  if (grain > 1) {
    grain = grain < (items + 7) / 8 ? grain : (items + 7) / 8;  // beyond a contiguous eighth is the same
    const int64_t run = 8 * grain;
    const int64_t g = (items + run - 1) / run * run;
    if (g <= cap)
      grid = (unsigned)g;  // every workgroup gets at most one item
    else
      grain = 1;  // beyond one grid the plain order strides over the items
  }
  hipLaunchKernelGGL(step_kernel<Op>, dim3(grid), dim3(kThreads), 0, stream, cx, st, grain);
  return hipGetLastError();
}

template <class Op>
hipError_t launch_step2_t(const KCtx& cx, int ia, int64_t na, int ib, int64_t nb, int64_t grain, hipStream_t stream) {
  const int64_t items = na + nb;
  if (items <= 0) return hipSuccess;
  const int64_t cap = int64_t(1) << 30;
  unsigned grid = (unsigned)(items < cap ? items : cap);
  if (grain > 1) {
    grain = grain < (items + 7) / 8 ? grain : (items + 7) / 8;
    const int64_t run = 8 * grain;
    const int64_t g = (items + run - 1) / run * run;
    if (g <= cap)
      grid = (unsigned)g;
    else
      grain = 1;
  }
  hipLaunchKernelGGL(step2_kernel<Op>, dim3(grid), dim3(kThreads), 0, stream, cx, ia, ib, na, items, grain);
  return hipGetLastError();
}

template <class Op>
hipError_t launch_persistent_t(const KCtx& cx, int grid, hipStream_t stream) {
  hipLaunchKernelGGL(persistent_kernel<Op>, dim3(grid), dim3(kThreads), 0, stream, cx);
  return hipGetLastError();
}

template <class Op>
hipError_t capacity_t(int* blocks) {
  int dev = 0, per_cu = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, persistent_kernel<Op>, kThreads, 0);
  if (e != hipSuccess) return e;
  *blocks = per_cu * cus;
  return hipSuccess;
}

#define PAT_DISPATCH(v, NT, CALL)                                           \
  switch (v) {                                                              \
    case kAgVec: return NT ? CALL((AgOp<v4u, PAT_UNROLL, true>)) : CALL((AgOp<v4u, PAT_UNROLL, false>)); \
    case kAgS4: return NT ? CALL((AgOp<uint32_t, kSU, true, kSTU>)) : CALL((AgOp<uint32_t, kSU, false, kSTU>)); \
    case kAgS2: return NT ? CALL((AgOp<uint16_t, kSU, true, kSTU>)) : CALL((AgOp<uint16_t, kSU, false, kSTU>)); \
    case kRsI32Vec: return NT ? CALL((RsOp<TI32V, true>)) : CALL((RsOp<TI32V, false>));                  \
    case kRsF32Vec: return NT ? CALL((RsOp<TF32V, true>)) : CALL((RsOp<TF32V, false>));                  \
    case kRsB16Vec: return NT ? CALL((RsOp<TB16V, true>)) : CALL((RsOp<TB16V, false>));                  \
    case kRsI32S: return NT ? CALL((RsOp<TI32S, true>)) : CALL((RsOp<TI32S, false>));                    \
    case kRsF32S: return NT ? CALL((RsOp<TF32S, true>)) : CALL((RsOp<TF32S, false>));                    \
    case kRsB16S: return NT ? CALL((RsOp<TB16S, true>)) : CALL((RsOp<TB16S, false>));                    \
    case kAgVecU: return NT ? CALL((AgOp<v4u, PAT_UNROLL, true, PAT_UNROLL, 2>)) : CALL((AgOp<v4u, PAT_UNROLL, false, PAT_UNROLL, 2>)); \
    case kRsI32VecU: return NT ? CALL((RsOp<TI32U, true>)) : CALL((RsOp<TI32U, false>));                \
    case kRsF32VecU: return NT ? CALL((RsOp<TF32U, true>)) : CALL((RsOp<TF32U, false>));                \
    case kRsB16VecU: return NT ? CALL((RsOp<TB16U, true>)) : CALL((RsOp<TB16U, false>));                \
    default: return hipErrorInvalidValue;                                   \
  }

}  // namespace

int variant_in_bytes(Variant v) {
  switch (v) {
    case kAgVec:
    case kRsI32Vec:
    case kRsF32Vec:
    case kAgVecU:
    case kRsI32VecU:
    case kRsF32VecU: return 16;
    case kRsB16Vec:
    case kRsB16VecU: return 8;
    case kAgS4:
    case kRsI32S:
    case kRsF32S: return 4;
    case kAgS2:
    case kRsB16S: return 2;
    default: return 0;
  }
}

bool variant_partial(Variant v) { return v == kAgVecU || v == kRsI32VecU || v == kRsF32VecU || v == kRsB16VecU; }
bool variant_partial_items(Variant v) { return v == kRsB16VecU; }

int variant_tile(Variant v) {
  switch (v) {
    case kAgVec: return AgOp<v4u, PAT_UNROLL, true>::kTile;
    case kAgS4: return AgOp<uint32_t, kSU, true, kSTU>::kTile;
    case kAgS2: return AgOp<uint16_t, kSU, true, kSTU>::kTile;
    case kRsI32Vec: return RsOp<TI32V, true>::kTile;
    case kRsF32Vec: return RsOp<TF32V, true>::kTile;
    case kRsB16Vec: return RsOp<TB16V, true>::kTile;
    case kRsI32S: return RsOp<TI32S, true>::kTile;
    case kRsF32S: return RsOp<TF32S, true>::kTile;
    case kRsB16S: return RsOp<TB16S, true>::kTile;
    case kAgVecU: return AgOp<v4u, PAT_UNROLL, true, PAT_UNROLL, 2>::kTile;
    case kRsI32VecU: return RsOp<TI32U, true>::kTile;
    case kRsF32VecU: return RsOp<TF32U, true>::kTile;
    case kRsB16VecU: return RsOp<TB16U, true>::kTile;
    default: return 0;
  }
}

int variant_pack_tile(Variant v) {
  switch (v) {
    case kAgVec: return AgOp<v4u, PAT_UNROLL, true>::kPackTile;
    case kAgS4: return AgOp<uint32_t, kSU, true, kSTU>::kPackTile;
    case kAgS2: return AgOp<uint16_t, kSU, true, kSTU>::kPackTile;
    case kRsI32Vec: return RsOp<TI32V, true>::kPackTile;
    case kRsF32Vec: return RsOp<TF32V, true>::kPackTile;
    case kRsB16Vec: return RsOp<TB16V, true>::kPackTile;
    case kRsI32S: return RsOp<TI32S, true>::kPackTile;
    case kRsF32S: return RsOp<TF32S, true>::kPackTile;
    case kRsB16S: return RsOp<TB16S, true>::kPackTile;
    case kAgVecU: return AgOp<v4u, PAT_UNROLL, true, PAT_UNROLL, 2>::kPackTile;
    case kRsI32VecU: return RsOp<TI32U, true>::kPackTile;
    case kRsF32VecU: return RsOp<TF32U, true>::kPackTile;
    case kRsB16VecU: return RsOp<TB16U, true>::kPackTile;
    default: return 0;
  }
}

#define PAT_UNPAREN(...) __VA_ARGS__

hipError_t launch_step(Variant v, bool streaming, int64_t grain, const KCtx& cx, const DevStep& st,
                       hipStream_t stream) {
#define PAT_STEP(OP) launch_step_t<PAT_UNPAREN OP>(cx, st, grain, stream)
  PAT_DISPATCH(v, streaming, PAT_STEP)
#undef PAT_STEP
}

hipError_t launch_step2(Variant v, bool streaming, int64_t grain, const KCtx& cx, int ia, const DevStep& a, int ib,
                        const DevStep& b, hipStream_t stream) {
#define PAT_STEP2(OP) launch_step2_t<PAT_UNPAREN OP>(cx, ia, a.items, ib, b.items, grain, stream)
  PAT_DISPATCH(v, streaming, PAT_STEP2)
#undef PAT_STEP2
}

template <class Op>
hipError_t launch_tree_t(const KCtx& cx, const TreeRange& tr, hipStream_t stream) {
  const int64_t grid = (int64_t)cx.N * tr.tiles;
  if (tr.s1 <= tr.s0 || grid <= 0) return hipSuccess;
  if (grid >= (int64_t(1) << 31) || tr.tile_vecs <= 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(tree_kernel<Op>, dim3((unsigned)grid), dim3(kTreeThreads), 0, stream, cx, tr);
  return hipGetLastError();
}

hipError_t launch_tree(Variant v, bool streaming, const KCtx& cx, const TreeRange& tr, hipStream_t stream) {
#define PAT_TREE(OP) launch_tree_t<PAT_UNPAREN OP>(cx, tr, stream)
  PAT_DISPATCH(v, streaming, PAT_TREE)
#undef PAT_TREE
}

hipError_t launch_persistent(Variant v, bool streaming, const KCtx& cx, int grid, hipStream_t stream) {
#define PAT_PERS(OP) launch_persistent_t<PAT_UNPAREN OP>(cx, grid, stream)
  PAT_DISPATCH(v, streaming, PAT_PERS)
#undef PAT_PERS
}

hipError_t launch_dataflow(Variant v, bool streaming, const KCtx& cx, bool small, int grid, hipStream_t stream) {
#define PAT_DF(OP) launch_dataflow_t<PAT_UNPAREN OP>(cx, small, grid, stream)
  PAT_DISPATCH(v, streaming, PAT_DF)
#undef PAT_DF
}

hipError_t persistent_capacity(Variant v, bool streaming, int* blocks) {
#define PAT_CAP(OP) capacity_t<PAT_UNPAREN OP>(blocks)
  PAT_DISPATCH(v, streaming, PAT_CAP)
#undef PAT_CAP
}

}  // namespace pat
