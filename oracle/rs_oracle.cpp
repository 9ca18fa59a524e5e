// Threaded CPU oracle of the PAT reduce-scatter (sum).
//
// TEST INFRASTRUCTURE ONLY.  Only tests/, __graft_entry__.smoke() and the
// cpu_baseline leg of bench.py load this library.  It shares no code, header,
// table or helper with the HIP library; the only header it includes from this
// repository is the seeded input generator (synth/synth_host.hpp), which holds
// none of the method's arithmetic.
//
// What it computes, for every destination chunk R and element i (section "All-
// gather and reduce-scatter algorithms" for the operation; section "Conversion
// to reduce-scatter operations" for the order of the additions):
//
//   O2  the plain sum over sending ranks, x = 0 .. N-1 in order, in double
//       (int32: the exact integer sum, which a wrapping int32 sum reduces
//       modulo 2^32), and the sum of absolute values, the scale of the
//       tolerance check;
//   O3  the sum in the PAT association: the reversed binomial tree of chunk R,
//       children added nearest first.  With v[q] the value of tree position q
//       (rank (R + q) mod N; all-gather data moves from r to r + d, so the
//       partials move from r + d to r) and L = ceil(log2 N):
//           S(lo, 1) = v[lo]
//           S(lo, w) = S(lo, w/2)                    if lo + w/2 >= N
//                    = S(lo, w/2) + S(lo + w/2, w/2) otherwise,
//       result S(0, 2^L).  The node at lo completes the half-span it keeps,
//       then adds the partial of its child at lo + w/2 -- the same closed form
//       as reversed_tree_sum in oracle/pat.py, evaluated here level by level
//       (spans 1, 2, 4, ...) instead of recursively.  Each add is one IEEE
//       float32 add, round to nearest even (int32: wraps modulo 2^32);
//       bfloat16 values are widened exactly and the float32 result is rounded
//       to bfloat16 once.  The association does not depend on the number of
//       parallel sub-trees or on pieces (far-first linear order).
//
// Inputs come either from an array (rank x's send buffer is row x of an
// [N][N * count] array) or from the seeded generator, regenerated element by
// element, so that a 64 GiB operation never has to sit in host memory.  Work
// is split over std::thread workers by (destination chunk, block of elements).
//
// Built with -ffp-contract=off and without fast-math: every float32 add is one
// rounding, and denormals are kept.
#include <sched.h>

#include <algorithm>
#include <atomic>
#include <cstdint>
#include <cstring>
#include <thread>
#include <vector>

#include "../synth/synth_host.hpp"

namespace {

enum : int { kInt32 = 0, kFloat32 = 1, kBfloat16 = 2 };

float as_float(uint32_t u) {
  float f;
  std::memcpy(&f, &u, 4);
  return f;
}

uint32_t as_bits(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  return u;
}

// float32 -> bfloat16, round to nearest, ties to even, written from the
// definition: keep the upper 16 bits, look at the 16 dropped ones, round up
// when they exceed half a unit, or equal it and the kept part is odd.  A carry
// out of the mantissa moves into the exponent, as it should (up to infinity).
// NaN stays NaN (quiet).
uint16_t bf16_nearest_even(float f) {
  const uint32_t u = as_bits(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return uint16_t((u >> 16) | 0x40u);
  uint32_t keep = u >> 16;
  const uint32_t dropped = u & 0xFFFFu;
  if (dropped > 0x8000u || (dropped == 0x8000u && (keep & 1u))) keep += 1;
  return uint16_t(keep);
}

struct Inputs {
  const void* array = nullptr;  // [N][N * count] raw elements, or null: the generator
  int64_t row_elems = 0;        // elements per row of the array
  int dtype = kFloat32;
  synth_host::Source gen;

  // Raw bits of elements [e0, e0 + n) of rank x's send buffer (bf16 in the
  // low half of each word).
  void row(int x, int64_t e0, int64_t n, uint32_t* out) const {
    if (!array) return gen.row(x, e0, n, out);
    const int64_t k = int64_t(x) * row_elems + e0;
    if (dtype == kBfloat16) {
      const uint16_t* p = static_cast<const uint16_t*>(array) + k;
      for (int64_t i = 0; i < n; ++i) out[i] = p[i];
    } else {
      std::memcpy(out, static_cast<const uint32_t*>(array) + k, size_t(n) * 4);
    }
  }
};

struct Job {
  Inputs in;
  int N = 0;
  int64_t count = 0;
  int r0 = 0, r1 = 0;
  int64_t block = 0;
  void* out_pat = nullptr;  // [r1 - r0][count]
  double* out_sum = nullptr;
  double* out_abs = nullptr;
};

// Per-thread work space.
struct Scratch {
  std::vector<uint32_t> v;  // [N][block]
  std::vector<double> s, a;  // [block]
};

// Destination chunk R, elements [i0, i1).
void run_item(const Job& j, int R, int64_t i0, int64_t i1, Scratch& w) {
  const int N = j.N;
  const int64_t B = i1 - i0;
  const int64_t out0 = int64_t(R - j.r0) * j.count + i0;
  uint32_t* v = w.v.data();
  double* s = w.s.data();
  double* a = w.a.data();
  std::fill(s, s + B, 0.0);
  std::fill(a, a + B, 0.0);
  // v[q * B + i]: the value of tree position q, as float32 bits (int32: the
  // integer bits).  Ranks are read in order x = 0 .. N-1, which is also the
  // order of the plain sum.
  for (int x = 0; x < N; ++x) {
    uint32_t* vq = v + int64_t((x - R + N) % N) * B;
    j.in.row(x, int64_t(R) * j.count + i0, B, vq);
    if (j.in.dtype == kInt32) {
      for (int64_t i = 0; i < B; ++i) {
        const double val = double(int32_t(vq[i]));
        s[i] += val;
        a[i] += val < 0 ? -val : val;
      }
    } else {
      if (j.in.dtype == kBfloat16)
        for (int64_t i = 0; i < B; ++i) vq[i] <<= 16;  // exact widening to float32
      for (int64_t i = 0; i < B; ++i) {
        const double val = double(as_float(vq[i]));
        s[i] += val;
        a[i] += val < 0 ? -val : val;
      }
    }
  }
  if (j.out_sum) std::memcpy(j.out_sum + out0, s, size_t(B) * sizeof(double));
  if (j.out_abs) std::memcpy(j.out_abs + out0, a, size_t(B) * sizeof(double));
  // The closed form, span by span: after the pass for `span`, position lo (a
  // multiple of 2 * span) holds S(lo, 2 * span).
  for (int span = 1; span < N; span *= 2) {
    for (int lo = 0; lo + span < N; lo += 2 * span) {
      uint32_t* dst = v + int64_t(lo) * B;
      const uint32_t* src = v + int64_t(lo + span) * B;
      if (j.in.dtype == kInt32) {
        for (int64_t i = 0; i < B; ++i) dst[i] = dst[i] + src[i];  // wraps modulo 2^32
      } else {
        for (int64_t i = 0; i < B; ++i) dst[i] = as_bits(as_float(dst[i]) + as_float(src[i]));
      }
    }
  }
  if (!j.out_pat) return;
  if (j.in.dtype == kBfloat16) {
    uint16_t* o = static_cast<uint16_t*>(j.out_pat) + out0;
    for (int64_t i = 0; i < B; ++i) o[i] = bf16_nearest_even(as_float(v[i]));
  } else {
    std::memcpy(static_cast<uint32_t*>(j.out_pat) + out0, v, size_t(B) * 4);
  }
}

int available_threads() {
  cpu_set_t set;
  if (sched_getaffinity(0, sizeof(set), &set) == 0) {
    const int n = CPU_COUNT(&set);
    if (n > 0) return n;
  }
  const unsigned h = std::thread::hardware_concurrency();
  return h ? int(h) : 1;
}

}  // namespace

extern "C" {

// Host threads the oracle uses by default: the CPUs this process may run on.
int oracle_threads(void) { return available_threads(); }

// Reduce-scatter (sum) expectations for destination chunks [r0, r1) of an
// N-rank operation with `count` elements per chunk.
//   inputs:  [N][N * count] raw elements (int32, float32, or bfloat16 bits), or
//            null to regenerate them with the seeded generator (kind, seed, lo,
//            span, table as in synth/synth_host.hpp);
//   dtype:   0 int32, 1 float32, 2 bfloat16;
//   out_pat: [r1 - r0][count] in the input dtype, the PAT association (O3), or null;
//   out_sum, out_abs: [r1 - r0][count] doubles (O2 and its absolute scale), or null;
//   threads: workers to use, <= 0 for every available CPU.
// Returns the number of threads used, or -1 for invalid arguments.
int oracle_reducescatter(const void* inputs, int kind, uint64_t seed, int64_t lo, uint64_t span,
                         const void* table, int nranks, int64_t count, int dtype, int r0, int r1,
                         void* out_pat, double* out_sum, double* out_abs, int threads) {
  if (nranks < 1 || count < 0 || dtype < kInt32 || dtype > kBfloat16) return -1;
  if (r0 < 0 || r1 > nranks || r0 > r1) return -1;
  if (!inputs && (kind < 0 || kind > 3 || (kind >= 2 && !table))) return -1;
  Job j;
  j.in.array = inputs;
  j.in.row_elems = int64_t(nranks) * count;
  j.in.dtype = dtype;
  j.in.gen.kind = kind;
  j.in.gen.seed = seed;
  j.in.gen.lo = lo;
  j.in.gen.span = span;
  j.in.gen.table = table;
  j.N = nranks;
  j.count = count;
  j.r0 = r0;
  j.r1 = r1;
  // Elements per work item: the block of N values stays within a few MiB.
  j.block = std::max<int64_t>(16, std::min<int64_t>(1024, (int64_t(1) << 18) / nranks));
  j.out_pat = out_pat;
  j.out_sum = out_sum;
  j.out_abs = out_abs;
  if (threads <= 0) threads = available_threads();
  const int64_t per_chunk = count > 0 ? (count + j.block - 1) / j.block : 0;
  const int64_t items = per_chunk * (r1 - r0);
  threads = int(std::max<int64_t>(1, std::min<int64_t>(threads, items)));
  std::atomic<int64_t> next{0};
  auto worker = [&]() {
    Scratch w;
    w.v.resize(size_t(nranks) * size_t(j.block));
    w.s.resize(size_t(j.block));
    w.a.resize(size_t(j.block));
    for (;;) {
      const int64_t k = next.fetch_add(1);
      if (k >= items) break;
      const int R = r0 + int(k / per_chunk);
      const int64_t i0 = (k % per_chunk) * j.block;
      run_item(j, R, i0, std::min<int64_t>(count, i0 + j.block), w);
    }
  };
  std::vector<std::thread> pool;
  for (int t = 1; t < threads; ++t) pool.emplace_back(worker);
  worker();
  for (auto& t : pool) t.join();
  return threads;
}

}  // extern "C"
