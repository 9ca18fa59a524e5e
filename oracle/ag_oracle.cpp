// Threaded CPU oracle of the all-gather.
//
// TEST INFRASTRUCTURE ONLY.  Only tests/, __graft_entry__.smoke() and the
// cpu_baseline leg of bench.py load this library.  It shares no code, header,
// table or helper with the HIP library; the only header it includes from this
// repository is the seeded input generator (synth/synth_host.hpp), which holds
// none of the method's arithmetic.
//
// What it computes (section "All-gather and reduce-scatter algorithms", the
// operation's definition; PAT reaches exactly this result, whatever its
// schedule): for every receiving rank r and every rank x,
//
//     out[r][x * count + i] = in[x][i],   i = 0 .. count - 1,
//
// the concatenation of all ranks' send buffers in rank order, the same for
// every receiver.  Bytes are copied as they are; nothing is converted.
//
// Inputs come either from an array ([N][count] elements) or from the seeded
// generator, each rank's chunk generated once per call; std::thread workers
// generate the chunks, one rank at a time, then fill the receivers' rows, a
// run of chunks of one row (about 64 KiB) per work item.
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

int cpus() {
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

// All-gather result rows of receivers [r0, r1) of an N-rank operation with
// `count` elements per rank.
//   inputs:  [N][count] raw elements (int32, float32, or bfloat16 bits), or
//            null to generate them with the seeded generator (kind, seed, lo,
//            span, table as in synth/synth_host.hpp);
//   dtype:   0 int32, 1 float32, 2 bfloat16 (4, 4 and 2 bytes per element);
//   out:     [r1 - r0][N * count] elements of the input dtype;
//   threads: workers to use, <= 0 for every available CPU.
// Returns the number of threads used, or -1 for invalid arguments.
int oracle_allgather(const void* inputs, int kind, uint64_t seed, int64_t lo, uint64_t span, const void* table,
                     int nranks, int64_t count, int dtype, int r0, int r1, void* out, int threads) {
  if (nranks < 1 || count < 0 || dtype < kInt32 || dtype > kBfloat16 || !out) return -1;
  if (r0 < 0 || r1 > nranks || r0 > r1) return -1;
  if (!inputs && (kind < 0 || kind > 3 || (kind >= 2 && !table))) return -1;
  if (threads <= 0) threads = cpus();
  if (count == 0 || r0 == r1) return 1;  // nothing to copy
  const size_t esize = dtype == kBfloat16 ? 2 : 4;
  const size_t chunk = size_t(count) * esize;
  // A work item: a run of `per` consecutive chunks of one receiver's row,
  // about 64 KiB.
  const int64_t per = std::max<int64_t>(1, std::min<int64_t>(nranks, int64_t(65536) / int64_t(std::max<size_t>(chunk, 1))));
  const int64_t runs = (nranks + per - 1) / per;
  const int64_t items = int64_t(r1 - r0) * runs;
  threads = int(std::max<int64_t>(1, std::min<int64_t>(threads, std::max<int64_t>(items, nranks))));
  auto run = [threads](auto&& work) {
    std::vector<std::thread> pool;
    for (int t = 1; t < threads; ++t) pool.emplace_back(work);
    work();
    for (auto& t : pool) t.join();
  };
  // Each rank's send buffer, as bytes; generated ranks are shared among the
  // workers.
  std::vector<unsigned char> generated;
  const unsigned char* src = static_cast<const unsigned char*>(inputs);
  if (!src) {
    generated.resize(size_t(nranks) * chunk);
    synth_host::Source gen;
    gen.kind = kind;
    gen.seed = seed;
    gen.lo = lo;
    gen.span = span;
    gen.table = table;
    std::atomic<int> next_rank{0};
    run([&]() {
      std::vector<uint32_t> words(static_cast<size_t>(count));
      for (int x; (x = next_rank.fetch_add(1)) < nranks;) {
        gen.row(x, 0, count, words.data());
        unsigned char* dst = generated.data() + size_t(x) * chunk;
        if (dtype == kBfloat16) {
          for (int64_t i = 0; i < count; ++i) {
            const uint16_t h = uint16_t(words[size_t(i)]);
            std::memcpy(dst + size_t(i) * 2, &h, 2);
          }
        } else {
          std::memcpy(dst, words.data(), chunk);
        }
      }
    });
    src = generated.data();
  }
  unsigned char* o = static_cast<unsigned char*>(out);
  std::atomic<int64_t> next{0};
  run([&]() {
    for (int64_t k; (k = next.fetch_add(1)) < items;) {
      const int64_t row = k / runs, x0 = (k % runs) * per;  // receiver r0 + row, chunks [x0, x1)
      const int64_t x1 = std::min<int64_t>(nranks, x0 + per);
      for (int64_t x = x0; x < x1; ++x)
        std::memcpy(o + (size_t(row) * nranks + size_t(x)) * chunk, src + size_t(x) * chunk, chunk);
    }
  });
  return threads;
}

}  // extern "C"
