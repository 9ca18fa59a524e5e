// Drives the threaded C++ oracle (oracle/rs_oracle.cpp, oracle/ag_oracle.cpp)
// under AddressSanitizer / UndefinedBehaviorSanitizer, or ThreadSanitizer:
// every generator kind and dtype, ranks from 1 to 100, empty and ragged
// counts, destination / receiver ranges and thread counts.  Results must not
// depend on the thread count, and the all-gather's array path must give what
// its generator path gives.
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

extern "C" int oracle_reducescatter(const void* inputs, int kind, uint64_t seed, int64_t lo, uint64_t span,
                                    const void* table, int nranks, int64_t count, int dtype, int r0, int r1,
                                    void* out_pat, double* out_sum, double* out_abs, int threads);
extern "C" int oracle_allgather(const void* inputs, int kind, uint64_t seed, int64_t lo, uint64_t span,
                                const void* table, int nranks, int64_t count, int dtype, int r0, int r1, void* out,
                                int threads);

static int failures = 0;
#define EXPECT(cond)                                                        \
  do {                                                                      \
    if (!(cond)) {                                                          \
      std::fprintf(stderr, "%s:%d: expected %s\n", __FILE__, __LINE__, #cond); \
      ++failures;                                                           \
    }                                                                       \
  } while (0)

int main() {
  // any 65536-entry tables will do for kinds 2 (16-bit) and 3 (32-bit)
  std::vector<uint16_t> t16(65536);
  std::vector<uint32_t> t32(65536);
  for (int i = 0; i < 65536; ++i) {
    t16[i] = uint16_t(0x3F80 + (i % 64) - 32);
    t32[i] = 0x3F800000u + uint32_t(i % 4096) - 2048u;
  }
  const int ns[] = {1, 2, 3, 7, 33, 100};
  const int64_t counts[] = {0, 1, 5, 257};
  long cases = 0;
  for (int n : ns)
    for (int64_t count : counts)
      for (int dtype = 0; dtype < 3; ++dtype)
        for (int kind = 0; kind < 4; ++kind) {
          if (dtype == 2 && kind != 2) continue;  // bf16 comes from the 16-bit table
          if (dtype != 2 && kind == 2) continue;
          const void* table = kind == 2 ? (const void*)t16.data() : kind == 3 ? (const void*)t32.data() : nullptr;
          const int64_t lo = -(int64_t(1) << 20);
          const uint64_t span = (uint64_t(1) << 21) + 1;
          const int r0 = n > 2 ? 1 : 0, r1 = n;
          const size_t rows = size_t(r1 - r0);
          const size_t es = dtype == 2 ? 2 : 4;
          // reduce-scatter
          std::vector<unsigned char> p1(rows * count * es + 1), p4(rows * count * es + 1);
          std::vector<double> s1(rows * count + 1), s4(rows * count + 1), a1(rows * count + 1), a4(rows * count + 1);
          const int u1 = oracle_reducescatter(nullptr, kind, 7, lo, span, table, n, count, dtype, r0, r1, p1.data(),
                                              s1.data(), a1.data(), 1);
          const int u4 = oracle_reducescatter(nullptr, kind, 7, lo, span, table, n, count, dtype, r0, r1, p4.data(),
                                              s4.data(), a4.data(), 4);
          EXPECT(u1 == 1 && u4 >= 1);
          EXPECT(std::memcmp(p1.data(), p4.data(), p1.size()) == 0);
          EXPECT(std::memcmp(s1.data(), s4.data(), s1.size() * sizeof(double)) == 0);
          EXPECT(std::memcmp(a1.data(), a4.data(), a1.size() * sizeof(double)) == 0);
          // all-gather: the generator path, then the array path fed with row 0
          const size_t row = size_t(n) * count * es;
          std::vector<unsigned char> g1(rows * row + 1), g4(rows * row + 1), first(row + 1), arr(rows * row + 1);
          EXPECT(oracle_allgather(nullptr, kind, 9, lo, span, table, n, count, dtype, r0, r1, g1.data(), 1) == 1);
          EXPECT(oracle_allgather(nullptr, kind, 9, lo, span, table, n, count, dtype, r0, r1, g4.data(), 4) >= 1);
          EXPECT(std::memcmp(g1.data(), g4.data(), g1.size()) == 0);
          EXPECT(oracle_allgather(nullptr, kind, 9, lo, span, table, n, count, dtype, 0, 1, first.data(), 3) >= 1);
          EXPECT(oracle_allgather(first.data(), 0, 0, 0, 0, nullptr, n, count, dtype, r0, r1, arr.data(), 4) >= 1);
          EXPECT(std::memcmp(arr.data(), g1.data(), rows * row) == 0);
          for (size_t r = 1; r < rows; ++r) EXPECT(std::memcmp(g1.data() + r * row, g1.data(), row) == 0);
          ++cases;
        }
  // invalid arguments are refused
  unsigned char buf[64];
  EXPECT(oracle_allgather(nullptr, 1, 0, 0, 0, nullptr, 0, 4, 1, 0, 0, buf, 1) == -1);
  EXPECT(oracle_allgather(nullptr, 2, 0, 0, 0, nullptr, 4, 4, 2, 0, 4, buf, 1) == -1);
  EXPECT(oracle_allgather(nullptr, 1, 0, 0, 0, nullptr, 4, 4, 1, 2, 5, buf, 1) == -1);
  EXPECT(oracle_allgather(nullptr, 1, 0, 0, 0, nullptr, 4, 4, 1, 0, 4, nullptr, 1) == -1);
  EXPECT(oracle_reducescatter(nullptr, 1, 0, 0, 0, nullptr, 4, 4, 3, 0, 4, buf, nullptr, nullptr, 1) == -1);
  std::printf("%ld oracle cases checked, %d failures\n", cases, failures);
  return failures ? 1 : 0;
}
