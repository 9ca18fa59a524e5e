// Host-only consistency driver for the plan code, built with sanitizers by
// tests/test_host_sanitizers.py.  For many (ranks, count, budget, order) it
// builds plans and checks their tables: every tree edge once per piece, slot
// indices inside the slot map, each non-root receiver starting from its own
// input exactly once.
#include <cstdio>
#include <cstdlib>
#include <vector>

#include "plan.hpp"

int main() {
  long plans = 0;
  const size_t budgets[] = {16, 4096, 65536, size_t(8) << 20};
  for (int N = 1; N <= 300; ++N) {
    for (int order = 0; order < 2; ++order) {
      for (size_t budget : budgets) {
        for (int coll = 0; coll < 2; ++coll) {
          for (int64_t count : {int64_t(1), int64_t(17), int64_t(1000)}) {
            pat::PlanDesc d;
            if (!pat::make_plan_desc(coll, N, count, coll ? 2 : 1, budget, order, &d)) {
              std::fprintf(stderr, "plan failed N=%d budget=%zu order=%d\n", N, budget, order);
              return 1;
            }
            ++plans;
            if (N == 1) continue;
            if ((int)d.entries.size() != N - 1) {
              std::fprintf(stderr, "N=%d: %zu entries\n", N, d.entries.size());
              return 1;
            }
            std::vector<int> own_starts(N, 0);
            for (const auto& e : d.entries) {
              const int vals[3] = {e.a, e.b, e.c};
              for (int v : vals)
                if (v >= d.slots.entries) {
                  std::fprintf(stderr, "N=%d: slot %d out of %d\n", N, v, d.slots.entries);
                  return 1;
                }
              if (coll == 1 && e.b == pat::kUser) own_starts[e.p]++;
            }
            if (coll == 1)
              for (int p = 0; p < N; ++p) {
                const bool receives = p == 0 || ((p & -p) >= 2 && p + 1 < N);
                if (own_starts[p] != (receives ? 1 : 0)) {
                  std::fprintf(stderr, "N=%d p=%d: own input enters %d times\n", N, p, own_starts[p]);
                  return 1;
                }
              }
          }
        }
      }
    }
  }
  std::printf("plans checked: %ld\n", plans);
  return 0;
}
