// Host-only consistency driver for the plan code, built with sanitizers by
// tests/test_host_sanitizers.py.  For many (ranks, count, budget, order) it
// builds plans and checks their tables: every tree edge once per piece, slot
// indices inside the slot map, each non-root receiver starting from its own
// input exactly once.  For N <= 64 it also runs the dataflow dependency table
// (dataflow_deps) symbolically: edges execute in orders that respect nothing
// but their counters (shuffled, and latest step first), and every transfer
// must find what the schedule promises -- the chunk a sender forwards, the
// partial sums a receiver adds -- with no edge left unable to run.  Plans with
// PAT_AGGREGATION_BUDGET (list schedules where they are shorter) get the same
// checks, plus: never more steps than the power-of-two plan, at most K =
// budget / chunk bytes chunks per step and per slot.
#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

#include "plan.hpp"

namespace {

struct Edge {
  int step, r, j;
};

// Returns an error message, or nullptr.
const char* simulate_dataflow(const pat::PlanDesc& d, uint32_t seed, bool latest_first) {
  const int N = d.N, E = d.slots.entries, root = E;
  std::vector<pat::DevDep> deps;
  if (!pat::dataflow_deps(d, &deps)) return "dataflow_deps refused the plan";
  std::vector<uint32_t> ctr(size_t(N) * (E + 1), 0);
  // Buffer contents: all-gather slots hold a chunk id (+1, 0 empty); reduce-
  // scatter accumulators hold (chunk id, mask of contributing ranks).
  std::vector<int> ag_slot(size_t(N) * E, 0);
  std::vector<uint64_t> ag_have(N, 0);
  std::vector<int> rs_chunk(size_t(N) * (E + 1), -1);
  std::vector<uint64_t> rs_mask(size_t(N) * (E + 1), 0);
  for (int r = 0; r < N; ++r) ag_have[r] = uint64_t(1) << r;
  std::vector<Edge> pending;
  for (int s = 0; s < (int)d.exec.size(); ++s)
    for (int r = 0; r < N; ++r)
      for (int i = 0; i < d.exec[s].k; ++i) pending.push_back({s, r, d.exec[s].first + i});
  std::mt19937 rng(seed);
  auto at = [&](int x, int e) { return size_t(x) * (E + 1) + e; };
  while (!pending.empty()) {
    std::shuffle(pending.begin(), pending.end(), rng);
    if (latest_first)
      std::stable_sort(pending.begin(), pending.end(), [](const Edge& a, const Edge& b) { return a.step > b.step; });
    std::vector<Edge> left;
    bool progress = false;
    for (const Edge& ed : pending) {
      const pat::StepSpec& st = d.exec[ed.step];
      const pat::DevEntry& en = d.entries[ed.j];
      const pat::DevDep& g = deps[ed.j];
      const int r = ed.r, peer = (r + st.d) % N;
      const int x1 = d.coll == 0 ? r : peer, x2 = d.coll == 0 ? peer : r;
      if ((g.e1 >= 0 && ctr[at(x1, g.e1)] < (uint32_t)g.need1) || (g.e2 >= 0 && ctr[at(x2, g.e2)] < (uint32_t)g.need2)) {
        left.push_back(ed);
        continue;
      }
      const int c = ((r - en.p) % N + N) % N;  // the tree (chunk) of this edge
      if (d.coll == 0) {
        if (en.p != 0 && ag_slot[size_t(r) * E + en.a] != c + 1) return "all-gather: sender's slot does not hold the chunk";
        if (ag_have[peer] >> c & 1) return "all-gather: chunk received twice";
        ag_have[peer] |= uint64_t(1) << c;
        if (en.b >= 0) ag_slot[size_t(peer) * E + en.b] = c + 1;
      } else {
        uint64_t child;
        if (en.a < 0) {
          child = uint64_t(1) << peer;
        } else {
          if (rs_chunk[at(peer, en.a)] != c) return "reduce-scatter: child's accumulator holds another chunk";
          child = rs_mask[at(peer, en.a)];
        }
        uint64_t own;
        const int ob = en.b >= 0 ? en.b : en.b == pat::kRoot ? root : -1;
        if (ob < 0) {
          own = uint64_t(1) << r;
        } else {
          if (rs_chunk[at(r, ob)] != c) return "reduce-scatter: own accumulator holds another chunk";
          own = rs_mask[at(r, ob)];
        }
        if (own & child) return "reduce-scatter: a contribution added twice";
        const int oc = en.c >= 0 ? en.c : root;
        rs_chunk[at(r, oc)] = c;
        rs_mask[at(r, oc)] = own | child;
      }
      if (g.e1 >= 0) ++ctr[at(x1, g.e1)];
      if (g.e2 >= 0) ++ctr[at(x2, g.e2)];
      progress = true;
    }
    if (!progress) return "dataflow deadlock: no pending edge can run";
    pending.swap(left);
  }
  const uint64_t all = N == 64 ? ~uint64_t(0) : (uint64_t(1) << N) - 1;
  for (int r = 0; r < N; ++r) {
    if (d.coll == 0 && ag_have[r] != all) return "all-gather: a rank misses a chunk";
    if (d.coll == 1 && (rs_chunk[at(r, root)] != r || rs_mask[at(r, root)] != all)) return "reduce-scatter: wrong sum";
  }
  return nullptr;
}

}  // namespace

int main() {
  long plans = 0, dataflow_runs = 0, list_plans = 0;
  // 204, 340 and 476 bytes are 3, 5 and 7 chunks of 17 four-byte elements: with
  // PAT_AGGREGATION_BUDGET they bring in the list schedule
  const size_t budgets[] = {16, 204, 340, 476, 4096, 65536, size_t(8) << 20};
  for (int N = 1; N <= 300; ++N) {
    for (int order = 0; order < 2; ++order) {
      for (size_t budget : budgets) {
        for (int coll = 0; coll < 2; ++coll) {
          for (int64_t count : {int64_t(1), int64_t(17), int64_t(1000)}) {
           for (int agg = 0; agg < 2; ++agg) {
            if (agg == 1 && (order == 1 || count != 17)) continue;
            pat::PlanDesc d;
            if (!pat::make_plan_desc(coll, N, count, coll ? 2 : 1, budget, order, &d, agg)) {
              std::fprintf(stderr, "plan failed N=%d budget=%zu order=%d agg=%d\n", N, budget, order, agg);
              return 1;
            }
            ++plans;
            if (agg == 1) {
              pat::PlanDesc p2;
              pat::make_plan_desc(coll, N, count, coll ? 2 : 1, budget, order, &p2, 0);
              const int64_t K = int64_t(budget / (size_t(count) * 4));
              if (d.exec.size() > p2.exec.size() || (d.sched.list && d.max_k > K)) {
                std::fprintf(stderr, "N=%d budget=%zu: list schedule %zu steps (max %d chunks) vs %zu\n", N, budget,
                             d.exec.size(), d.max_k, p2.exec.size());
                return 1;
              }
              if (d.sched.list) {
                ++list_plans;
                for (int c = 0; c < (int)d.slots.cap.size(); ++c)
                  if (d.slots.cap[c] > K) {
                    std::fprintf(stderr, "N=%d budget=%zu: %d chunks in one slot\n", N, budget, d.slots.cap[c]);
                    return 1;
                  }
              }
            }
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
            if (N <= 64 && count == 17) {
              for (int mode = 0; mode < 2; ++mode) {
                if (const char* err = simulate_dataflow(d, uint32_t(N * 7919 + order * 31 + coll), mode == 1)) {
                  std::fprintf(stderr, "N=%d coll=%d budget=%zu order=%d agg=%d: %s\n", N, coll, budget, order, agg,
                               err);
                  return 1;
                }
                ++dataflow_runs;
              }
            }
           }
          }
        }
      }
    }
  }
  std::printf("plans checked: %ld (list schedules: %ld), dataflow simulations: %ld\n", plans, list_plans,
              dataflow_runs);
  return 0;
}
