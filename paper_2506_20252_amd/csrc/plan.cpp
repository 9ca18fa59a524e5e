// Host-side PAT plan: schedule, slot layout, byte model.  See plan.hpp.
#include "plan.hpp"

#include <algorithm>
#include <set>
#include <tuple>
#include <utility>

namespace pat {

int ceil_log2(int64_t n) {
  int L = 0;
  while ((int64_t(1) << L) < n) ++L;
  return L;
}

// Far-first pre-order walk of a full sub-tree of span `span`: from a node, the
// farthest child first, and that child's whole sub-tree before the next, closer
// child.  An explicit stack holds "edge (q, d) still to emit".
static void far_first_walk(int span, std::vector<std::pair<int, int>>* out) {
  std::vector<std::pair<int, int>> stack;
  if (span >= 2) stack.emplace_back(0, span / 2);
  while (!stack.empty()) {
    const auto [q, d] = stack.back();
    stack.pop_back();
    out->emplace_back(q, d);
    if (d >= 2) {
      stack.emplace_back(q, d / 2);      // then the next closer child of q
      stack.emplace_back(q + d, d / 2);  // first: the sub-tree just reached
    }
  }
}

// Close-first pre-order walk: from a node, the nearest child first, each
// child's whole sub-tree right after the edge that reached it.
static void close_first_walk(int q, int span, std::vector<std::pair<int, int>>* out) {
  for (int d = 1; d < span; d <<= 1) {
    out->emplace_back(q, d);
    close_first_walk(q + d, d, out);
  }
}

Schedule make_schedule(int N, int t, int order) {
  Schedule s;
  s.N = N;
  if (N <= 1) return s;
  s.L = ceil_log2(N);
  s.t = std::max(0, std::min(t, s.L - 1));
  s.T = 1 << s.t;
  s.M = 1 << (s.L - s.t);
  // Top: one fully aggregated step per distance, farthest first.  Before the
  // step of distance d the positions holding data are the multiples of 2d.
  for (int d = 1 << (s.L - 1); d >= s.M; d >>= 1) {
    StepSpec st{d, 0, (int32_t)s.pos.size()};
    for (int p = 0; p + d < N; p += 2 * d) s.pos.push_back(p);
    st.k = (int32_t)s.pos.size() - st.first;
    s.steps.push_back(st);
  }
  // Linear part: the walk of one span-M sub-tree, taken by all T at once.
  std::vector<std::pair<int, int>> walk;
  if (order == kCloseFirst)
    close_first_walk(0, s.M, &walk);
  else
    far_first_walk(s.M, &walk);
  for (const auto& [q, d] : walk) {
    StepSpec st{d, 0, (int32_t)s.pos.size()};
    for (int b = 0; b < s.T; ++b) {
      const int p = b * s.M + q;
      if (p + d < N) s.pos.push_back(p);
    }
    st.k = (int32_t)s.pos.size() - st.first;
    if (st.k > 0) s.steps.push_back(st);
  }
  return s;
}

int max_chunks_per_step(const Schedule& s) {
  int m = 0;
  for (const auto& st : s.steps) m = std::max(m, (int)st.k);
  return m;
}

static bool needs_slot(int N, int p) {
  if (p <= 0 || p >= N) return false;
  const int D = p & -p;
  return D >= 2 && p + 1 < N;  // has at least one child: p + 1
}

int32_t SlotMap::index(int p) const {
  if (!table.empty()) return p >= 0 && p < (int)table.size() ? table[p] : -1;
  if (!needs_slot(N, p)) return -1;
  const int D = p & -p;
  return base[ceil_log2(D)] + p / std::max(2 * D, M);
}

SlotMap make_slot_map(int N, int L, int M) {
  SlotMap m;
  m.N = N;
  m.L = L;
  m.M = M;
  m.base.assign(std::max(L, 1), 0);
  m.cap.assign(std::max(L, 1), 0);
  for (int p = 1; p < N; ++p) {
    if (!needs_slot(N, p)) continue;
    const int D = p & -p;
    const int l = ceil_log2(D);
    m.cap[l] = std::max(m.cap[l], p / std::max(2 * D, M) + 1);
  }
  int32_t acc = 0;
  for (size_t l = 0; l < m.cap.size(); ++l) {
    m.base[l] = acc;
    acc += m.cap[l];
    if (m.cap[l] > 0) ++m.dims;
  }
  m.entries = acc;
  return m;
}

Schedule make_list_schedule(int N, int K, SlotMap* slots) {
  Schedule s;
  s.N = N;
  s.list = true;
  s.T = std::max(1, K);
  s.M = 0;
  slots->table.clear();
  if (N <= 1) return s;
  const int L = ceil_log2(N);
  s.L = L;
  K = std::max(1, K);
  // Children of every position, farthest first; sub-tree sizes (children sit
  // at larger positions).
  std::vector<std::vector<std::pair<int, int>>> kids(N);
  for (int p = 0; p < N; ++p) {
    const int reach = p == 0 ? (1 << L) : (p & -p);
    for (int d = reach / 2; d >= 1; d /= 2)
      if (p + d < N) kids[p].emplace_back(p + d, d);
  }
  std::vector<int64_t> sz(N, 1);
  for (int p = N - 1; p >= 0; --p)
    for (const auto& [c, d] : kids[p]) sz[p] += sz[c];
  // Ready edges by the log2 of their distance, in priority order (larger
  // sub-tree first, then smaller position); apart, those into nodes that
  // forward and those into leaves.
  using Key = std::pair<int64_t, int>;  // (-size of the child's sub-tree, sender)
  std::vector<std::set<Key>> fwd(L), leaf(L);
  auto add_ready = [&](int p, const std::vector<int>& nxt) {
    if (nxt[p] >= (int)kids[p].size()) return;
    const auto [c, d] = kids[p][nxt[p]];
    const int l = ceil_log2(d);
    (kids[c].empty() ? leaf : fwd)[l].insert(Key(-sz[c], p));
  };
  std::vector<int> nxt(N, 0), color(N, -1), dim_of(N, -1);
  std::vector<std::vector<char>> used(L);
  std::vector<int> cap(L, 0), occ(L, 0);
  add_ready(0, nxt);
  int sent = 0;
  while (sent < N - 1) {
    int best_l = -1;
    std::pair<int64_t, int> best_key(-1, -1);
    std::vector<int> best_take;
    for (int l = L - 1; l >= 0; --l) {
      // merge the two priority orders; into forwarding nodes only while the slot has room
      std::vector<int> take;
      int64_t weight = 0;
      int room = K - occ[l];
      auto f = fwd[l].begin(), g = leaf[l].begin();
      while ((int)take.size() < K) {
        const bool fok = f != fwd[l].end() && room > 0;
        const bool gok = g != leaf[l].end();
        if (!fok && !gok) break;
        if (fok && (!gok || *f < *g)) {
          take.push_back(f->second);
          weight += -f->first;
          --room;
          ++f;
        } else {
          take.push_back(g->second);
          weight += -g->first;
          ++g;
        }
      }
      if (take.empty()) continue;
      const std::pair<int64_t, int> key(weight, (int)take.size());
      if (key > best_key) {
        best_key = key;
        best_l = l;
        best_take = take;
      }
    }
    if (best_l < 0) {
      s.steps.clear();
      s.pos.clear();
      return s;
    }
    std::sort(best_take.begin(), best_take.end());
    StepSpec st{1 << best_l, (int32_t)best_take.size(), (int32_t)s.pos.size()};
    std::vector<int> done_senders;
    for (int p : best_take) {
      const auto [c, d] = kids[p][nxt[p]];
      (kids[c].empty() ? leaf : fwd)[best_l].erase(Key(-sz[c], p));
      s.pos.push_back(p);
      ++nxt[p];
      ++sent;
      if (!kids[c].empty()) {  // c keeps the chunk in the slot of distance d until its last forward
        auto& u = used[best_l];
        int col = 0;
        while (col < (int)u.size() && u[col]) ++col;
        if (col == (int)u.size()) u.push_back(0);
        u[col] = 1;
        color[c] = col;
        dim_of[c] = best_l;
        cap[best_l] = std::max(cap[best_l], col + 1);
        ++occ[best_l];
        add_ready(c, nxt);
      }
      add_ready(p, nxt);
      if (nxt[p] == (int)kids[p].size()) done_senders.push_back(p);
    }
    // a sender that has forwarded to all of its children frees its entry after the step
    for (int p : done_senders)
      if (dim_of[p] >= 0) {
        used[dim_of[p]][color[p]] = 0;
        --occ[dim_of[p]];
      }
    s.steps.push_back(st);
  }
  slots->N = N;
  slots->L = L;
  slots->M = 0;
  slots->base.assign(L, 0);
  slots->cap.assign(L, 0);
  slots->dims = 0;
  int32_t acc = 0;
  for (int l = 0; l < L; ++l) {
    slots->base[l] = acc;
    slots->cap[l] = cap[l];
    acc += cap[l];
    if (cap[l] > 0) ++slots->dims;
  }
  slots->entries = acc;
  slots->table.assign(N, -1);
  for (int p = 0; p < N; ++p)
    if (dim_of[p] >= 0) slots->table[p] = slots->base[dim_of[p]] + color[p];
  return s;
}

static int elem_bytes(int dtype) { return dtype == 2 ? 2 : 4; }

bool make_plan_desc(int coll, int N, int64_t count, int dtype, size_t budget, int order, PlanDesc* out,
                    int aggregation, bool pipeline) {
  if (coll < 0 || coll > 1 || N < 1 || count < 0 || dtype < 0 || dtype > 2) return false;
  if (order != kFarFirst && order != kCloseFirst) return false;
  if (aggregation != kAggPow2 && aggregation != kAggBudget) return false;
  PlanDesc d;
  d.coll = coll;
  d.order = order;
  d.N = N;
  d.dtype = dtype;
  d.count = count;
  d.esize_in = elem_bytes(dtype);
  d.esize_slot = (coll == 1 && dtype == 2) ? 4 : d.esize_in;
  const double c_slot = double(count) * d.esize_slot;

  int t = 0;
  if (N > 1) {
    const int L = ceil_log2(N);
    for (t = L - 1; t > 0; --t) {
      const Schedule s = make_schedule(N, t, order);
      if (double(max_chunks_per_step(s)) * c_slot <= double(budget)) break;
    }
  }
  d.sched = make_schedule(N, t, order);
  d.max_k = max_chunks_per_step(d.sched);

  // A chunk larger than the budget is processed in pieces (T = 1 then); with
  // the pipeline, pieces of half the budget, two of them in flight.
  d.pieces = 1;
  d.piece_elems = count;
  if (pipeline && c_slot > double(budget) && budget >= 2 * size_t(d.esize_slot)) {
    d.pipelined = true;
    budget /= 2;
  }
  if (c_slot > double(budget)) {
    int64_t pe = int64_t(budget / size_t(d.esize_slot));
    if (pe <= 0) return false;
    if (pe >= 8) pe -= pe % 8;  // keep 128-bit vectors whole
    d.piece_elems = pe;
    d.pieces = int((count + pe - 1) / pe);
  }

  const int M = d.sched.M;
  d.slots = make_slot_map(N, d.sched.L, M);
  // With the budget's chunks per step not a power of two, a list schedule may
  // need fewer steps; it replaces the power-of-two one only then.
  if (aggregation == kAggBudget && N > 2 && d.pieces == 1) {
    const int64_t K = c_slot > 0 ? int64_t(double(budget) / c_slot) : 1;
    if (K >= 2 && K < int64_t(N) && (int)d.sched.steps.size() > d.sched.L) {
      SlotMap ls;
      Schedule alt = make_list_schedule(N, (int)std::min<int64_t>(K, N), &ls);
      if (!alt.steps.empty() && alt.steps.size() < d.sched.steps.size()) {
        d.sched = std::move(alt);
        d.slots = std::move(ls);
        d.max_k = max_chunks_per_step(d.sched);
      }
    }
  }
  const auto& S = d.sched;
  if (coll == 0) {
    for (const auto& st : S.steps) {
      d.exec.push_back({st.d, st.k, (int32_t)d.entries.size()});
      for (int j = 0; j < st.k; ++j) {
        const int p = S.pos[st.first + j];
        DevEntry e{};
        e.p = p;
        e.a = p == 0 ? kUser : d.slots.index(p);
        const int32_t to = d.slots.index(p + st.d);
        e.b = to >= 0 ? to : kUser;
        e.c = kUser;  // unused by the all-gather
        if (p != 0 && e.a < 0) return false;  // a forwarding node always has a slot
        d.entries.push_back(e);
      }
    }
  } else {
    // A receiver's first receive starts from its own input, and the root's
    // last receive writes the receive buffer; which receives those are
    // follows from the execution order (far-first: distance 1 first and the
    // farthest distance last; close-first reverses the linear part).
    std::vector<int32_t> first(N, -1), last(N, -1);
    int32_t idx = 0;
    for (auto it = S.steps.rbegin(); it != S.steps.rend(); ++it)
      for (int j = 0; j < it->k; ++j, ++idx) {
        const int p = S.pos[it->first + j];
        if (first[p] < 0) first[p] = idx;
        last[p] = idx;
      }
    idx = 0;
    for (auto it = S.steps.rbegin(); it != S.steps.rend(); ++it) {
      const auto& st = *it;
      d.exec.push_back({st.d, st.k, (int32_t)d.entries.size()});
      for (int j = 0; j < st.k; ++j, ++idx) {
        const int p = S.pos[st.first + j];
        DevEntry e{};
        e.p = p;
        const int32_t child = d.slots.index(p + st.d);
        e.a = child >= 0 ? child : kUser;  // a leaf child sends its raw input
        if (first[p] == idx) {
          e.b = kUser;
        } else if (p == 0) {
          e.b = kRoot;
        } else {
          e.b = d.slots.index(p);
          if (e.b < 0) return false;
        }
        if (p == 0) {
          e.c = last[p] == idx ? kRootFinal : kRoot;
        } else {
          e.c = d.slots.index(p);
          if (e.c < 0) return false;
        }
        d.entries.push_back(e);
      }
    }
  }
  d.alg_bytes = algorithmic_bytes(d);
  *out = std::move(d);
  return true;
}

bool dataflow_deps(const PlanDesc& d, std::vector<DevDep>* deps) {
  const int root = d.slots.entries;  // counter index of the own chunk's accumulator
  std::vector<int32_t> done(size_t(root) + 1, 0);  // accesses completed before the current step
  deps->assign(d.entries.size(), DevDep{-1, 0, -1, 0});
  for (const auto& st : d.exec) {
    std::vector<int32_t> now(done);
    for (int j = 0; j < st.k; ++j) {
      const DevEntry& e = d.entries[st.first + j];
      DevDep& g = (*deps)[st.first + j];
      if (d.coll == 0) {
        g.e1 = e.a >= 0 ? e.a : -1;  // the sender's slot (-1: its own send buffer)
        g.e2 = e.b >= 0 ? e.b : -1;  // the receiver's slot (-1: receive buffer only)
      } else {
        g.e1 = e.a >= 0 ? e.a : -1;     // the child's accumulator (-1: a leaf's raw input)
        g.e2 = e.c >= 0 ? e.c : root;   // the receiver's accumulator or its own chunk's
      }
      for (int32_t* ep : {&g.e1, &g.e2}) {
        if (*ep < 0) continue;
        if (now[*ep] != done[*ep]) return false;  // a second access in one step
        ++now[*ep];
      }
      if (g.e1 >= 0) g.need1 = done[g.e1];
      if (g.e2 >= 0) g.need2 = done[g.e2];
    }
    done.swap(now);
  }
  return true;
}

double step_bytes(const PlanDesc& d, int s, int64_t elems) {
  if (d.N <= 1 || elems <= 0 || s < 0 || s >= (int)d.exec.size()) return 0.0;
  const double ei = d.esize_in, es = d.esize_slot;
  double per_elem = 0.0;  // bytes per element of a chunk, over one rank's entries of this step
  const StepSpec& st = d.exec[s];
  for (int j = 0; j < st.k; ++j) {
    const DevEntry& e = d.entries[st.first + j];
    if (d.coll == 0) {
      per_elem += ei + ei + (e.b >= 0 ? ei : 0.0);
    } else {
      per_elem += (e.a == kUser) ? ei : es;
      per_elem += (e.b == kUser) ? ei : es;
      per_elem += (e.c == kRootFinal) ? ei : es;
    }
  }
  if (d.coll == 0 && s == 0) per_elem += ei;  // the own chunk's copy into the receive buffer
  return double(d.N) * per_elem * double(elems);
}

double algorithmic_bytes(const PlanDesc& d) {
  if (d.count == 0) return 0.0;
  if (d.N == 1) return 2.0 * double(d.count) * d.esize_in;  // a copy
  // Every piece runs every step, and step_bytes is linear in the piece's
  // length, whose sum over the pieces is `count`.
  double total = 0.0;
  for (int s = 0; s < (int)d.exec.size(); ++s) total += step_bytes(d, s, d.count);
  return total;
}

}  // namespace pat
