// Host-side PAT plan: schedule, slot layout, byte model.  See plan.hpp.
#include "plan.hpp"

#include <algorithm>
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

static int elem_bytes(int dtype) { return dtype == 2 ? 2 : 4; }

bool make_plan_desc(int coll, int N, int64_t count, int dtype, size_t budget, int order, PlanDesc* out) {
  if (coll < 0 || coll > 1 || N < 1 || count < 0 || dtype < 0 || dtype > 2) return false;
  if (order != kFarFirst && order != kCloseFirst) return false;
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

  // A chunk larger than the budget is processed in pieces (T = 1 then).
  d.pieces = 1;
  d.piece_elems = count;
  if (c_slot > double(budget)) {
    int64_t pe = int64_t(budget / size_t(d.esize_slot));
    if (pe <= 0) return false;
    if (pe >= 8) pe -= pe % 8;  // keep 128-bit vectors whole
    d.piece_elems = pe;
    d.pieces = int((count + pe - 1) / pe);
  }

  const int M = d.sched.M;
  d.slots = make_slot_map(N, d.sched.L, M);
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
  double total = 0.0;
  for (int piece = 0; piece < d.pieces; ++piece) {
    const int64_t e0 = int64_t(piece) * d.piece_elems;
    const int64_t len = std::min<int64_t>(d.piece_elems, d.count - e0);
    for (int s = 0; s < (int)d.exec.size(); ++s) total += step_bytes(d, s, len);
  }
  return total;
}

}  // namespace pat
