// Checkpointing schedules (host only).
//
// Counting follows binomial checkpointing (Griewank and Walther), which the
// paper uses as R(n, s) in Section 3: with s slots, the one that holds the
// interval's first state included, reversing l steps needs at least
//   F(l, s) = r l - beta(s + 1, r - 1)   advanced steps,
// beta(s, r) = C(s + r, s), r the integer with beta(s, r-1) < l <= beta(s, r).
// Schedules are built recursively: advance m steps, snapshot, reverse the
// right part with one slot fewer, restore, reverse the left part.  Every m in
// [max(1, l - beta(s-1, r), beta(s, r-2)), min(l-1, beta(s, r-1),
// l - beta(s-1, r-1))] is optimal; the largest is taken.
//
// The two-level policy (Section 2) stores every I-th state of the forward
// sweep to the slow level, prefetches interval starts one interval ahead in
// the reverse sweep, and reverses each interval with the remaining fast slots;
// I = ceil(T_T / T_A) (Section 3), raised to ceil(n / (H+1)) so the stored
// states fit H slow slots.  Fast slots 0 and 1 alternate as interval bases.
// If the result would not need strictly fewer forward evaluations than plain
// Revolve at the same s, plain Revolve is used (generalising the fallback at
// the end of Section 3).
#include "schedule.hpp"

#include <algorithm>
#include <cstdio>
#include <functional>
#include <memory>
#include <queue>
#include <stdexcept>
#include <unordered_map>

namespace ambptt {

int64_t binom_beta(int64_t s, int64_t r) {
  if (s < 0 || r < 0) return 0;
  const int64_t N = s + r;
  const int64_t k = std::min(s, r);
  int64_t c = 1;
  for (int64_t i = 1; i <= k; ++i) {
    const int64_t f = N - k + i;
    if (c > kBig / f) return kBig;
    c = c * f / i;  // c == C(N - k + i, i), exact
  }
  return c;
}

static int64_t revolve_r(int64_t l, int64_t s) {
  int64_t r = 0;
  while (binom_beta(s, r) < l) ++r;
  return r;
}

int64_t revolve_advances(int64_t l, int64_t s) {
  if (l < 1 || s < 1) return -1;
  const int64_t r = revolve_r(l, s);
  return r * l - binom_beta(s + 1, r - 1);
}

int64_t revolve_split(int64_t l, int64_t s) {
  const int64_t r = revolve_r(l, s);
  int64_t hi = l - 1;
  hi = std::min(hi, binom_beta(s, r - 1));
  hi = std::min(hi, l - binom_beta(s - 1, r - 1));
  return hi;
}

void plan_counts(int64_t n, int32_t s, int64_t H, int64_t interval_min, bool* async,
                 int64_t* interval, int64_t* evals) {
  if (n < 1 || s < 1 || H < 0 || interval_min < 0)
    throw std::invalid_argument("schedule: need n >= 1, s >= 1, H >= 0, I_min >= 0");
  const int64_t plain = revolve_advances(n, s) + 1;
  *async = false;
  *interval = 0;
  *evals = plain;
  if (H <= 0 || s < 2) return;
  int64_t I = std::max<int64_t>(interval_min, 1);
  I = std::max<int64_t>(I, (n + H) / (H + 1));  // ceil(n / (H + 1))
  if (I >= n) return;
  const int64_t K = (n + I - 1) / I;
  const int64_t last = n - (K - 1) * I;
  const int64_t ev = (K - 1) * I + revolve_advances(last, s - 1) + 1 +
                     (K - 1) * revolve_advances(I, s - 1);
  if (ev >= plain) return;
  *async = true;
  *interval = I;
  *evals = ev;
}

namespace {

struct Builder {
  int64_t n;
  std::vector<Action>* out;
  int64_t live = 0;
  std::vector<char> busy;  // fast slot occupied by an active snapshot
  // split of a reversal of [a, a + l) with s >= 2 slots (default: Revolve's largest optimal one)
  std::function<int64_t(int64_t, int64_t, int64_t)> split;

  void push(Op op, int64_t a, int64_t b = 0, int64_t c = 0) { out->push_back({op, a, b, c}); }
  void turn(int64_t t) { push(t == n - 1 ? Op::First : Op::Youturn, t); }
  void restore(int64_t k, int64_t a) {
    if (live != a) {
      push(Op::Restore, k, a);
      live = a;
    }
  }
  void advance(int64_t t0, int64_t t1) {
    push(Op::Advance, t0, t1);
    live = t1;
  }
  int64_t take_slot() {
    for (size_t k = 0; k < busy.size(); ++k)
      if (!busy[k]) {
        busy[k] = 1;
        return int64_t(k);
      }
    throw std::logic_error("schedule: no free slot");
  }

  // Reverse [a, a + l) with s slots; x_a sits in slot `base`.
  void reverse(int64_t a, int64_t l, int64_t s, int64_t base) {
    for (;;) {
      if (l == 1) {
        restore(base, a);
        turn(a);
        return;
      }
      if (s == 1) {
        for (int64_t i = l - 1; i >= 0; --i) {
          restore(base, a);
          if (i > 0) advance(a, a + i);
          turn(a + i);
        }
        return;
      }
      const int64_t m = split ? split(a, l, s) : revolve_split(l, s);
      restore(base, a);
      advance(a, a + m);
      const int64_t k = take_slot();
      push(Op::Snap, k, a + m);
      reverse(a + m, l - m, s - 1, k);
      busy[size_t(k)] = 0;
      l = m;  // the left part, same slots and base
    }
  }
};

// The two-level policy over interval starts t_0 = 0 < t_1 < ... < t_{K-1}
// (Section 2): the sweep snapshots each start but the last into fast slot
// k % 2 and stores it to host slot k; the reverse takes the intervals from the
// last, prefetching the previous start one interval ahead, and reverses each
// with Revolve on s - 1 slots (fast slots 0 and 1 hold the starts; Revolve
// works in 2 .. s-1).
void two_level(Builder& b, int32_t s, const std::vector<int64_t>& starts) {
  const int64_t K = int64_t(starts.size());
  b.busy[0] = b.busy[1] = 1;
  for (int64_t k = 0; k + 1 < K; ++k) {
    b.push(Op::Snap, k % 2, starts[size_t(k)]);
    b.push(Op::Store, k % 2, k, starts[size_t(k)]);
    b.advance(starts[size_t(k)], starts[size_t(k + 1)]);
  }
  for (int64_t k = K - 1; k >= 0; --k) {
    const int64_t a = starts[size_t(k)];
    const int64_t l = (k == K - 1 ? b.n : starts[size_t(k + 1)]) - a;
    const int64_t base = k % 2;
    if (k == K - 1) b.push(Op::Snap, base, a);
    if (k >= 1) b.push(Op::Prefetch, k - 1, (k - 1) % 2, starts[size_t(k - 1)]);
    b.reverse(a, l, s - 1, base);
  }
}

}  // namespace

namespace {

// Least cost of reversing [a, a + l) with k slots for unequal step costs, and
// the split that reaches it.  Queries come top-down, one reversal at a time:
// a query outside the current root reversal fills a new table for that root,
// bottom-up over (k, l, a), dense and indexed by (a - a0, l, k).
class WeightedSplits {
 public:
  WeightedSplits(const std::vector<double>& costs, int64_t max_table) : max_table_(max_table) {
    pre_.assign(costs.size() + 1, 0.0);
    for (size_t t = 0; t < costs.size(); ++t) pre_[t + 1] = pre_[t] + costs[t];
  }
  double C(int64_t a, int64_t b) const { return pre_[size_t(b)] - pre_[size_t(a)]; }
  int64_t split(int64_t a, int64_t l, int64_t k) {
    if (!(a >= a0_ && a + l <= a0_ + L_ && k <= K_)) fill(a, l, k);
    return m_[idx(a, l, k)];
  }

 private:
  size_t idx(int64_t a, int64_t l, int64_t k) const { return size_t(((a - a0_) * (L_ + 1) + l) * (K_ + 1) + k); }
  void fill(int64_t a0, int64_t L, int64_t K) {
    if (L * (L + 1) * (K + 1) > max_table_) throw std::length_error("schedule: cost table too large");
    a0_ = a0, L_ = L, K_ = K;
    v_.assign(size_t(L * (L + 1) * (K + 1)), 0.0);
    m_.assign(v_.size(), 0);
    // one slot: restore x_a and advance i steps for i = l-1 .. 1, summed in increasing i
    for (int64_t a = a0; a < a0 + L; ++a)
      for (int64_t l = 2; a + l <= a0 + L; ++l) v_[idx(a, l, 1)] = v_[idx(a, l - 1, 1)] + C(a, a + l - 1);
    for (int64_t k = 2; k <= K; ++k)
      for (int64_t l = 2; l <= L; ++l)
        for (int64_t a = a0; a + l <= a0 + L; ++a) {
          double best = 0.0;
          int64_t bm = -1;
          for (int64_t m = 1; m < l; ++m) {
            const double v = C(a, a + m) + v_[idx(a + m, l - m, k - 1)] + v_[idx(a, m, k)];
            if (bm < 0 || v <= best) best = v, bm = m;
          }
          v_[idx(a, l, k)] = best;
          m_[idx(a, l, k)] = int32_t(bm);
        }
  }
  std::vector<double> pre_;
  std::vector<double> v_;
  std::vector<int32_t> m_;
  int64_t a0_ = 0, L_ = 0, K_ = 0, max_table_;
};

}  // namespace

Plan make_plan(int64_t n, int32_t s, int64_t H, int64_t interval_min) {
  Plan p;
  p.n = n;
  p.s = s;
  p.H = H;
  plan_counts(n, s, H, interval_min, &p.async, &p.interval, &p.evals);
  Builder b{n, &p.acts, 0, std::vector<char>(size_t(s), 0)};
  if (!p.async) {
    b.push(Op::Snap, 0, 0);
    b.busy[0] = 1;
    b.reverse(0, n, s, 0);
    return p;
  }
  std::vector<int64_t> starts;
  for (int64_t t = 0; t < n; t += p.interval) starts.push_back(t);
  two_level(b, s, starts);
  p.host_slots_used = int64_t(starts.size()) - 1;
  return p;
}

Plan make_plan_starts(int64_t n, int32_t s, int64_t H, const std::vector<int64_t>& starts,
                      const std::vector<double>* costs, double* cost_out) {
  if (n < 1 || s < 2 || H < 0 || starts.empty() || starts[0] != 0 || starts.back() >= n ||
      int64_t(starts.size()) - 1 > H)
    throw std::invalid_argument("schedule: need s >= 2 and starts 0 = t_0 < ... < t_{K-1} < n, K - 1 <= H");
  for (size_t k = 1; k < starts.size(); ++k)
    if (starts[k] <= starts[k - 1]) throw std::invalid_argument("schedule: interval starts must increase");
  if (costs && int64_t(costs->size()) != n) throw std::invalid_argument("schedule: need one cost per step");
  if (costs)
    for (double c : *costs)
      if (!(c > 0.0) || !(c < 1e300)) throw std::invalid_argument("schedule: step costs must be positive and finite");
  Plan p;
  p.n = n;
  p.s = s;
  p.H = H;
  p.async = true;
  p.dynamic = true;
  Builder b{n, &p.acts, 0, std::vector<char>(size_t(s), 0), {}};
  std::unique_ptr<WeightedSplits> ws;
  if (costs) {
    ws.reset(new WeightedSplits(*costs, int64_t(1) << 20));
    b.split = [&ws](int64_t a, int64_t l, int64_t k) { return ws->split(a, l, k); };
    p.weighted = true;
  }
  two_level(b, s, starts);
  p.host_slots_used = int64_t(starts.size()) - 1;
  p.evals = 1;
  double cost = costs ? (*costs)[size_t(n - 1)] : 0.0;
  for (const Action& x : p.acts)
    if (x.op == Op::Advance) {
      p.evals += x.b - x.a;
      if (ws) cost += ws->C(x.a, x.b);
    }
  if (cost_out) *cost_out = costs ? cost : double(p.evals);
  return p;
}

int64_t OnlinePlacement::reverse_cost(const std::vector<int64_t>& h, int64_t end) const {
  int64_t c = 0;
  for (size_t j = 0; j < h.size(); ++j) {
    const int64_t l = (j + 1 < h.size() ? h[j + 1] : end) - h[j];
    c += revolve_advances(l, m_ - int64_t(j));
  }
  return c;
}

bool OnlinePlacement::decide(int64_t t, int64_t* dropped) {
  *dropped = -1;
  if (int64_t(held_.size()) < m_) {
    held_.push_back(t);
    return true;
  }
  const size_t k = held_.size() - 1;
  std::vector<int64_t> must, cand;
  for (;;) {
    // points of the phase-end placement already passed: they must stay held
    must.assign(1, a_);
    int64_t acc = a_;
    for (int64_t j = 0; j + 1 < m_; ++j) {
      acc += cap(j);
      if (acc > t) break;
      must.push_back(acc);
    }
    bool all_held = true, all_but_t = true;  // every passed point held (or equal to t)
    for (int64_t q : must) {
      const bool in = std::binary_search(held_.begin(), held_.end(), q);
      all_held = all_held && in;
      all_but_t = all_but_t && (in || q == t);
    }
    int64_t best = -1, best_j = -1;
    bool best_skip = false;
    for (size_t j = 1; j <= k && all_but_t; ++j) {
      const int64_t nxt = j < k ? held_[j + 1] : t;
      if (nxt - held_[j - 1] > cap(int64_t(j) - 1)) continue;
      if (std::binary_search(must.begin(), must.end(), held_[j])) continue;
      cand.assign(held_.begin(), held_.end());
      cand.erase(cand.begin() + long(j));
      cand.push_back(t);
      const int64_t c = reverse_cost(cand, t + 1);
      if (best < 0 || c < best) best = c, best_j = int64_t(j);
    }
    if (all_held && t + 1 - held_[k] <= cap(int64_t(k))) {
      const int64_t c = reverse_cost(held_, t + 1);
      if (best < 0 || c < best) best = c, best_skip = true;
    }
    if (best >= 0) {
      if (best_skip) return false;
      *dropped = held_[size_t(best_j)];
      held_.erase(held_.begin() + long(best_j));
      held_.push_back(t);
      return true;
    }
    ++r_;
  }
}

Plan make_plan_online(int64_t n, int32_t s, int64_t H, int64_t interval_min) {
  if (n < 1 || s < 1 || H < 0 || interval_min < 0)
    throw std::invalid_argument("schedule: need n >= 1, s >= 1, H >= 0, I_min >= 0");
  Plan p;
  p.n = n;
  p.s = s;
  p.H = H;
  p.online = true;
  const bool two = H > 0 && s >= 2;
  p.async = two;
  p.interval = two ? std::max<int64_t>(interval_min, 1) : 0;
  Builder b{n, &p.acts, 0, std::vector<char>(size_t(s), 0)};
  const int64_t m = two ? s - 1 : s;
  const int64_t w0 = two ? 2 : 1;  // first working slot
  std::vector<int64_t> slot_of_t(size_t(n), -1);  // fast slot of a held state
  std::vector<char> used(size_t(s), 0);
  auto lowest_free_work = [&]() {
    for (int64_t k = w0; k < s; ++k)
      if (!used[size_t(k)]) return k;
    throw std::logic_error("schedule: no free working slot");
  };
  int64_t run = 0;  // first step of the advance not yet emitted
  auto flush = [&](int64_t t) {
    if (run < t) b.advance(run, t);
    run = t;
  };
  b.push(Op::Snap, 0, 0);
  slot_of_t[0] = 0;
  int64_t base = 0, I = p.interval;
  OnlinePlacement pol(m, 0);
  struct Start {
    int64_t t, h;
  };
  std::vector<Start> starts;
  std::priority_queue<int64_t, std::vector<int64_t>, std::greater<int64_t>> released;
  int64_t fresh = 1;  // next never-used host slot
  if (two) {
    b.push(Op::Store, 0, 0, 0);
    starts.push_back({0, 0});
  }
  for (int64_t t = 1; t < n - 1; ++t) {
    if (two && t % I == 0) {
      while (released.empty() && fresh >= H && t % I == 0) {  // no host slot: double I
        I *= 2;
        std::vector<Start> keep;
        for (const Start& st : starts) {
          if (st.t % I == 0) keep.push_back(st);
          else released.push(st.h);
        }
        starts.swap(keep);
      }
      if (t % I == 0) {  // x_t starts an interval
        flush(t);
        for (int64_t k = w0; k < s; ++k) used[size_t(k)] = 0;
        base = 1 - base;
        b.push(Op::Snap, base, t);
        int64_t h;
        if (!released.empty()) {
          h = released.top();
          released.pop();
        } else {
          h = fresh++;
        }
        b.push(Op::Store, base, h, t);
        starts.push_back({t, h});
        pol = OnlinePlacement(m, t);
        slot_of_t[size_t(t)] = base;
        continue;
      }
    }
    int64_t dropped;
    if (!pol.decide(t, &dropped)) continue;
    if (dropped >= 0) used[size_t(slot_of_t[size_t(dropped)])] = 0;
    const int64_t k = lowest_free_work();
    used[size_t(k)] = 1;
    flush(t);
    b.push(Op::Snap, k, t);
    slot_of_t[size_t(t)] = k;
  }
  flush(n - 1);
  if (two && starts.size() >= 2) {
    const Start& st = starts[starts.size() - 2];
    b.push(Op::Prefetch, st.h, 1 - base, st.t);
  }
  b.turn(n - 1);
  // the placement's segments, from the last down; segment j has m - j slots
  const std::vector<int64_t>& held = pol.held();
  for (size_t j = held.size(); j-- > 0;) {
    const int64_t l = (j + 1 < held.size() ? held[j + 1] : n - 1) - held[j];
    if (l <= 0) continue;
    std::fill(b.busy.begin(), b.busy.end(), 0);
    if (two) b.busy[0] = b.busy[1] = 1;
    for (size_t i = 0; i <= j; ++i) b.busy[size_t(slot_of_t[size_t(held[i])])] = 1;
    b.reverse(held[j], l, m - int64_t(j), slot_of_t[size_t(held[j])]);
  }
  if (two) {
    std::fill(b.busy.begin(), b.busy.end(), 0);
    b.busy[0] = b.busy[1] = 1;
    for (size_t k = starts.size() - 1; k-- > 0;) {
      base = 1 - base;
      if (k >= 1) b.push(Op::Prefetch, starts[k - 1].h, 1 - base, starts[k - 1].t);
      b.reverse(starts[k].t, starts[k + 1].t - starts[k].t, s - 1, base);
    }
    p.host_slots_used = fresh;
  }
  p.evals = 1;
  for (const Action& x : p.acts)
    if (x.op == Op::Advance) p.evals += x.b - x.a;
  return p;
}

Plan make_plan_costs(int64_t n, int32_t s, int64_t H, int64_t interval_min, const std::vector<double>& costs,
                     double* cost_out, int64_t max_table) {
  if (int64_t(costs.size()) != n) throw std::invalid_argument("schedule: need one cost per step");
  for (double c : costs)
    if (!(c > 0.0) || !(c < 1e300)) throw std::invalid_argument("schedule: step costs must be positive and finite");
  Plan p;
  p.n = n;
  p.s = s;
  p.H = H;
  plan_counts(n, s, H, interval_min, &p.async, &p.interval, &p.evals);
  p.weighted = true;
  WeightedSplits ws(costs, max_table);
  Builder b{n, &p.acts, 0, std::vector<char>(size_t(s), 0), {}};
  b.split = [&ws](int64_t a, int64_t l, int64_t k) { return ws.split(a, l, k); };
  if (!p.async) {
    b.push(Op::Snap, 0, 0);
    b.busy[0] = 1;
    b.reverse(0, n, s, 0);
  } else {
    std::vector<int64_t> starts;
    for (int64_t t = 0; t < n; t += p.interval) starts.push_back(t);
    two_level(b, s, starts);
    p.host_slots_used = int64_t(starts.size()) - 1;
  }
  p.evals = 1;
  double cost = 0.0;
  for (const Action& x : p.acts)
    if (x.op == Op::Advance) {
      p.evals += x.b - x.a;
      cost += ws.C(x.a, x.b);
    }
  cost += costs[size_t(n - 1)];
  if (cost_out) *cost_out = cost;
  return p;
}

std::string plan_text(const Plan& p) {
  std::string t;
  t.reserve(p.acts.size() * 12 + 96);
  t += "ambptt-schedule v1 n=" + std::to_string(p.n) + " s=" + std::to_string(p.s) +
       " H=" + std::to_string(p.H) + " I=" + std::to_string(p.dynamic ? 0 : p.interval) +
       " mode=" + (p.online ? "online" : p.dynamic ? "dynamic" : p.async ? "async" : "revolve") +
       (p.sized ? " split=size" : p.weighted ? " split=cost" : "") + "\n";
  char line[96];
  for (const Action& x : p.acts) {
    int len = 0;
    switch (x.op) {
      case Op::Advance: len = snprintf(line, sizeof line, "A %lld %lld\n", (long long)x.a, (long long)x.b); break;
      case Op::Snap: len = snprintf(line, sizeof line, "S %lld %lld\n", (long long)x.a, (long long)x.b); break;
      case Op::Restore: len = snprintf(line, sizeof line, "R %lld %lld\n", (long long)x.a, (long long)x.b); break;
      case Op::First: len = snprintf(line, sizeof line, "F %lld\n", (long long)x.a); break;
      case Op::Youturn: len = snprintf(line, sizeof line, "Y %lld\n", (long long)x.a); break;
      case Op::Store:
        len = snprintf(line, sizeof line, "W %lld %lld %lld\n", (long long)x.a, (long long)x.b, (long long)x.c);
        break;
      case Op::Prefetch:
        len = snprintf(line, sizeof line, "P %lld %lld %lld\n", (long long)x.a, (long long)x.b, (long long)x.c);
        break;
    }
    t.append(line, size_t(len));
  }
  return t;
}

namespace {

// Least cost of reversing [a, a + l) with M units free above x_a when the
// states differ in size, and the split that reaches it (0: the chain).  One
// dense table per root reversal [a0, a0 + L) with budget M0, filled
// bottom-up over (M, l, a) and indexed by (a - a0, l, M).  A part whose
// states x_{a+1} .. x_{a+l-1} all fit in M needs no table: splitting at 1 at
// every level advances each step once, which every other split exceeds by a
// positive cost, so it is the recursion's unique optimum.
class SizedSplits {
 public:
  SizedSplits(const std::vector<int64_t>& sizes, const std::vector<double>* costs, int64_t max_table)
      : z_(sizes), max_table_(max_table) {
    const size_t n = sizes.size() - 1;
    pre_.assign(n + 1, 0.0);
    for (size_t t = 0; t < n; ++t) pre_[t + 1] = pre_[t] + (costs ? (*costs)[t] : 1.0);
    zpre_.assign(n + 2, 0);
    for (size_t t = 0; t <= n; ++t) zpre_[t + 1] = zpre_[t] + sizes[t];
  }
  double C(int64_t a, int64_t b) const { return pre_[size_t(b)] - pre_[size_t(a)]; }
  bool fits(int64_t a, int64_t l, int64_t M) const {
    return l <= 1 || zpre_[size_t(a + l)] - zpre_[size_t(a + 1)] <= M;
  }
  int64_t split(int64_t a, int64_t l, int64_t M) {
    if (fits(a, l, M)) return 1;
    ensure(a, l, M);
    return m_[idx(a, l, M)];
  }
  double T(int64_t a, int64_t l, int64_t M) {
    if (fits(a, l, M)) return l <= 1 ? 0.0 : C(a, a + l - 1);
    ensure(a, l, M);
    return v_[idx(a, l, M)];
  }
  int64_t z(int64_t t) const { return z_[size_t(t)]; }

 private:
  void ensure(int64_t a, int64_t l, int64_t M) {
    if (!(a >= a0_ && a + l <= a0_ + L_ && M <= M0_)) fill(a, l, M);
  }
  size_t idx(int64_t a, int64_t l, int64_t M) const { return size_t(((a - a0_) * (L_ + 1) + l) * (M0_ + 1) + M); }
  void fill(int64_t a0, int64_t L, int64_t M0) {
    if (M0 < 0) M0 = 0;
    if (double(L) * double(L + 1) * double(M0 + 1) > double(max_table_))
      throw std::length_error("schedule: sized table too large");
    a0_ = a0, L_ = L, M0_ = M0;
    v_.assign(size_t(L * (L + 1) * (M0 + 1)), 0.0);
    m_.assign(v_.size(), 0);
    std::vector<double> chain(size_t(L + 1));
    for (int64_t M = 0; M <= M0; ++M)
      for (int64_t a = a0; a < a0 + L; ++a) {
        // the chain from x_a: restore it and advance i steps, i = l-1 .. 1
        chain[1] = 0.0;
        for (int64_t l = 2; a + l <= a0 + L; ++l) chain[size_t(l)] = chain[size_t(l - 1)] + C(a, a + l - 1);
        for (int64_t l = 2; a + l <= a0 + L; ++l) {
          double best = 0.0;
          int64_t bm = 0;
          for (int64_t m = 1; m < l; ++m) {
            const int64_t zm = z_[size_t(a + m)];
            if (zm > M) continue;
            const double v = C(a, a + m) + v_[idx(a + m, l - m, M - zm)] + v_[idx(a, m, M)];
            if (bm == 0 || v <= best) best = v, bm = m;
          }
          if (bm == 0) best = chain[size_t(l)];
          v_[idx(a, l, M)] = best;
          m_[idx(a, l, M)] = int32_t(bm);
        }
      }
  }
  std::vector<int64_t> z_, zpre_;
  std::vector<double> pre_, v_;
  std::vector<int32_t> m_;
  int64_t a0_ = 0, L_ = 0, M0_ = -1, max_table_;
};

struct SizedBuilder {
  Builder& b;
  SizedSplits& ss;
  // Reverse [a, a + l) with M units free above x_a (in slot `base`); the next
  // snapshot goes to slot `depth`, the top of the stack.
  void reverse(int64_t a, int64_t l, int64_t M, int64_t base, int64_t depth) {
    for (;;) {
      if (l == 1) {
        b.restore(base, a);
        b.turn(a);
        return;
      }
      const int64_t m = ss.split(a, l, M);
      if (m == 0) {
        for (int64_t i = l - 1; i >= 0; --i) {
          b.restore(base, a);
          if (i > 0) b.advance(a, a + i);
          b.turn(a + i);
        }
        return;
      }
      b.restore(base, a);
      b.advance(a, a + m);
      b.push(Op::Snap, depth, a + m);
      reverse(a + m, l - m, M - ss.z(a + m), depth, depth + 1);
      l = m;
    }
  }
};

// The sweep and reverse of the two-level policy with the sized recursion in
// every interval (M units above each start).
void two_level_sized(Builder& b, SizedSplits& ss, const std::vector<int64_t>& starts, int64_t M) {
  const int64_t K = int64_t(starts.size());
  for (int64_t k = 0; k + 1 < K; ++k) {
    b.push(Op::Snap, k % 2, starts[size_t(k)]);
    b.push(Op::Store, k % 2, k, starts[size_t(k)]);
    b.advance(starts[size_t(k)], starts[size_t(k + 1)]);
  }
  SizedBuilder sb{b, ss};
  for (int64_t k = K - 1; k >= 0; --k) {
    const int64_t a = starts[size_t(k)];
    const int64_t l = (k == K - 1 ? b.n : starts[size_t(k + 1)]) - a;
    if (k == K - 1) b.push(Op::Snap, k % 2, a);
    if (k >= 1) b.push(Op::Prefetch, k - 1, (k - 1) % 2, starts[size_t(k - 1)]);
    sb.reverse(a, l, M, k % 2, 2);
  }
}

// Unit offsets of every action's fast slot in the stack layout.
void sized_offsets(Plan& p, const std::vector<int64_t>& z, bool two) {
  const int64_t zmax = *std::max_element(z.begin(), z.end());
  std::vector<int64_t> content;
  auto off = [&](int64_t k) -> int64_t {
    if (two && k <= 1) return k * zmax;
    int64_t o = two ? 2 * zmax : 0;
    for (int64_t j = two ? 2 : 0; j < k; ++j) {
      if (size_t(j) >= content.size() || content[size_t(j)] < 0) throw std::logic_error("schedule: empty slot below");
      o += z[size_t(content[size_t(j)])];
    }
    return o;
  };
  int64_t ids = 0;
  for (Action& x : p.acts) {
    int64_t k = -1, t = -1;
    if (x.op == Op::Snap) k = x.a, t = x.b;
    else if (x.op == Op::Restore || x.op == Op::Store) k = x.a;
    else if (x.op == Op::Prefetch) k = x.b, t = x.c;
    if (k < 0) continue;
    ids = std::max(ids, k + 1);
    x.off = off(k);
    if (t >= 0) {
      if (content.size() <= size_t(k)) content.resize(size_t(k) + 1, -1);
      content[size_t(k)] = t;
    }
  }
  p.slot_ids = ids;
}

void sized_check_args(int64_t n, int32_t s, int64_t H, const std::vector<int64_t>& sizes,
                      const std::vector<double>* costs) {
  if (n < 1 || s < 1 || H < 0 || int64_t(sizes.size()) != n + 1)
    throw std::invalid_argument("schedule: need n >= 1, s >= 1, H >= 0 and n + 1 sizes");
  for (int64_t z : sizes)
    if (z < 1 || z > (int64_t(1) << 40)) throw std::invalid_argument("schedule: sizes must be positive");
  if (costs) {
    if (int64_t(costs->size()) != n) throw std::invalid_argument("schedule: need one cost per step");
    for (double c : *costs)
      if (!(c > 0.0) || !(c < 1e300)) throw std::invalid_argument("schedule: step costs must be positive and finite");
  }
}

void sized_finish(Plan& p, SizedSplits& ss, const std::vector<double>* costs, double* cost_out) {
  p.sized = true;
  p.weighted = costs != nullptr;
  p.evals = 1;
  double cost = 0.0;
  for (const Action& x : p.acts)
    if (x.op == Op::Advance) {
      p.evals += x.b - x.a;
      cost += ss.C(x.a, x.b);
    }
  cost += ss.C(p.n - 1, p.n);
  if (cost_out) *cost_out = cost;
}

}  // namespace

Plan make_plan_sized(int64_t n, int32_t s, int64_t H, int64_t interval_min, const std::vector<int64_t>& sizes,
                     const std::vector<double>* costs, double* cost_out, int64_t max_table) {
  sized_check_args(n, s, H, sizes, costs);
  if (interval_min < 0) throw std::invalid_argument("schedule: interval_min must be >= 0");
  SizedSplits ss(sizes, costs, max_table);
  const int64_t zmax = *std::max_element(sizes.begin(), sizes.end());
  const int64_t P = int64_t(s) * zmax;
  // the plain reversal's cost; a table too large for it leaves only two levels
  double plain = 0.0;
  bool plain_ok = true;
  try {
    plain = ss.T(0, n, P - sizes[0]);
  } catch (const std::length_error&) {
    plain_ok = false;
  }
  Plan p;
  p.n = n;
  p.s = s;
  p.H = H;
  std::vector<int64_t> starts;
  if (H > 0 && s >= 2) {
    const int64_t I = std::max<int64_t>({interval_min, 1, (n + H) / (H + 1)});
    if (I < n) {
      for (int64_t t = 0; t < n; t += I) starts.push_back(t);
      double c = ss.C(0, starts.back());
      for (size_t k = 0; k < starts.size(); ++k) {
        const int64_t e = k + 1 < starts.size() ? starts[k + 1] : n;
        c += ss.T(starts[k], e - starts[k], P - 2 * zmax);
      }
      if (!plain_ok || c < plain) {
        p.async = true;
        p.interval = I;
      }
    }
  }
  if (!p.async && !plain_ok) throw std::length_error("schedule: sized table too large");
  Builder b{n, &p.acts, 0, std::vector<char>(size_t(s), 0), {}};
  if (!p.async) {
    b.push(Op::Snap, 0, 0);
    SizedBuilder{b, ss}.reverse(0, n, P - sizes[0], 0, 1);
  } else {
    two_level_sized(b, ss, starts, P - 2 * zmax);
    p.host_slots_used = int64_t(starts.size()) - 1;
  }
  sized_offsets(p, sizes, p.async);
  sized_finish(p, ss, costs, cost_out);
  return p;
}

Plan make_plan_sized_starts(int64_t n, int32_t s, int64_t H, const std::vector<int64_t>& starts,
                            const std::vector<int64_t>& sizes, const std::vector<double>* costs, double* cost_out,
                            int64_t max_table) {
  sized_check_args(n, s, H, sizes, costs);
  if (s < 2 || starts.empty() || starts[0] != 0 || starts.back() >= n || int64_t(starts.size()) - 1 > H)
    throw std::invalid_argument("schedule: need s >= 2 and starts 0 = t_0 < ... < t_{K-1} < n, K - 1 <= H");
  for (size_t k = 1; k < starts.size(); ++k)
    if (starts[k] <= starts[k - 1]) throw std::invalid_argument("schedule: interval starts must increase");
  SizedSplits ss(sizes, costs, max_table);
  const int64_t zmax = *std::max_element(sizes.begin(), sizes.end());
  Plan p;
  p.n = n;
  p.s = s;
  p.H = H;
  p.async = true;
  p.dynamic = true;
  Builder b{n, &p.acts, 0, std::vector<char>(size_t(s), 0), {}};
  two_level_sized(b, ss, starts, int64_t(s - 2) * zmax);
  p.host_slots_used = int64_t(starts.size()) - 1;
  sized_offsets(p, sizes, true);
  sized_finish(p, ss, costs, cost_out);
  return p;
}

}  // namespace ambptt
