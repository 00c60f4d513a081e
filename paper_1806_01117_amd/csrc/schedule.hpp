// Host-side checkpointing schedule generator: binomial (Revolve) schedules
// within one memory level, and the asynchronous two-level policy of
// Section 2 with the interval rule of Section 3.  Pure C++, no HIP.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

namespace ambptt {

enum class Op : uint8_t { Advance, Snap, Restore, First, Youturn, Store, Prefetch };

// Action operands:
//   Advance  a = t0, b = t1        Snap/Restore  a = slot, b = t
//   First/Youturn  a = t           Store    a = slot, b = host, c = t
//   Prefetch a = host, b = slot, c = t
struct Action {
  Op op;
  int64_t a, b, c;
  // sized plans: offset of the action's fast slot in units of the pool's
  // granule (Snap, Restore, Store, Prefetch); -1 elsewhere
  int64_t off = -1;
};

struct Plan {
  int64_t n = 0;
  int32_t s = 0;
  int64_t H = 0;
  int64_t interval = 0;  // 0 in Revolve mode
  bool async = false;
  bool dynamic = false;  // interval starts decided during the sweep
  bool online = false;   // placement decided without knowing n (interval = the first I)
  bool weighted = false; // splits chosen for unequal step costs
  bool sized = false;    // states of different sizes in a byte-addressed pool (Action::off set)
  int64_t slot_ids = 0;  // fast slot ids used (sized plans may stack more states than s)
  int64_t evals = 0;     // forward-step evaluations
  int64_t host_slots_used = 0;
  std::vector<Action> acts;
};

// C(s + r, s), saturating at kBig.
constexpr int64_t kBig = int64_t(1) << 60;
int64_t binom_beta(int64_t s, int64_t r);
// Least advanced steps that reverse l steps with s slots.
int64_t revolve_advances(int64_t l, int64_t s);
// Largest optimal first split for reversing l steps with s >= 2 slots.
int64_t revolve_split(int64_t l, int64_t s);

// Chooses the mode and interval and builds the action list.  Throws
// std::invalid_argument on bad arguments.
Plan make_plan(int64_t n, int32_t s, int64_t H, int64_t interval_min);
// The two-level plan over interval starts decided during the sweep (the
// starts increase from 0, stay below n and number at most H + 1; s >= 2).
// Throws std::invalid_argument otherwise.
// With costs (one per step, see make_plan_costs) every reversal is split for
// them; *cost_out (nullable) then receives the cost of the forward evaluations.
Plan make_plan_starts(int64_t n, int32_t s, int64_t H, const std::vector<int64_t>& starts,
                      const std::vector<double>* costs = nullptr, double* cost_out = nullptr);
// Online checkpointing: every decision about x_t is taken when x_t is
// computed, knowing only that step t exists; the actions before the sweep
// reaches x_{n-1} are the same for every longer n.  H = 0 (or s = 1): one
// level, placement in s fast slots.  H > 0: interval starts every I =
// max(I_min, 1) steps go to the host (I doubles and the starts that are not
// its multiples give their host slots back when a start finds none free),
// with the placement inside each interval on s - 1 slots.
Plan make_plan_online(int64_t n, int32_t s, int64_t H, int64_t interval_min);

// Placement of fast-slot checkpoints for a sweep from x_a whose end is not
// known.  Phase r: segment j (from the j-th held state to the next one, the
// last one to the live state) is at most beta(m - j, r - 1) steps long, so
// that reversing it with the m - j slots it then has advances every step at
// most r - 1 more times; the phase-end placement (every segment at its cap)
// must stay reachable.  Among the admissible moves (hold x_t in a free slot;
// give up the j-th held state for x_t; hold nothing new) the one with the
// least reversal cost if the sweep ended at step t + 1 is taken, holding
// before not, then the smallest j; with no admissible move the phase grows.
class OnlinePlacement {
 public:
  OnlinePlacement(int64_t m, int64_t a) : m_(m), a_(a), held_(1, a) {}
  // x_t has been computed and step t exists.  Returns true when x_t is to be
  // held; *dropped is then the time given up, or -1.
  bool decide(int64_t t, int64_t* dropped);
  const std::vector<int64_t>& held() const { return held_; }
  // Advances needed to reverse [a, end) from the placement h.
  int64_t reverse_cost(const std::vector<int64_t>& h, int64_t end) const;

 private:
  int64_t cap(int64_t j) const { return binom_beta(m_ - j, r_ - 1); }
  int64_t m_, a_, r_ = 1;
  std::vector<int64_t> held_;
};

// The schedule of make_plan (same mode, interval and slots) with every
// reversal of l >= 2 steps on k >= 2 slots split where it costs least for
// forward steps of unequal cost (costs[t] > 0 for step t), by dynamic
// programming over the same recursion:
//   T(a, 1, k) = 0,  T(a, l, 1) = sum_{i=1}^{l-1} C(a, a+i),
//   T(a, l, k) = min_m C(a, a+m) + T(a+m, l-m, k-1) + T(a, m, k),
// C(a, b) the cost of steps a .. b-1, ties to the largest m (equal costs give
// make_plan's schedule).  The table of one reversal of l steps on k slots has
// l (l + 1) (k + 1) entries and takes about l^3 k / 6 operations.
// *cost_out (nullable) receives the cost of every forward evaluation of the
// schedule.  Throws std::invalid_argument on bad arguments and
// std::length_error when a reversal's table would exceed max_table entries.
Plan make_plan_costs(int64_t n, int32_t s, int64_t H, int64_t interval_min, const std::vector<double>& costs,
                     double* cost_out, int64_t max_table = int64_t(1) << 20);

// States of different sizes: sizes[t] (t = 0 .. n, >= 1) is the size of
// x_t in units of a common granule, and the fast pool holds s * max(sizes)
// units.  Snapshots stack: the one taken at recursion depth k (slot k) sits
// above the states in slots below it (in two levels slots 0 and 1 are the
// interval starts' regions of max(sizes) units each, the stack starting at
// 2 max(sizes)).  Every reversal of [a, a + l) with M units free above x_a
// splits by dynamic programming over Revolve's recursion with a budget:
//   T(a, 1, M) = 0,
//   T(a, l, M) = min over m with sizes[a+m] <= M of
//                C(a, a+m) + T(a+m, l-m, M - sizes[a+m]) + T(a, m, M),
// ties to the largest m, the chain (sum_{i=1}^{l-1} C(a, a+i)) when no
// snapshot fits; C(a, b) the cost of steps a .. b-1 (costs, or 1 each).
// Plain: M = s max(sizes) - sizes[0] over [0, n); two levels (H > 0, s >= 2,
// I = max(I_min, 1, ceil(n / (H + 1))) < n) when strictly cheaper, every
// interval on M = (s - 2) max(sizes).  Unit sizes give make_plan's
// schedule.  Sets Action::off and slot_ids; *cost_out (nullable) receives the
// cost of the forward evaluations.  Throws std::invalid_argument on bad
// arguments and std::length_error when the table of the reversal the plan
// runs would exceed max_table entries (l (l + 1) (M + 1) per reversal).
Plan make_plan_sized(int64_t n, int32_t s, int64_t H, int64_t interval_min, const std::vector<int64_t>& sizes,
                     const std::vector<double>* costs, double* cost_out, int64_t max_table = int64_t(1) << 20);
// The two-level plan over interval starts decided during the sweep (as
// make_plan_starts) with every interval reversed by the sized recursion.
Plan make_plan_sized_starts(int64_t n, int32_t s, int64_t H, const std::vector<int64_t>& starts,
                            const std::vector<int64_t>& sizes, const std::vector<double>* costs, double* cost_out,
                            int64_t max_table = int64_t(1) << 20);

// Mode, interval and forward evaluations only (no action list).
void plan_counts(int64_t n, int32_t s, int64_t H, int64_t interval_min, bool* async,
                 int64_t* interval, int64_t* evals);

std::string plan_text(const Plan& p);

}  // namespace ambptt
