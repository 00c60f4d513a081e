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
};

struct Plan {
  int64_t n = 0;
  int32_t s = 0;
  int64_t H = 0;
  int64_t interval = 0;  // 0 in Revolve mode
  bool async = false;
  bool dynamic = false;  // interval starts decided during the sweep
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
Plan make_plan_starts(int64_t n, int32_t s, int64_t H, const std::vector<int64_t>& starts);
// Mode, interval and forward evaluations only (no action list).
void plan_counts(int64_t n, int32_t s, int64_t H, int64_t interval_min, bool* async,
                 int64_t* interval, int64_t* evals);

std::string plan_text(const Plan& p);

}  // namespace ambptt
