// Schedule -> resident kernel program.  The state bookkeeping (the live state
// aliases a slot after a RESTORE, a TAKESHOT right after an ADVANCE becomes
// that step's output, a prefetch into a slot that already holds its state is
// skipped) follows the per-step executor; on top of it the compiler places
// the extra barriers and waits that the kernel's transfer rules need.
#include "resident_prog.hpp"

#include <stdexcept>

namespace ambptt {

std::vector<int32_t> compile_resident(const Plan& plan, int nslots, bool elide_prefetch, ResidentCounts* counts) {
  ResidentCounts c;
  std::vector<int32_t> prog;
  const int L0 = nslots, L1 = nslots + 1, nbuf = nslots + 2;
  int cur = L0;                        // buffer holding the live state
  bool live_dead = false;              // the live state was consumed by an adjoint
  std::vector<int64_t> slot_t(size_t(nslots), -1);
  std::vector<int64_t> last_read(size_t(nbuf), 0);  // barrier of the last step reading the buffer
  int64_t bar = 0;                     // barriers so far
  int pend_pref = -1;                  // slot whose prefetch data wait for the next barrier

  auto emit = [&](int32_t op, int64_t y, int64_t z, int64_t w) {
    prog.push_back(op);
    prog.push_back(int32_t(y));
    prog.push_back(int32_t(z));
    prog.push_back(int32_t(w));
  };
  auto barrier_op = [&](int32_t op, int64_t y, int64_t z, int64_t w) {
    emit(op, y, z, w);
    ++bar;
    pend_pref = -1;  // flushed right after this barrier
  };
  auto sync = [&]() {
    barrier_op(kPSync, 0, 0, 0);
    c.extra_syncs++;
  };
  auto step = [&](int32_t op, int64_t t, int src, int64_t w) {
    if (pend_pref == src) sync();  // its data become readable only after one more barrier
    if (op == kPFwd && pend_pref == int(w)) sync();
    barrier_op(op, t, src, w);
    last_read[size_t(src)] = bar;
  };
  auto copy = [&](int src, int dst) {
    if (pend_pref == src || pend_pref == dst) sync();
    const int64_t wait = (bar > 0 && last_read[size_t(dst)] == bar) ? bar : 0;
    emit(kPCopy, wait, src, dst);
  };
  auto other_live = [&]() { return cur == L0 ? L1 : L0; };

  const auto& acts = plan.acts;
  for (size_t i = 0; i < acts.size(); ++i) {
    const Action& A = acts[i];
    switch (A.op) {
      case Op::Advance: {
        int fuse_k = -1;
        if (i + 1 < acts.size() && acts[i + 1].op == Op::Snap && acts[i + 1].b == A.b && acts[i + 1].a != cur)
          fuse_k = int(acts[i + 1].a);
        for (int64_t t = A.a; t < A.b; ++t) {
          const bool last = (t + 1 == A.b);
          const int dst = (last && fuse_k >= 0) ? fuse_k : other_live();
          step(kPFwd, t, cur, dst);
          c.forward_evals++;
          cur = dst;
        }
        if (fuse_k >= 0) {
          slot_t[size_t(fuse_k)] = A.b;
          c.takeshots++;
          ++i;
        }
        live_dead = false;
        break;
      }
      case Op::Snap: {
        c.takeshots++;
        if (cur == int(A.a)) {
          slot_t[size_t(A.a)] = A.b;
          break;
        }
        copy(cur, int(A.a));
        c.takeshot_copies++;
        slot_t[size_t(A.a)] = A.b;
        break;
      }
      case Op::Restore:
        c.restores++;
        cur = int(A.a);
        live_dead = false;
        break;
      case Op::First:
      case Op::Youturn: {
        const bool first = A.op == Op::First;
        step(kPAdj, A.a, cur, first ? 1 : 0);
        if (first) c.forward_evals++;
        c.adjoints++;
        live_dead = true;
        break;
      }
      case Op::Store: {
        if (pend_pref == int(A.a)) sync();
        // right after the step that wrote the slot, each workgroup still
        // holds its slice in LDS and need not read it back from HBM
        const size_t m = prog.size();
        const bool staged = m >= 4 && prog[m - 4] == kPFwd && prog[m - 1] == int32_t(A.a);
        emit(kPStore | (staged ? kPStaged : 0), 0, A.a, A.b);
        c.stores++;
        break;
      }
      case Op::Prefetch: {
        const int64_t h = A.a, k = A.b, t = A.c;
        c.prefetches++;
        if (elide_prefetch && slot_t[size_t(k)] == t) {
          c.prefetches_elided++;
          break;
        }
        if (cur == int(k) && !live_dead) {  // the live state aliases the target: keep it
          copy(int(k), L0);
          cur = L0;
        }
        if (pend_pref >= 0) sync();
        emit(kPPref, 0, h, k);
        pend_pref = int(k);
        slot_t[size_t(k)] = t;
        break;
      }
    }
  }
  barrier_op(kPEnd, 0, 0, 0);
  c.barriers = bar;
  // Each prefetch names the entry of the next one (y), whose host read the
  // kernel may then start when this one lands, as long as every store into
  // that host slot comes earlier in the program.
  {
    const size_t m = prog.size() / 4;
    std::vector<int64_t> last_store;  // host slot -> last entry storing it
    std::vector<size_t> prefs;
    for (size_t i = 0; i < m; ++i) {
      if ((prog[4 * i] & 0xFF) == kPPref) prefs.push_back(i);
    }
    for (size_t j = 0; j + 1 < prefs.size(); ++j) {
      const size_t i0 = prefs[j], i1 = prefs[j + 1];
      const int32_t h = prog[4 * i1 + 2];
      bool later_store = false;
      for (size_t i = i0; i < i1 && !later_store; ++i)
        later_store = (prog[4 * i] & 0xFF) == kPStore && prog[4 * i + 3] == h;
      if (!later_store) prog[4 * i0 + 1] = int32_t(i1);
    }
    (void)last_store;
  }
  if (c.forward_evals != plan.evals) throw std::logic_error("resident program: forward count differs from the schedule");
  if (counts) *counts = c;
  return prog;
}

}  // namespace ambptt
