// Compiles a checkpoint schedule into the action program of the resident
// whole-pass kernel.  Pure C++, no HIP.
#pragma once

#include <cstdint>
#include <vector>

#include "schedule.hpp"

namespace ambptt {

// Program entries are 4 ints {op, y, z, w}:
//   kPFwd   y = t, z = src buffer, w = dst buffer       forward step t
//   kPAdj   y = t, z = src buffer, w = 1 if first       adjoint step t
//   kPCopy  y = wait (0: none), z = src, w = dst        copy of a state
//   kPStore z = slot, w = host slot                     slot -> host tier
//           (| kPStaged: taken from the previous step's output in LDS)
//   kPPref  y = entry of the next kPPref whose host read may start when
//               this one lands (0: none), z = host slot, w = slot
//                                                       host tier -> slot
//   kPSync                                              group barrier only
//   kPEnd                                               dL/dx_0, dW, loss
// Buffer ids: 0 .. nslots-1 are the HBM slots, nslots and nslots+1 the two
// live buffers.  Every kPFwd, kPAdj, kPSync and kPEnd is one barrier of the
// workgroups that share batch rows; barriers are numbered 1, 2, ... in
// program order.  The kernel's rules, which the compiler keeps:
//   - a step writes its output after its barrier, so every member has left
//     the previous step;
//   - a prefetch's data reach the slot right after the next barrier and are
//     readable from the barrier after that, so a step reading a slot with a
//     prefetch in flight is preceded by a kPSync, and so is a second
//     prefetch;
//   - a copy into a buffer that the latest step read waits until every
//     member has read that step's inputs (y = that barrier's number).
enum ResidentOp : int32_t { kPEnd = 0, kPFwd = 1, kPAdj = 2, kPCopy = 3, kPStore = 4, kPPref = 5, kPSync = 6 };
// flag on kPStore (op | kPStaged): the previous entry is the forward step that
// wrote the slot, whose output slice the workgroup still holds in LDS
constexpr int32_t kPStaged = 1 << 8;

struct ResidentCounts {
  int64_t forward_evals = 0, adjoints = 0, takeshots = 0, takeshot_copies = 0, restores = 0;
  int64_t stores = 0, prefetches = 0, prefetches_elided = 0;
  int64_t barriers = 0, extra_syncs = 0;
};

std::vector<int32_t> compile_resident(const Plan& plan, int nslots, bool elide_prefetch, ResidentCounts* counts);

}  // namespace ambptt
