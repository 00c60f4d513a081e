// C-ABI runtime: context, checkpoint tiers, executor and calibration.
//
// Level 1 is the caller's HBM slot pool (s slots); Level 2 is pinned host
// memory owned here (Section 2).  The executor walks the action list on the
// host and enqueues:
//   - step kernels and state copies on the caller's compute stream,
//   - stores (slot -> host) and prefetches (host -> slot) on one copy stream,
// with event edges that keep the two streams race-free:
//   1. a store of slot k waits for the compute work that wrote slot k;
//   2. a later write of slot k by compute waits for that store to finish;
//   3. a prefetch into slot k waits for compute's earlier readers of slot k;
//   4. compute reads slot k only after the prefetch into it finished;
//   5. a prefetch of host slot h follows the store that filled it because one
//      in-order copy stream carries both directions.
// The copy stream never blocks the compute stream except through edges 2 and
// 4, which the interval rule I = ceil(T_T / T_A) (Section 3) is meant to keep
// already satisfied by the time they are reached.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <numeric>
#include <mutex>
#include <stdexcept>
#include <string>
#include <thread>
#include <vector>

#include "ambptt.h"
#include "kernels.hpp"
#include "resident_prog.hpp"
#include "schedule.hpp"
#include "tier_file.hpp"

using namespace ambptt;

namespace {

thread_local std::string g_err;

ambptt_status fail(ambptt_status s, const std::string& msg) {
  g_err = msg;
  return s;
}

#define HIPCK(expr)                                                                      \
  do {                                                                                   \
    hipError_t e_ = (expr);                                                              \
    if (e_ != hipSuccess) return fail(AMBPTT_EHIP, std::string(#expr) + ": " + hipGetErrorString(e_)); \
  } while (0)

constexpr size_t kAlign = 256;
size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

double now_us() {
  using namespace std::chrono;
  return duration<double, std::micro>(steady_clock::now().time_since_epoch()).count();
}

struct Layout {
  int G = 1, dsize = 4, window = 1;
  size_t h_bytes = 0, c_bytes = 0, state_bytes = 0, stride = 0;
  size_t off_live[2] = {0, 0}, off_wht = 0, off_zbar = 0, off_hwin = 0, off_cbar[2] = {0, 0};
  size_t off_wpk = 0, off_whpk = 0;  // wide bf16 cell: W and W_h^T in fragment order
  int ld_wht = 0;        // row stride of WhT in elements
  size_t off_loss = 0, off_lossout = 0, total = 0;
  int loss_slots = 0;
  StepCfg cfg{1, 1, 1};  // single-launch path
  bool small = false;    // one-launch small-batch path (step_small)
  bool mlp = false;      // residual MLP (per-layer weights, one-step dW windows)
  bool mlpv = false;     // MLP of layers of different widths (per-layer weights, states of different sizes)
  // wide-batch bf16 path (B >= 48): cell / layer kernels over up to 128 rows,
  // the adjoint's products as launches of their own (wide_bf16.hip)
  bool wide = false;
  size_t off_hbar = 0;   // fp32 [B][H]: hbar_{t+1} (cell) or ybar_{l+2} + zbar_{l+1} W_{l+1} (MLP)
  bool hsep = false;     // fp32 step kernels of large batches: the h-adjoint product may run as its own launch
  // resident whole-pass kernel (fp32 RNN / LSTM whose weights fit in registers)
  bool res = false;
  int r_mtiles = 0, r_ng = 0, r_nwg = 0, r_S = 0;
  size_t r_prog_cap = 0;  // program entries
  size_t off_prog = 0, off_ready = 0, off_consumed = 0, off_oflag = 0, off_status = 0, off_Z = 0, off_P = 0;
  size_t off_dWp = 0, off_dbp = 0;
};

// Device memory for ambptt_run_noalloc: the workspace of a pass, for callers
// that cannot allocate.  Every GPU that loads the library holds one copy until
// the process ends; all passes on a GPU share it.  Host code never uses the
// array's name as an address: ambptt_create looks up each device's copy with
// hipGetSymbolAddress (with that device current) and keeps it in g_scratch.
constexpr size_t kScratchBytes = size_t(64) << 20;
static __device__ __align__(256) char scratch[kScratchBytes];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
char* g_scratch[kMaxDevices] = {};

// Largest grid of the resident kernel the layout provisions for; the device's
// own limit is checked when a context is created.
constexpr int kResidentMaxWg = 1024;

ambptt_status validate(const ambptt_problem* p) {
  if (!p) return fail(AMBPTT_EINVAL, "problem is NULL");
  if (p->cell != AMBPTT_CELL_TANH_RNN && p->cell != AMBPTT_CELL_LSTM && p->cell != AMBPTT_CELL_RESMLP &&
      p->cell != AMBPTT_CELL_MLP)
    return fail(AMBPTT_EINVAL, "unknown cell");
  if (p->dtype != AMBPTT_F32 && p->dtype != AMBPTT_BF16) return fail(AMBPTT_EINVAL, "unknown dtype");
  if (p->loss < AMBPTT_LOSS_HALF_SQ_LAST || p->loss > AMBPTT_LOSS_MEAN_LAST) return fail(AMBPTT_EINVAL, "unknown loss");
  if (p->batch < 1 || p->hidden < 1 || p->input < 0) return fail(AMBPTT_EINVAL, "sizes must be positive");
  if (p->n_steps < 1) return fail(AMBPTT_EINVAL, "n_steps must be >= 1");
  if (p->fast_slots < 1) return fail(AMBPTT_EINVAL, "fast_slots must be >= 1");
  if (p->slow_slots < 0) return fail(AMBPTT_EINVAL, "slow_slots must be >= 0");
  if (p->interval_min < 0) return fail(AMBPTT_EINVAL, "interval_min must be >= 0");
  if (p->hidden % 16 || p->input % 16)
    return fail(AMBPTT_EUNSUPPORTED, "hidden and input sizes must be multiples of 16");
  if (p->dtype == AMBPTT_BF16 && (p->hidden % 32 || p->input % 32))
    return fail(AMBPTT_EUNSUPPORTED, "bf16 operands need hidden and input sizes that are multiples of 32");
  if (p->cell == AMBPTT_CELL_RESMLP && p->input != 0) return fail(AMBPTT_EINVAL, "the residual MLP has no step input");
  if (p->cell == AMBPTT_CELL_MLP && p->input != 0) return fail(AMBPTT_EINVAL, "the MLP has no step input");
  if (p->cell == AMBPTT_CELL_MLP && p->dtype != AMBPTT_F32)
    return fail(AMBPTT_EUNSUPPORTED, "the MLP of layers of different widths runs in fp32");
  if ((int64_t)p->batch * p->hidden > (int64_t(1) << 31)) return fail(AMBPTT_EUNSUPPORTED, "state too large");
  return AMBPTT_OK;
}

int auto_window(const ambptt_problem* p) {
  if (p->cell == AMBPTT_CELL_RESMLP) return 1;  // every layer has its own dW
  // every layer has its own dW; a window's layers go in one grouped launch,
  // which saves the host the cost of a stream handoff per layer
  if (p->cell == AMBPTT_CELL_MLP) return kMlpvDwGroup;
  // rows per window: each window reads and writes dW (fp32) once, so a window
  // must hold enough rows for its products to outweigh that; the bf16 path's
  // dW is large against its operands (4 bytes per weight against 2 bytes per
  // operand element), hence the longer windows.  On the large-batch fp32
  // path windows of 4096 rows (8 steps of the 4096-LSTM) ran 1.7 % faster
  // than windows of 1024, and windows of 8192 (a 1.3 GB ring) 0.3 % faster
  // again.
  const int rows = p->dtype == AMBPTT_BF16 || p->batch >= 256 ? 8192 : 1024;
  int w = (rows + p->batch - 1) / p->batch;
  return std::max(1, std::min(64, w));
}

Layout make_layout(const ambptt_problem* p, int window) {
  Layout L;
  L.G = p->cell == AMBPTT_CELL_LSTM ? 4 : 1;
  L.dsize = p->dtype == AMBPTT_BF16 ? 2 : 4;
  L.window = window > 0 ? window : auto_window(p);
  L.mlp = p->cell == AMBPTT_CELL_RESMLP;
  L.mlpv = p->cell == AMBPTT_CELL_MLP;
  const size_t BH = (size_t)p->batch * p->hidden;
  const size_t GH = (size_t)L.G * p->hidden;
  L.h_bytes = BH * L.dsize;
  L.c_bytes = p->cell == AMBPTT_CELL_LSTM ? BH * 4 : 0;
  L.state_bytes = align_up(L.h_bytes) + L.c_bytes;
  L.stride = align_up(L.state_bytes);
  L.cfg = pick_step_cfg(L.G, p->batch, p->input, p->hidden);
  dim3 grid, block;
  step_grid(L.cfg, p->batch, p->hidden, &grid, &block);
  L.loss_slots = int(grid.x * grid.y);
  // Problems with fewer than 1024 tiles of 16 rows x 16 units run the
  // small-batch kernels, which spread even a 64-row batch over all CUs.
  const long tiles = (long)((p->batch + 15) / 16) * (p->hidden / 16);
  L.small = tiles < 1024 || p->dtype == AMBPTT_BF16;
  if (L.small) {
    step_small_grid(L.G, p->batch, p->hidden, &grid, &block);
    L.loss_slots = int(grid.x * grid.y);
  }
  if (L.mlp) {
    L.small = false;
    resmlp_grid(p->batch, p->hidden, &grid, &block);
    L.loss_slots = int(grid.x * grid.y);
  }
  if (p->dtype == AMBPTT_BF16 && p->batch >= 48 &&
      (L.mlp ? mlp_wide_fits(p->batch, p->hidden) : cell_wide_fits(L.G, p->batch, p->input, p->hidden))) {
    L.wide = true;
    const int tiles = L.mlp ? mlp_wide_tiles(p->batch, p->hidden) : cell_wide_tiles(L.G, p->batch, p->hidden);
    L.loss_slots = std::max(L.loss_slots, 8 * ((tiles + 7) / 8));
  }
  if (!L.mlp && !L.mlpv && p->dtype == AMBPTT_F32) {
    const int U = resident_units(L.G);
    const int K1 = p->input + p->hidden;
    const int mtiles = (p->batch + 15) / 16, ng = p->hidden / U;
    const long nwg = (long)mtiles * ng;
    const double evr = double(revolve_advances(p->n_steps, p->fast_slots)) + 1.0;
    const double cap = 2.0 * (evr + 3.0 * double(p->n_steps)) + 256.0;
    const int S = p->hidden % U == 0 ? resident_octet(ng, p->hidden) : 0;
    if (K1 <= resident_max_k(L.G) && p->hidden <= resident_max_h(L.G) && p->hidden % U == 0 && S > 0 &&
        nwg <= kResidentMaxWg && cap < 8.0e6) {
      L.res = true;
      L.r_S = S;
      L.r_mtiles = mtiles;
      L.r_ng = ng;
      L.r_nwg = int(nwg);
      L.r_prog_cap = size_t(cap);
      L.loss_slots = std::max(L.loss_slots, L.r_nwg);
    }
  }
  if (!L.small && !L.mlp && !L.mlpv && p->dtype == AMBPTT_F32 &&
      cell_gemm_f32_fits(L.G, p->batch, p->input, p->hidden))
    L.loss_slots = std::max(L.loss_slots, cell_gemm_f32_tiles(L.G, p->batch, p->hidden));
  size_t o = 0;
  L.off_live[0] = o; o += L.stride;
  L.off_live[1] = o; o += L.stride;
  if (L.mlpv) {
    L.small = false;
    L.loss_slots = mlpv_tiles(p->batch, p->hidden);
  }
  // the large-batch fp32 kernels read WhT rows in 64-wide stages; rows padded
  // by 32 floats keep a power-of-two row length from mapping every row's
  // stage onto the same L2 sets
  const bool pad_wht = !L.small && !L.mlp && !L.mlpv && p->dtype == AMBPTT_F32;
  L.ld_wht = int(GH) + (pad_wht ? 32 : 0);
  L.off_wht = o; o += (L.mlp || L.mlpv) ? 0 : align_up((size_t)p->hidden * L.ld_wht * L.dsize);
  if (L.wide && !L.mlp) {
    L.off_wpk = o; o += align_up(GH * size_t(p->input + p->hidden) * 2);
    L.off_whpk = o; o += align_up(size_t(p->hidden) * GH * 2);
  }
  L.off_zbar = o; o += align_up(2 * (size_t)L.window * p->batch * GH * L.dsize);
  L.off_hwin = o; o += align_up(2 * (size_t)L.window * BH * L.dsize);
  L.off_cbar[0] = o; o += align_up(BH * 4);
  L.off_cbar[1] = o; o += align_up(BH * 4);
  L.off_loss = o; o += align_up((size_t)L.loss_slots * 8);
  L.off_lossout = o; o += kAlign;
  L.hsep = !L.small && !L.mlp && !L.mlpv && p->dtype == AMBPTT_F32;
  if (L.wide || L.hsep || L.mlpv) {  // the fp32 large-batch path may hold the product in split parts
    L.off_hbar = o; o += align_up(BH * 4 * (L.hsep ? kProdSplitMax : 1));
  }
  if (L.res) {
    const size_t U = size_t(resident_units(L.G)), K1 = size_t(p->input + p->hidden);
    const size_t mt = size_t(L.r_mtiles), ng = size_t(L.r_ng), nwg = size_t(L.r_nwg);
    L.off_prog = o; o += align_up(L.r_prog_cap * 16);
    L.off_ready = o; o += align_up(nwg * 4);
    L.off_consumed = o; o += align_up(nwg * 4);
    L.off_oflag = o; o += align_up(nwg * 4);
    L.off_status = o; o += kAlign;
    L.off_Z = o; o += align_up(2 * mt * ng * 16 * GH / ng * 4);
    L.off_P = o; o += align_up(2 * mt * (ng / size_t(L.r_S)) * size_t(p->hidden) * 16 * 4);
    L.off_dWp = o; o += align_up(mt * GH * K1 * 4);
    L.off_dbp = o; o += align_up(mt * GH * 4);
  }
  L.total = o;
  return L;
}

}  // namespace

struct ambptt_ctx {
  ambptt_problem p{};
  Layout L;
  int device = 0;
  hipStream_t cs = nullptr;  // compute (caller's)
  hipStream_t xs = nullptr;  // copy stream (owned)
  hipStream_t ds = nullptr;  // weight-gradient stream (owned)
  hipEvent_t ev_dw[2] = {nullptr, nullptr};  // last dW launch per ring half
  hipEvent_t ev_c2 = nullptr;
  std::vector<hipEvent_t> tpool;  // timing events, reused across runs
  char* pool = nullptr;
  char* ws = nullptr;
  // Pinned host tier: chunks of host_per_chunk slots of host_slot_bytes each
  // (one pinned allocation of tens of GiB fails well below the per-process
  // pinned limit, so a large tier comes in chunks); host is the first chunk,
  // the whole tier where a caller needs it contiguous.
  std::vector<std::pair<char*, size_t>> host_chunks;
  size_t host_slot_bytes = 0, host_per_chunk = 0;
  char* host = nullptr;
  bool no_alloc = false;  // inside ambptt_run_noalloc: any allocation is an error
  double* host_loss = nullptr;  // pinned scalar
  std::vector<hipEvent_t> ev_slot;
  std::vector<int> pend;  // 0 none, 1 store in flight, 2 prefetch in flight
  hipEvent_t ev_c = nullptr;
  int64_t interval_min = 0;
  int64_t timing_sample = 0;
  bool elide_prefetch = true;
  int window_opt = 0;
  int path_opt = 0;            // 0: resident kernel when it fits, 1: per-step launches, 2: resident kernel
  bool wide_opt = true;        // use the wide-batch bf16 kernels where the layout provides them
  int res_cap = -1;            // resident workgroups the device holds at once (-1: not queried)
  int64_t res_timeout_ms = 2000;
  bool res_test_stall = false;  // tests of the abort path: the first entry waits for a barrier that never comes
  bool res_coop = true;          // cooperative launch of the resident kernel (residency guaranteed)
  int dw_stream = -1;            // weight-gradient windows: 1 on their own stream, 0 on the compute stream, -1 by path
  // Executor events order work between the library's streams on one device
  // and time kernels; none of them publishes device memory to the host, so
  // by default they carry no system-scope fence (each such fence writes back
  // and invalidates the caches of every XCD, several microseconds between two
  // kernels).
  bool sys_fence = false;
  int store_policy = 0;  // 0: every I-th state; 1: the next state once the previous store has completed
  bool online = false;   // online checkpointing: placement decided without knowing n
  int interval_rule = 1;  // 0: smallest I with T_T <= I T_A; 1: I minimising the modelled time per step
  std::vector<double> step_costs;  // relative forward step costs (empty: equal)
  double plan_cost = 0.0;          // cost of the forward evaluations of the last plan built
  Plan cost_plan;                  // the plan for step_costs, kept while its inputs stay the same
  int64_t cost_plan_key[3] = {-1, -1, -1};  // interval_min, slow capacity, costs version
  double cost_plan_cost = 0.0;
  int64_t costs_version = 0;
  Plan sized_plan;                 // the plan of states of different sizes, kept likewise
  int64_t sized_plan_key[6] = {-1, -1, -1, -1, -1, -1};
  double sized_plan_cost = 0.0;
  int64_t widths_version = 0;
  bool hadj_launch = true;  // fp32 large-batch path: the adjoint's h-adjoint product as a launch of its own
  bool prod_split = true;   // ... on 128 x 128 tiles with the reduction split, when that fills the device
  int lds_gemm = 1;         // fp32 large-batch path: LDS-tiled kernels (0 off, 1 when they fill the device twice over, 2 always)
  // tests of the stream ordering: a host-side delay before every host-tier
  // copy and weight-gradient window on their streams, and NaN bytes written
  // into a fast slot before a prefetch refills it
  int64_t test_copy_delay_us = 0;
  bool test_poison = false;
  // the MLP of layers of different widths: w_0 .. w_n, the offsets of each
  // layer's weights and bias, and the state sizes in units of `unit` bytes
  std::vector<int32_t> widths;
  std::vector<size_t> woff, boff;
  std::vector<int64_t> zunits;
  size_t unit = 0;
  bool uniform_sizes = false;  // plan as if every state had the largest size (for comparison)
  int host_waits = -1;      // slot dependencies on host-tier copies: 1 waited for on the host, 0 stream waits, -1 by path
  hipEvent_t ev_end[8] = {};  // end events recorded by compute dispatches (host-tier copies and sweep pacing wait on them)
  Plan last_plan;        // the schedule the last ambptt_run executed
  FileTier* ftier = nullptr;        // a file below the pinned host tier (per-step path)
  std::vector<hipEvent_t> ev_file;  // per pinned buffer: its last device copy (system scope: the host reads the data)
  int32_t* prog_host = nullptr;  // pinned staging of the resident program
  size_t prog_host_cap = 0;
  unsigned* status_host = nullptr;  // pinned copy of the resident kernel's status words
  hipEvent_t ev_r[2] = {nullptr, nullptr};
};

namespace {

enum { kNone = 0, kStorePending = 1, kPrefetchPending = 2 };

// Slow slots the schedule may use: the pinned host tier's, or the file's below it.
int64_t slow_capacity(const ambptt_ctx* C) { return C->ftier ? C->ftier->capacity() : C->p.slow_slots; }

// The interval from measured timings (Section 3).  Rule 0, the paper's: the
// smallest I whose forward sweep hides one transfer, ceil(T_T / T_A), less a
// relative slack for transfers that lengthen a step only a little.  Rule 1:
// among I = 1 .. that I, the one with the least modelled time per step,
//   (max(I T_A, T_T) + F(I, s - 1) T_A) / I,
// a sweep interval being as slow as its store when the link is the bottleneck
// (the next store into the same fast slot must wait for it) and the reverse
// recomputing F(I, s - 1) steps of it; ties go to the smaller I.
int64_t interval_from_timings(double ta, double tt, int64_t s, int rule, double slack) {
  ta = std::max(ta, 1e-3);
  const int64_t strict = std::max<int64_t>(1, (int64_t)std::ceil(tt / ta - slack));
  if (rule == 0 || s < 2) return strict;
  int64_t best = 1;
  double best_c = 0.0;
  for (int64_t I = 1; I <= strict; ++I) {
    const double c = (std::max(double(I) * ta, tt) + double(revolve_advances(I, s - 1)) * ta) / double(I);
    if (I == 1 || c < best_c) best = I, best_c = c;
  }
  return best;
}

// The schedule a pass runs: the online one when the context asks for it.
std::vector<int64_t> plan_units(const ambptt_ctx* C);

Plan pass_plan(ambptt_ctx* C) {
  const ambptt_problem& p = C->p;
  const int64_t I = std::max<int64_t>(C->interval_min, 1);
  if (C->L.mlpv) {  // states of different sizes: the sized recursion in every reversal
    if (C->online) throw std::invalid_argument("online checkpointing is not available for states of different sizes");
    // built once per set of inputs: its tables take a visible time on the host
    const int64_t key[6] = {I, slow_capacity(C), C->costs_version, int64_t(C->step_costs.empty()),
                            C->widths_version, int64_t(C->uniform_sizes)};
    if (!std::equal(key, key + 6, C->sized_plan_key)) {
      C->sized_plan = make_plan_sized(p.n_steps, p.fast_slots, slow_capacity(C), I, plan_units(C),
                                      C->step_costs.empty() ? nullptr : &C->step_costs, &C->sized_plan_cost);
      std::copy(key, key + 6, C->sized_plan_key);
    }
    C->plan_cost = C->sized_plan_cost;
    return C->sized_plan;
  }
  if (C->online) return make_plan_online(p.n_steps, p.fast_slots, p.slow_slots, I);
  if (!C->step_costs.empty() && C->store_policy == 1 && C->path_opt != 2) {
    // stores decided during the sweep: the reverse is built from the chosen
    // starts, so the fixed intervals' cost splits are not needed; the uniform
    // plan, whose mode the cost splits keep, decides whether the host tier is
    // used (if not, plain Revolve with the cost splits runs)
    Plan u = make_plan(p.n_steps, p.fast_slots, slow_capacity(C), I);
    if (u.async) return u;
  }
  if (!C->step_costs.empty()) {  // the dynamic program runs once per set of inputs
    const int64_t key[3] = {I, slow_capacity(C), C->costs_version};
    if (!std::equal(key, key + 3, C->cost_plan_key)) {
      C->cost_plan = make_plan_costs(p.n_steps, p.fast_slots, key[1], I, C->step_costs, &C->cost_plan_cost);
      std::copy(key, key + 3, C->cost_plan_key);
    }
    C->plan_cost = C->cost_plan_cost;
    return C->cost_plan;
  }
  return make_plan(p.n_steps, p.fast_slots, slow_capacity(C), I);
}

// Widths of the MLP's layers: weight and bias offsets, state sizes in units
// of their greatest common divisor (every size is a multiple of 256 bytes).
void set_layer_widths(ambptt_ctx* C, const std::vector<int32_t>& w) {
  C->widths = w;
  C->widths_version++;
  const size_t n = w.size() - 1;
  C->woff.assign(n + 1, 0);
  C->boff.assign(n + 1, 0);
  for (size_t l = 0; l < n; ++l) {
    C->woff[l + 1] = C->woff[l] + size_t(w[l + 1]) * size_t(w[l]);
    C->boff[l + 1] = C->boff[l] + size_t(w[l + 1]);
  }
  std::vector<size_t> bytes(n + 1);
  size_t g = 0;
  for (size_t t = 0; t <= n; ++t) {
    bytes[t] = align_up(size_t(C->p.batch) * size_t(w[t]) * 4);
    g = std::gcd(g, bytes[t]);
  }
  C->unit = g;
  C->zunits.resize(n + 1);
  for (size_t t = 0; t <= n; ++t) C->zunits[t] = int64_t(bytes[t] / g);
}

// The state sizes the sized schedules plan with: the states' own, or the
// largest for every state (knob "uniform_sizes": slots of the largest size).
std::vector<int64_t> plan_units(const ambptt_ctx* C) {
  if (!C->uniform_sizes) return C->zunits;
  const int64_t m = *std::max_element(C->zunits.begin(), C->zunits.end());
  return std::vector<int64_t>(C->zunits.size(), m);
}

unsigned event_flags(const ambptt_ctx* C, bool timing) {
  return (timing ? 0u : unsigned(hipEventDisableTiming)) | (C->sys_fence ? 0u : unsigned(hipEventDisableSystemFence));
}

// (Re)creates the executor's synchronisation events with the context's fence
// scope; timing events are recreated on demand.
hipError_t make_sync_events(ambptt_ctx* C) {
  auto remake = [&](hipEvent_t& ev) {
    if (ev) (void)hipEventDestroy(ev);
    ev = nullptr;
    return hipEventCreateWithFlags(&ev, event_flags(C, false));
  };
  hipError_t e;
  if ((e = remake(C->ev_c)) != hipSuccess) return e;
  if ((e = remake(C->ev_c2)) != hipSuccess) return e;
  for (auto& ev : C->ev_dw)
    if ((e = remake(ev)) != hipSuccess) return e;
  for (auto& ev : C->ev_slot)
    if ((e = remake(ev)) != hipSuccess) return e;
  for (auto& ev : C->ev_end) {
    if (ev) (void)hipEventDestroy(ev);
    ev = nullptr;
    if ((e = hipEventCreateWithFlags(&ev, event_flags(C, true))) != hipSuccess) return e;
  }
  for (auto& ev : C->tpool) (void)hipEventDestroy(ev);
  C->tpool.clear();
  return hipSuccess;
}

constexpr size_t kHostChunkBytes = size_t(8) << 30;

void free_host(ambptt_ctx* C) {
  if (C->host_chunks.empty()) return;
  if (C->xs) (void)hipStreamSynchronize(C->xs);
  for (auto& c : C->host_chunks) (void)hipHostFree(c.first);
  C->host_chunks.clear();
  C->host = nullptr;
  C->host_slot_bytes = C->host_per_chunk = 0;
}

int64_t host_capacity(const ambptt_ctx* C) {
  if (!C->host_slot_bytes) return 0;
  int64_t n = 0;
  for (auto& c : C->host_chunks) n += int64_t(c.second / C->host_slot_bytes);
  return n;
}

// Pinned memory for `slots` host slots of slot_bytes: in one allocation when
// `contiguous` (the resident kernel's and the file ring's), else in chunks
// that host_slot() addresses.  Keeps what is there when it suffices.
ambptt_status ensure_host(ambptt_ctx* C, int64_t slots, size_t slot_bytes, bool contiguous) {
  const size_t need = size_t(slots) * slot_bytes;
  if (need == 0) return AMBPTT_OK;
  if (!C->host_chunks.empty() && C->host_chunks[0].second >= need) {
    if (!contiguous) {  // the first chunk holds the whole tier
      C->host_slot_bytes = slot_bytes;
      C->host_per_chunk = C->host_chunks[0].second / slot_bytes;
    }
    return AMBPTT_OK;
  }
  if (!contiguous && C->host_slot_bytes == slot_bytes && host_capacity(C) >= slots) return AMBPTT_OK;
  if (C->no_alloc)
    return fail(AMBPTT_EINVAL, "this pass needs " + std::to_string(need) +
                                   " bytes of pinned host tier that are not reserved (ambptt_set_int \"reserve\")");
  free_host(C);
  const size_t per = contiguous ? size_t(slots) : std::max<size_t>(1, kHostChunkBytes / slot_bytes);
  for (int64_t h = 0; h < slots; h += int64_t(per)) {
    const size_t bytes = std::min<size_t>(per, size_t(slots - h)) * slot_bytes;
    void* ptr = nullptr;
    if (hipHostMalloc(&ptr, bytes, hipHostMallocDefault) != hipSuccess || !ptr) {
      (void)hipGetLastError();
      free_host(C);
      return fail(AMBPTT_ENOMEM, "hipHostMalloc of " + std::to_string(bytes) + " bytes for the host tier failed (" +
                                     std::to_string(need) + " bytes in total)");
    }
    C->host_chunks.push_back({(char*)ptr, bytes});
  }
  C->host = C->host_chunks[0].first;
  C->host_slot_bytes = slot_bytes;
  C->host_per_chunk = per;
  return AMBPTT_OK;
}

char* host_slot(const ambptt_ctx* C, int64_t h) {
  return C->host_chunks[size_t(h) / C->host_per_chunk].first + (size_t(h) % C->host_per_chunk) * C->host_slot_bytes;
}

// Stream callback of the copy-delay test knob: holds its stream for a bounded time.
void delay_cb(void* us) { std::this_thread::sleep_for(std::chrono::microseconds((intptr_t)us)); }

// Sized plans may stack more snapshots than there are fast slots: slot ids
// up to `ids` get their synchronisation events.
ambptt_status grow_slot_events(ambptt_ctx* C, int64_t ids) {
  if (ids <= int64_t(C->pend.size())) return AMBPTT_OK;
  if (C->no_alloc) return fail(AMBPTT_EINVAL, "this pass needs slot events that are not reserved (ambptt_set_int \"reserve\")");
  const size_t k0 = C->ev_slot.size();
  C->ev_slot.resize(size_t(ids), nullptr);
  for (size_t k = k0; k < C->ev_slot.size(); ++k)
    HIPCK(hipEventCreateWithFlags(&C->ev_slot[k], event_flags(C, false)));
  C->pend.resize(size_t(ids), kNone);
  return AMBPTT_OK;
}

struct Sample {
  int cls;
  hipEvent_t a, b;
};

struct Exec {
  ambptt_ctx* C;
  const Layout& L;
  const ambptt_problem& p;
  const char* x;   // operand dtype, [n][B][D]
  const void* W;
  const float* b;
  void* WhT;
  void* Wpk = nullptr;   // wide bf16 cell: W in fragment order (the gate products)
  void* WhPk = nullptr;  // ... and W_h^T (the h-adjoint products)
  ambptt_stats st{};
  char* cur = nullptr;
  int cur_slot = -1;  // slot index the live state aliases, or -1
  int cur_live = -1;  // live buffer index, or -1
  std::vector<int64_t> slot_t;
  int64_t calls[6] = {0, 0, 0, 0, 0, 0};
  std::vector<Sample> samples;
  bool live_dead = false;  // the live state was consumed by an adjoint step
  // Host-tier copies must follow the compute work before them.  When a store
  // or prefetch comes next in the action list, the compute launches carry an
  // end event of their own (recorded by the dispatch), which the copy stream
  // then waits for: no marker packet is put between two kernels.
  bool want_tail = false;        // the next compute launches carry an end event for a copy after them
  bool want_end = false;         // ... or for the host's pacing of the sweep
  bool tail_ok = false;          // tail_ev marks the end of the latest compute-stream work
  hipEvent_t tail_ev = nullptr;
  hipEvent_t last_end = nullptr;  // end event of the latest compute launch that carried one
  unsigned end_cur = 0;           // next event of the ring (8 deep: reused 8 launches later)
  bool wide = false;       // wide-batch bf16 kernels
  bool sep32 = false;      // fp32 step kernels with the h-adjoint product as a launch of its own
  bool lds_cell = false;   // ... whose gate products run on the LDS-tiled kernel
  bool lds_prod = false;   // ... whose h-adjoint products run on the LDS-tiled kernel
  float* hbuf = nullptr;   // the adjoint's product (fp32 [B][H]) on those two paths
  int hparts = 1;          // split parts of the fp32 LDS-tiled product (summed by the adjoint)

  Exec(ambptt_ctx* c, const void* x_, const void* W_, const float* b_)
      : C(c), L(c->L), p(c->p), x((const char*)x_), W(W_), b(b_), slot_t(c->pend.size(), -1) {
    slot_off.resize(C->pend.size());
    for (size_t k = 0; k < slot_off.size(); ++k) slot_off[k] = k * L.stride;
    WhT = C->ws + L.off_wht;
    wide = L.wide && C->wide_opt;
    sep32 = L.hsep && C->hadj_launch;
    if (L.hsep) {
      const int G = L.G, B = p.batch, D = p.input, H = p.hidden;
      // by default only shapes that give every CU its two workgroups
      lds_cell = C->lds_gemm > 0 && cell_gemm_f32_fits(G, B, D, H) &&
                 (C->lds_gemm == 2 || cell_gemm_f32_tiles(G, B, H) >= 256);
      lds_prod = sep32 && C->lds_gemm > 0 && prod_gemm_f32_fits(B, H, G * H) &&
                 (C->lds_gemm == 2 || prod_gemm_f32_tiles(B, H) >= 256);
      // the split parts are summed by the LDS-tiled adjoint only
      if (lds_prod && lds_cell && C->prod_split) hparts = prod_split_f32_parts(B, H, G * H);
    }
    if (wide || sep32 || L.mlpv) hbuf = (float*)(C->ws + L.off_hbar);
    if (wide && !L.mlp) {
      Wpk = C->ws + L.off_wpk;
      WhPk = C->ws + L.off_whpk;
    }
  }
  const void* x_at(int64_t t) const { return x + (size_t)t * p.batch * p.input * L.dsize; }

  // byte offset of every fast slot: k * stride, or in sized plans the stacked
  // offset the plan's action names (set when the slot is written)
  std::vector<size_t> slot_off;
  char* slot(int64_t k) const { return C->pool + slot_off[size_t(k)]; }
  // bytes of state x_t (the MLP's states differ in size)
  size_t bytes_of(int64_t t) const {
    return L.mlpv ? align_up(size_t(p.batch) * size_t(C->widths[size_t(t)]) * 4) : L.state_bytes;
  }
  ambptt_status grow_slots(int64_t ids) {
    const ambptt_status s = grow_slot_events(C, ids);
    if (s != AMBPTT_OK) return s;
    for (size_t k = slot_off.size(); k < C->pend.size(); ++k) slot_off.push_back(k * L.stride);
    slot_t.resize(C->pend.size(), -1);
    return AMBPTT_OK;
  }
  // a sized plan's action places slot k at A.off units; a write moves the
  // slot there, a read must find it there; the state must lie in the pool
  ambptt_status place(const Action& A, int64_t k, int64_t t, bool write) {
    if (A.off < 0) return AMBPTT_OK;
    const size_t o = size_t(A.off) * C->unit;
    if (o + bytes_of(t) > size_t(p.fast_slots) * L.stride)
      return fail(AMBPTT_EINTERNAL, "sized plan: a state past the end of the slot pool");
    if (write) slot_off[size_t(k)] = o;
    else if (slot_off[size_t(k)] != o) return fail(AMBPTT_EINTERNAL, "sized plan: a slot read away from where it was written");
    return AMBPTT_OK;
  }
  char* live(int i) const { return C->ws + L.off_live[i]; }
  void* hpart(char* s) const { return s; }
  float* cpart(char* s) const { return (float*)(s + align_up(L.h_bytes)); }

  // Compute reads a prefetched slot, or overwrites a slot being stored, only
  // after that copy.  A copy still in flight when the host gets here costs a
  // wait: a stream wait on the compute stream, whose barrier packet costs
  // several microseconds between two kernels even when the copy has long
  // finished, or, on the paths whose kernels each take tens of microseconds
  // or more, a wait on the host: the copy was issued an interval or more
  // before, so the device still has that much work queued while the host
  // waits.
  ambptt_status wait_slot(int64_t k, bool for_write) {
    int& pd = C->pend[size_t(k)];
    if (pd == kPrefetchPending || (for_write && pd == kStorePending)) {
      const hipError_t q = hipEventQuery(C->ev_slot[size_t(k)]);
      if (q == hipErrorNotReady) {
        if (C->host_waits < 0 ? (wide || L.hsep) : C->host_waits != 0) HIPCK(hipEventSynchronize(C->ev_slot[size_t(k)]));
        else HIPCK(hipStreamWaitEvent(C->cs, C->ev_slot[size_t(k)], 0));
        st.compute_waits++;
      } else if (q != hipSuccess) {
        HIPCK(q);
      }
      pd = kNone;
    }
    return AMBPTT_OK;
  }

  // Runs one launch.  Every timing_sample-th launch of a class carries a pair
  // of events that the dispatch itself records at the kernel's start and end
  // (hipExtLaunchKernel): no marker packet joins the stream, and the interval
  // is the kernel's execution time.
  template <class F>
  ambptt_status timed(int cls, F launch, hipStream_t strm = nullptr) {
    const bool compute = strm == nullptr || strm == C->cs;
    const bool sample = C->timing_sample > 0 && (calls[cls] % C->timing_sample) == 0 && samples.size() < 4096 &&
                        (!C->no_alloc || C->tpool.size() >= 2 * (samples.size() + 1));
    Sample smp{cls, nullptr, nullptr};
    if (sample) {
      const size_t need = 2 * (samples.size() + 1);
      while (C->tpool.size() < need) {
        hipEvent_t e;
        HIPCK(hipEventCreateWithFlags(&e, event_flags(C, true)));
        C->tpool.push_back(e);
      }
      smp.a = C->tpool[need - 2];
      smp.b = C->tpool[need - 1];
    }
    hipEvent_t end = smp.b;
    if (compute && (want_tail || want_end) && !end) end = C->ev_end[end_cur++ & 7];
    HIPCK(launch(smp.a, end));
    if (compute) {
      tail_ok = want_tail;
      tail_ev = end;
      last_end = end;
    }
    if (sample) samples.push_back(smp);
    calls[cls]++;
    st.kernel_launches++;
    return AMBPTT_OK;
  }

  StepArgs base_args() const {
    StepArgs a{};
    a.B = p.batch;
    a.D = p.input;
    a.H = p.hidden;
    a.W = W;
    a.bias = b;
    a.WhT = WhT;
    a.ld_wht = L.ld_wht;
    a.loss = p.loss;
    a.inv_bh = 1.0f / float((double)p.batch * p.hidden);
    return a;
  }

  // the fp32 h-adjoint product out = zbar W_h
  hipError_t prod32(const ProdArgs& pa, hipEvent_t e0, hipEvent_t e1) const {
    return lds_prod ? launch_prod_gemm_f32(pa, C->cs, e0, e1) : launch_prod_f32(pa, C->cs, e0, e1);
  }

  hipError_t launch(int mode, const StepArgs& a, hipEvent_t e0, hipEvent_t e1) const {
    if (wide && mode != kFinal) {
      StepArgs w = a;
      w.W = Wpk;
      return launch_cell_wide(L.G, mode, w, C->cs, e0, e1);
    }
    if (lds_cell && (mode == kForward || (mode == kAdjoint && (a.first || a.hbar_in))))
      return launch_cell_gemm_f32(L.G, mode, a, C->cs, e0, e1);
    return L.small ? launch_step_small(L.G, p.dtype == AMBPTT_BF16, mode, a, C->cs, e0, e1)
                   : launch_step(L.G, mode, L.cfg, a, C->cs, e0, e1);
  }

  // one forward step: state at `src` -> `dst`
  // residual MLP: layer t's weights and bias
  const void* W_of(int64_t t) const {
    return (const char*)W + (size_t)t * p.hidden * p.hidden * L.dsize;
  }
  MlpArgs mlp_args(int64_t t) const {
    MlpArgs a{};
    a.W = W_of(t);
    a.bias = b + (size_t)t * p.hidden;
    a.B = p.batch;
    a.w = p.hidden;
    a.loss = p.loss;
    a.inv_bw = 1.0f / float((double)p.batch * p.hidden);
    return a;
  }

  // layer t of the MLP of different widths: M = B rows, N = w_{t+1}, K = w_t
  MlpvArgs mlpv_args(int64_t t) const {
    MlpvArgs a{};
    a.W = (const float*)W + C->woff[size_t(t)];
    a.bias = b + C->boff[size_t(t)];
    a.M = p.batch;
    a.N = C->widths[size_t(t) + 1];
    a.K = C->widths[size_t(t)];
    a.loss = p.loss;
    a.last = t == p.n_steps - 1;
    a.inv = 1.0f / float(double(p.batch) * double(a.N));
    return a;
  }

  ambptt_status fwd_step(int64_t t, char* src, char* dst) {
    st.forward_evals++;
    if (L.mlpv) {
      MlpvArgs a = mlpv_args(t);
      a.A = (const float*)src;
      a.out = (float*)dst;
      return timed(AMBPTT_K_FWD, [&](hipEvent_t e0, hipEvent_t e1) { return launch_mlpv(kForward, a, C->cs, e0, e1); });
    }
    if (L.mlp) {
      MlpArgs a = mlp_args(t);
      a.y = src;
      a.y_out = dst;
      return timed(AMBPTT_K_FWD, [&](hipEvent_t e0, hipEvent_t e1) {
        return wide ? launch_mlp_wide(kForward, a, C->cs, e0, e1)
                    : launch_resmlp(p.dtype == AMBPTT_BF16, kForward, a, C->cs, e0, e1);
      });
    }
    StepArgs a = base_args();
    a.x = x_at(t);
    a.h = hpart(src);
    a.c = L.G == 4 ? cpart(src) : nullptr;
    a.h_out = hpart(dst);
    a.c_out = L.G == 4 ? cpart(dst) : nullptr;
    return timed(AMBPTT_K_FWD, [&](hipEvent_t e0, hipEvent_t e1) { return launch(kForward, a, e0, e1); });
  }

  int64_t ring(int64_t t) const { return t % (2 * (int64_t)L.window); }
  void* zbar_at(int64_t t) const {
    return C->ws + L.off_zbar + (size_t)ring(t) * p.batch * L.G * p.hidden * L.dsize;
  }
  void* hwin_at(int64_t t) const { return C->ws + L.off_hwin + (size_t)ring(t) * p.batch * p.hidden * L.dsize; }
  float* cbar(int64_t t) const { return (float*)(C->ws + L.off_cbar[t & 1]); }

  // ring half of the z-bar / h window that step t writes
  int half_of(int64_t t) const { return int((t / L.window) & 1); }
  bool dw_pending[2] = {false, false};

  ambptt_status adjoint(int64_t t, float* dW, float* db) {
    const int64_t n = p.n_steps;
    const bool first = (t == n - 1);
    if (first) st.forward_evals++;  // the first turn's forward step
    st.adjoints++;
    const int64_t w = L.window;
    // the window half this step writes was last read by the dW launch two
    // windows later in t; wait for it if it is still running
    const int hf = half_of(t);
    if (dw_pending[hf]) {
      const hipError_t q = hipEventQuery(C->ev_dw[hf]);
      if (q == hipErrorNotReady) {
        HIPCK(hipStreamWaitEvent(C->cs, C->ev_dw[hf], 0));
        st.compute_waits++;
      } else if (q != hipSuccess) {
        HIPCK(q);
      }
      dw_pending[hf] = false;
    }
    ambptt_status s;
    if (L.mlpv) {
      MlpvArgs a = mlpv_args(t);
      a.A = (const float*)cur;
      a.zbar_out = (float*)zbar_at(t);
      a.ywin_out = (float*)hwin_at(t);  // y_t beside zbar_t for the layer's weight gradient
      a.loss_acc = (double*)(C->ws + L.off_loss);
      if (!first) {  // u = zbar_{t+1} W_{t+1} in the same launch: N = w_{t+1}, K2 = w_{t+2}
        a.A2 = (const float*)zbar_at(t + 1);
        a.W2 = (const float*)W + C->woff[size_t(t) + 1];
        a.K2 = C->widths[size_t(t) + 2];
      }
      s = timed(AMBPTT_K_ADJ, [&](hipEvent_t e0, hipEvent_t e1) { return launch_mlpv(kAdjoint, a, C->cs, e0, e1); });
      if (s != AMBPTT_OK) return s;
    } else if (L.mlp) {
      MlpArgs a = mlp_args(t);
      a.y = cur;
      a.first = first;
      a.Wn = first ? nullptr : W_of(t + 1);
      a.zbar_in = first ? nullptr : zbar_at(t + 1);
      a.ybar_in = first ? nullptr : cbar(t + 1);
      a.zbar_out = zbar_at(t);
      a.ybar_out = cbar(t);
      a.ywin_out = hwin_at(t);
      a.loss_acc = (double*)(C->ws + L.off_loss);
      if (wide) {
        if (!first) {  // ybar_{l+2} + zbar_{l+1} W_{l+1}
          ProdArgs pa{a.zbar_in, a.Wn, a.ybar_in, hbuf, p.batch, p.hidden, p.hidden};
          s = timed(AMBPTT_K_HADJ, [&](hipEvent_t e0, hipEvent_t e1) { return launch_prod_nn(pa, C->cs, e0, e1); });
          if (s != AMBPTT_OK) return s;
          a.nn_in = hbuf;
        }
        s = timed(AMBPTT_K_ADJ, [&](hipEvent_t e0, hipEvent_t e1) { return launch_mlp_wide(kAdjoint, a, C->cs, e0, e1); });
      } else {
        s = timed(AMBPTT_K_ADJ, [&](hipEvent_t e0, hipEvent_t e1) {
          return launch_resmlp(p.dtype == AMBPTT_BF16, kAdjoint, a, C->cs, e0, e1);
        });
      }
    } else {
      StepArgs a = base_args();
      a.x = x_at(t);
      a.h = hpart(cur);
      a.c = L.G == 4 ? cpart(cur) : nullptr;
      a.first = first;
      a.last = first;
      a.zbar_in = first ? nullptr : zbar_at(t + 1);
      a.cbar_in = first ? nullptr : cbar(t + 1);
      a.zbar_out = zbar_at(t);
      a.cbar_out = cbar(t);
      a.hwin_out = hwin_at(t);
      a.loss_acc = (double*)(C->ws + L.off_loss);
      if ((wide || sep32) && !first) {  // hbar_{t+1} = zbar_{t+1} W_h
        ProdArgs pa{a.zbar_in, wide ? WhPk : WhT, nullptr, hbuf, p.batch, p.hidden, L.G * p.hidden, L.ld_wht};
        s = timed(AMBPTT_K_HADJ, [&](hipEvent_t e0, hipEvent_t e1) {
          if (hparts > 1) return launch_prod_split_f32(pa, hparts, C->cs, e0, e1);
          return wide ? launch_prod_nt(pa, C->cs, e0, e1) : prod32(pa, e0, e1);
        });
        if (s != AMBPTT_OK) return s;
        a.hbar_in = hbuf;
        a.hbar_parts = hparts;
      }
      s = timed(AMBPTT_K_ADJ, [&](hipEvent_t e0, hipEvent_t e1) { return launch(kAdjoint, a, e0, e1); });
    }
    if (s != AMBPTT_OK) return s;
    live_dead = true;
    if (t % w == 0) {  // window [t, min(t + w, n)) complete: its weight gradient, here or on the dW stream
      const int64_t cnt = std::min(w, n - t);
      DwArgs d{};
      d.zbar = zbar_at(t);
      d.x = p.input > 0 ? x_at(t) : nullptr;
      d.hwin = hwin_at(t);
      d.dW = dW;
      d.db = db;
      d.R = int(cnt * p.batch);
      d.D = p.input;
      d.H = p.hidden;
      d.GH = L.G * p.hidden;
      d.accumulate = 1;
      if (L.mlp) {  // layer t's own gradient, written once
        d.dW = dW + (size_t)t * p.hidden * p.hidden;
        d.db = db + (size_t)t * p.hidden;
        d.accumulate = 0;
      }
      DwArgs grp[kMlpvDwGroup];
      if (L.mlpv) {  // each layer's own gradient [w_{t+i+1}][w_{t+i}], written once
        for (int64_t i = 0; i < cnt; ++i) {
          DwArgs& g = grp[i];
          g = DwArgs{};
          g.zbar = zbar_at(t + i);
          g.hwin = hwin_at(t + i);
          g.dW = dW + C->woff[size_t(t + i)];
          g.db = db + C->boff[size_t(t + i)];
          g.R = p.batch;
          g.H = C->widths[size_t(t + i)];
          g.GH = C->widths[size_t(t + i) + 1];
          g.accumulate = 0;
        }
      }
      // the wide-batch bf16 kernels and the large-batch fp32 kernels each fill
      // the device: beside them a window only competes for the same units, so
      // it runs in line on the compute stream; so does the grouped window of
      // the MLP of different widths (measured at the same rate either way,
      // without a stream handoff per window)
      const bool own = C->dw_stream < 0 ? !(wide || L.hsep || L.mlpv) : C->dw_stream != 0;
      hipStream_t ws = own ? C->ds : C->cs;
      if (own) {
        HIPCK(hipEventRecord(C->ev_c2, C->cs));
        HIPCK(hipStreamWaitEvent(C->ds, C->ev_c2, 0));
        if ((s = test_delay(C->ds)) != AMBPTT_OK) return s;
      }
      s = timed(
          AMBPTT_K_DW,
          [&](hipEvent_t e0, hipEvent_t e1) {
            return L.mlpv ? launch_mlpv_dw(grp, int(cnt), ws, e0, e1)
                          : p.dtype == AMBPTT_BF16 ? launch_dw_bf16(d, ws, e0, e1) : launch_dw(d, ws, e0, e1);
          },
          ws);
      if (s != AMBPTT_OK) return s;
      if (own) {  // the ring half stays taken until this event (in line, stream order keeps it)
        HIPCK(hipEventRecord(C->ev_dw[hf], ws));
        dw_pending[hf] = true;
      }
    }
    return AMBPTT_OK;
  }

  // dL/dx_0 = (zbar_0 W_h, cbar_0)
  ambptt_status final_step(float* dh0, float* dc0) {
    if (L.mlpv) {  // dL/dy_0 = zbar_0 W_0: N = w_0, K = w_1
      MlpvArgs u = mlpv_args(0);
      u.A = (const float*)zbar_at(0);
      u.out = dh0;
      u.N = C->widths[0];
      u.K = C->widths[1];
      return timed(AMBPTT_K_OTHER, [&](hipEvent_t e0, hipEvent_t e1) { return launch_mlpv(kFinal, u, C->cs, e0, e1); });
    }
    if (L.mlp) {
      MlpArgs a = mlp_args(0);
      a.Wn = W_of(0);
      a.zbar_in = zbar_at(0);
      a.ybar_in = cbar(0);
      a.dy0 = dh0;
      if (wide) {  // dL/dy_0 = ybar_1 + zbar_0 W_0
        ProdArgs pa{a.zbar_in, a.Wn, a.ybar_in, dh0, p.batch, p.hidden, p.hidden};
        return timed(AMBPTT_K_OTHER, [&](hipEvent_t e0, hipEvent_t e1) { return launch_prod_nn(pa, C->cs, e0, e1); });
      }
      return timed(AMBPTT_K_OTHER, [&](hipEvent_t e0, hipEvent_t e1) {
        return launch_resmlp(p.dtype == AMBPTT_BF16, kFinal, a, C->cs, e0, e1);
      });
    }
    StepArgs a = base_args();
    a.zbar_in = zbar_at(0);
    a.cbar_in = cbar(0);
    a.dh0 = dh0;
    a.dc0 = dc0;
    if (wide || sep32) {  // dL/dh_0 = zbar_0 W_h, dL/dc_0 = cbar_0
      ProdArgs pa{a.zbar_in, wide ? WhPk : WhT, nullptr, dh0, p.batch, p.hidden, L.G * p.hidden, L.ld_wht};
      ambptt_status s = timed(AMBPTT_K_OTHER, [&](hipEvent_t e0, hipEvent_t e1) {
        return wide ? launch_prod_nt(pa, C->cs, e0, e1) : prod32(pa, e0, e1);
      });
      if (s != AMBPTT_OK) return s;
      if (L.G == 4) HIPCK(hipMemcpyAsync(dc0, a.cbar_in, (size_t)p.batch * p.hidden * 4, hipMemcpyDeviceToDevice, C->cs));
      return AMBPTT_OK;
    }
    return timed(AMBPTT_K_OTHER, [&](hipEvent_t e0, hipEvent_t e1) { return launch(kFinal, a, e0, e1); });
  }

  // the copy-delay test knob: the next work on stream `strm` starts late
  ambptt_status test_delay(hipStream_t strm) {
    if (C->test_copy_delay_us > 0) HIPCK(hipLaunchHostFunc(strm, delay_cb, (void*)(intptr_t)C->test_copy_delay_us));
    return AMBPTT_OK;
  }

  ambptt_status copy_state(char* dst, char* src, size_t bytes) {
    HIPCK(hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToDevice, C->cs));
    tail_ok = false;
    return AMBPTT_OK;
  }
  // the copy stream waits for all compute work enqueued so far
  ambptt_status copy_after_compute() {
    hipEvent_t dep = tail_ok ? tail_ev : C->ev_c;
    if (!tail_ok) HIPCK(hipEventRecord(C->ev_c, C->cs));
    HIPCK(hipStreamWaitEvent(C->xs, dep, 0));
    return AMBPTT_OK;
  }
  static bool copy_follows(const std::vector<Action>& acts, size_t j) {
    if (j >= acts.size()) return false;
    if (acts[j].op == Op::Store || acts[j].op == Op::Prefetch) return true;
    return acts[j].op == Op::Snap && j + 1 < acts.size() && acts[j + 1].op == Op::Store;
  }

  char* other_live() {
    const int i = (cur_live == 0) ? 1 : 0;
    return live(i);
  }
  void set_cur_live(char* ptr) {
    cur = ptr;
    cur_slot = -1;
    cur_live = (ptr == live(0)) ? 0 : 1;
  }
  void set_cur_slot(int64_t k) {
    cur = slot(k);
    cur_slot = int(k);
    cur_live = -1;
  }

  ambptt_status run(const Plan& plan, float* dW, float* db) { return run_acts(plan.acts, 0, dW, db); }

  // The two-level policy with the interval starts decided during the sweep
  // (the non-uniform policy of Section 6): the output of forward step t
  // becomes the next interval start when the store of the previous start has
  // completed by the time step t is issued, and at least `spacing` steps have
  // passed since that start (ceil(n / (H + 1)), so that H host slots span the
  // sequence).  The host stays at most kAhead steps ahead of the device, so
  // that "completed" reflects the device's progress.  A start after which at
  // most as many steps remain as have passed since the previous start is the
  // last one (kept in HBM only), so the sweep ends within one interval of n;
  // so is the start that takes the last host slot's successor.  Needs n >= 2,
  // s >= 2, H >= 1.  Returns the starts; the reverse is built from them.
  ambptt_status dynamic_sweep(std::vector<int64_t>& starts, float* dW, float* db) {
    constexpr int kAhead = 3;
    const int64_t n = p.n_steps, H = slow_capacity(C);
    const int64_t spacing = std::max<int64_t>(1, (n + H) / (H + 1));
    ambptt_status s;
    starts.assign(1, 0);
    const std::vector<Action> head = {{Op::Snap, 0, 0, 0}, {Op::Store, 0, 0, 0}};
    if ((s = run_acts(head, 0, dW, db)) != AMBPTT_OK) return s;
    hipEvent_t pace[kAhead] = {};  // end events of the last kAhead steps (recorded by their dispatches)
    want_end = true;
    for (int64_t t = 0;; ++t) {
      const int64_t k = int64_t(starts.size()) - 1, tk = starts.back(), t1 = t + 1;
      if (t >= kAhead) HIPCK(hipEventSynchronize(pace[t % kAhead]));
      const hipError_t q = hipEventQuery(C->ev_slot[size_t(k % 2)]);
      if (q != hipSuccess && q != hipErrorNotReady) HIPCK(q);
      const bool near_end = n - t1 <= t1 - tk;  // t1 <= n - 1 holds: n - t1 >= 1 until then
      const bool start = near_end || (q == hipSuccess && t1 - tk >= spacing);
      const bool last = start && (near_end || k + 1 >= H);
      if (start) {  // x_{t1} is start k + 1: step t writes it into its fast slot
        const int64_t ks = (k + 1) % 2;
        if ((s = wait_slot(ks, true)) != AMBPTT_OK) return s;
        want_tail = !last;  // its store follows
        if ((s = fwd_step(t, cur, slot(ks))) != AMBPTT_OK) return s;
        set_cur_slot(ks);
        starts.push_back(t1);
        if (last) {
          want_end = false;
          return AMBPTT_OK;  // the reverse begins by snapshotting it (already there)
        }
        pace[t % kAhead] = last_end;
        const std::vector<Action> sw = {{Op::Snap, ks, t1, 0}, {Op::Store, ks, k + 1, t1}};
        if ((s = run_acts(sw, 0, dW, db)) != AMBPTT_OK) return s;
      } else {
        char* dst = other_live();
        want_tail = false;
        if ((s = fwd_step(t, cur, dst)) != AMBPTT_OK) return s;
        set_cur_live(dst);
        pace[t % kAhead] = last_end;
      }
    }
  }

  ambptt_status run_acts(const std::vector<Action>& acts, size_t from, float* dW, float* db) {
    ambptt_status s;
    for (size_t i = from; i < acts.size(); ++i) {
      const Action& A = acts[i];
      want_tail = copy_follows(acts, i + 1);
      switch (A.op) {
        case Op::Advance: {
          int64_t fuse_k = -1;
          if (i + 1 < acts.size() && acts[i + 1].op == Op::Snap && acts[i + 1].b == A.b &&
              acts[i + 1].a != cur_slot)
            fuse_k = acts[i + 1].a;
          for (int64_t t = A.a; t < A.b; ++t) {
            const bool last = (t + 1 == A.b);
            if (last && fuse_k >= 0) {
              if ((s = wait_slot(fuse_k, true)) != AMBPTT_OK) return s;
              if ((s = place(acts[i + 1], fuse_k, A.b, true)) != AMBPTT_OK) return s;
              if ((s = fwd_step(t, cur, slot(fuse_k))) != AMBPTT_OK) return s;
              set_cur_slot(fuse_k);
            } else {
              char* dst = other_live();
              if ((s = fwd_step(t, cur, dst)) != AMBPTT_OK) return s;
              set_cur_live(dst);
            }
          }
          if (fuse_k >= 0) {
            slot_t[size_t(fuse_k)] = A.b;
            st.takeshots++;
            ++i;
          }
          live_dead = false;
          break;
        }
        case Op::Snap: {
          st.takeshots++;
          if (cur_slot == A.a) {  // already there
            if ((s = place(A, A.a, A.b, false)) != AMBPTT_OK) return s;
            slot_t[size_t(A.a)] = A.b;
            break;
          }
          if ((s = wait_slot(A.a, true)) != AMBPTT_OK) return s;
          if ((s = place(A, A.a, A.b, true)) != AMBPTT_OK) return s;
          if ((s = copy_state(slot(A.a), cur, bytes_of(A.b))) != AMBPTT_OK) return s;
          st.takeshot_copies++;
          slot_t[size_t(A.a)] = A.b;
          break;
        }
        case Op::Restore: {
          st.restores++;
          if ((s = place(A, A.a, A.b, false)) != AMBPTT_OK) return s;
          if ((s = wait_slot(A.a, false)) != AMBPTT_OK) return s;
          set_cur_slot(A.a);
          live_dead = false;
          break;
        }
        case Op::First:
        case Op::Youturn:
          if ((s = adjoint(A.a, dW, db)) != AMBPTT_OK) return s;
          break;
        case Op::Store: {
          const int64_t k = A.a, h = A.b;
          char* dst = host_slot(C, h);
          if (C->ftier && !(dst = C->ftier->store_buffer(h))) return fail(AMBPTT_EINTERNAL, C->ftier->error());
          if ((s = place(A, k, A.c, false)) != AMBPTT_OK) return s;
          if ((s = copy_after_compute()) != AMBPTT_OK) return s;
          if ((s = test_delay(C->xs)) != AMBPTT_OK) return s;
          HIPCK(hipMemcpyAsync(dst, slot(k), bytes_of(A.c), hipMemcpyDeviceToHost, C->xs));
          HIPCK(hipEventRecord(C->ev_slot[size_t(k)], C->xs));
          if (C->ftier) {  // written behind to the file once the copy has landed
            hipEvent_t ev = C->ev_file[size_t(h % int64_t(C->ev_file.size()))];
            HIPCK(hipEventRecord(ev, C->xs));
            C->ftier->stored(h, [ev] { return hipEventSynchronize(ev) == hipSuccess; });
          }
          if (C->pend[size_t(k)] != kPrefetchPending) C->pend[size_t(k)] = kStorePending;
          st.stores++;
          st.bytes_d2h += (int64_t)bytes_of(A.c);
          break;
        }
        case Op::Prefetch: {
          const int64_t h = A.a, k = A.b, t = A.c;
          st.prefetches++;
          if ((s = place(A, k, t, true)) != AMBPTT_OK) return s;
          if (C->elide_prefetch && slot_t[size_t(k)] == t) {
            st.prefetches_elided++;
            if (C->ftier) C->ftier->prefetched(h, [] { return true; });  // nothing copied out of the buffer
            break;
          }
          if (cur_slot == k && !live_dead) {  // the live state aliases the target: keep it
            char* dst = live(0);
            if ((s = copy_state(dst, cur, bytes_of(slot_t[size_t(k)]))) != AMBPTT_OK) return s;
            set_cur_live(dst);
          }
          const char* src = host_slot(C, h);
          if (C->ftier && !(src = C->ftier->prefetch_buffer(h))) return fail(AMBPTT_EINTERNAL, C->ftier->error());
          if ((s = copy_after_compute()) != AMBPTT_OK) return s;
          // the poison test knob: until the prefetch lands the slot holds NaNs,
          // so compute reading it too early shows in the gradients
          if (C->test_poison) HIPCK(hipMemsetAsync(slot(k), 0xFF, L.state_bytes, C->xs));
          if ((s = test_delay(C->xs)) != AMBPTT_OK) return s;
          HIPCK(hipMemcpyAsync(slot(k), src, bytes_of(t), hipMemcpyHostToDevice, C->xs));
          HIPCK(hipEventRecord(C->ev_slot[size_t(k)], C->xs));
          if (C->ftier) {  // the buffer takes the slot h - R from the file once this copy is done
            hipEvent_t ev = C->ev_file[size_t(h % int64_t(C->ev_file.size()))];
            HIPCK(hipEventRecord(ev, C->xs));
            C->ftier->prefetched(h, [ev] { return hipEventSynchronize(ev) == hipSuccess; });
          }
          C->pend[size_t(k)] = kPrefetchPending;
          slot_t[size_t(k)] = t;
          st.bytes_h2d += (int64_t)bytes_of(t);
          break;
        }
      }
    }
    return AMBPTT_OK;
  }
};

ambptt_status prepare_inputs(ambptt_ctx* C, const void* W, const void* h0, const float* c0, Exec& E) {
  const Layout& L = C->L;
  const ambptt_problem& p = C->p;
  if (L.mlp || L.mlpv) {
    // no transposed weights: the residual MLP kernels transpose W tiles in LDS
  } else if (p.dtype == AMBPTT_BF16) {
    HIPCK(launch_transpose_wh_bf16(W, E.WhT, L.G * p.hidden, p.input, p.hidden, C->cs));
    if (E.Wpk) {  // the wide kernels' fragment-order copies
      const int GH = L.G * p.hidden, K1 = p.input + p.hidden;
      HIPCK(launch_pack_nt_bf16(W, GH, K1, K1, E.Wpk, C->cs));
      HIPCK(launch_pack_nt_bf16(E.WhT, p.hidden, GH, L.ld_wht, E.WhPk, C->cs));
    }
  } else {
    HIPCK(launch_transpose_wh((const float*)W, (float*)E.WhT, L.G * p.hidden, p.input, p.hidden, L.ld_wht, C->cs));
  }
  // live state <- x_0
  char* l0 = E.live(0);
  // the MLP's y_0 is [B][w_0]
  const size_t hb = L.mlpv ? size_t(p.batch) * size_t(C->widths[0]) * 4 : L.h_bytes;
  HIPCK(hipMemcpyAsync(l0, h0, hb, hipMemcpyDeviceToDevice, C->cs));
  if (L.G == 4) HIPCK(hipMemcpyAsync(E.cpart(l0), c0, L.c_bytes, hipMemcpyDeviceToDevice, C->cs));
  E.set_cur_live(l0);
  return AMBPTT_OK;
}

// ---- resident whole-pass kernel ----------------------------------------------

bool resident_possible(ambptt_ctx* C) {
  // the resident program is compiled before the launch: it takes no decision at run time
  if (!C->L.res || C->path_opt == 1 || C->store_policy == 1 || C->ftier) return false;
  if (C->res_cap < 0) {
    int cap = 0;
    if (resident_capacity(C->L.G, C->p.input, C->p.hidden, &cap) != hipSuccess) {
      (void)hipGetLastError();
      cap = 0;
    }
    C->res_cap = cap;
  }
  return C->L.r_nwg <= C->res_cap;
}

ambptt_status ensure_prog_host(ambptt_ctx* C, size_t ints) {
  if (ints <= C->prog_host_cap) return AMBPTT_OK;
  if (C->no_alloc)
    return fail(AMBPTT_EINVAL, "the resident program's staging buffer is not reserved (ambptt_set_int \"reserve\")");
  if (C->prog_host) {
    HIPCK(hipStreamSynchronize(C->cs));
    HIPCK(hipHostFree(C->prog_host));
    C->prog_host = nullptr;
    C->prog_host_cap = 0;
  }
  void* ptr = nullptr;
  HIPCK(hipHostMalloc(&ptr, ints * sizeof(int32_t), hipHostMallocDefault));
  C->prog_host = (int32_t*)ptr;
  C->prog_host_cap = ints;
  return AMBPTT_OK;
}

ambptt_status resident_args(ambptt_ctx* C, const void* x, const void* W, const float* b, ResidentArgs* out) {
  const Layout& L = C->L;
  const ambptt_problem& p = C->p;
  ResidentArgs a{};
  a.prog = (const int*)(C->ws + L.off_prog);
  a.x = (const float*)x;
  a.W = (const float*)W;
  a.bias = b;
  a.pool = C->pool;
  a.live0 = C->ws + L.off_live[0];
  a.live1 = C->ws + L.off_live[1];
  a.stride = L.stride;
  a.c_off = align_up(L.h_bytes);
  a.nslots = p.fast_slots;
  a.host = nullptr;
  if (C->host) HIPCK(hipHostGetDevicePointer((void**)&a.host, C->host, 0));
  a.Z = (float*)(C->ws + L.off_Z);
  a.P = (float*)(C->ws + L.off_P);
  a.dWp = (float*)(C->ws + L.off_dWp);
  a.dbp = (float*)(C->ws + L.off_dbp);
  a.loss_acc = (double*)(C->ws + L.off_loss);
  a.ready = (unsigned*)(C->ws + L.off_ready);
  a.consumed = (unsigned*)(C->ws + L.off_consumed);
  a.oflag = (unsigned*)(C->ws + L.off_oflag);
  a.status = (unsigned*)(C->ws + L.off_status);
  a.timeout = (long long)C->res_timeout_ms * 100000LL;  // s_memrealtime runs at 100 MHz
  a.B = p.batch;
  a.D = p.input;
  a.H = p.hidden;
  a.loss = p.loss;
  a.mtiles = L.r_mtiles;
  a.ng = L.r_ng;
  a.S = L.r_S;
  a.xcd_map = (L.r_nwg % 8 == 0 && 8 % L.r_mtiles == 0 && L.r_ng % (8 / L.r_mtiles) == 0) ? 1 : 0;
  a.inv_bh = 1.0f / float((double)p.batch * p.hidden);
  *out = a;
  return AMBPTT_OK;
}

// live state <- x_0 (the resident kernel reads no transposed weights)
ambptt_status resident_inputs(ambptt_ctx* C, const void* h0, const float* c0) {
  const Layout& L = C->L;
  char* l0 = C->ws + L.off_live[0];
  HIPCK(hipMemcpyAsync(l0, h0, L.h_bytes, hipMemcpyDeviceToDevice, C->cs));
  if (L.G == 4) HIPCK(hipMemcpyAsync(l0 + align_up(L.h_bytes), c0, L.c_bytes, hipMemcpyDeviceToDevice, C->cs));
  return AMBPTT_OK;
}

// Uploads the program, clears the barrier flags and launches the kernel.  The
// pinned staging buffer is rewritten only after the caller synchronised.
ambptt_status resident_launch(ambptt_ctx* C, ResidentArgs a, const std::vector<int32_t>& prog, bool timed) {
  const Layout& L = C->L;
  const size_t n = prog.size();
  if (n / 4 > L.r_prog_cap) return fail(AMBPTT_EINTERNAL, "resident program exceeds its workspace");
  ambptt_status s = ensure_prog_host(C, n);
  if (s != AMBPTT_OK) return s;
  std::memcpy(C->prog_host, prog.data(), n * sizeof(int32_t));
  HIPCK(hipMemcpyAsync(C->ws + L.off_prog, C->prog_host, n * sizeof(int32_t), hipMemcpyHostToDevice, C->cs));
  a.nprog = int(n / 4);
  HIPCK(launch_fill32(C->ws + L.off_ready, size_t(L.r_nwg), 0u, C->cs));
  HIPCK(launch_fill32(C->ws + L.off_consumed, size_t(L.r_nwg), 0u, C->cs));
  HIPCK(launch_fill32(C->ws + L.off_oflag, size_t(L.r_nwg), 0u, C->cs));
  HIPCK(launch_fill32(C->ws + L.off_status, 4, 0u, C->cs));
  if (timed) HIPCK(hipEventRecord(C->ev_r[0], C->cs));
  HIPCK(launch_resident(L.G, a, C->cs, C->res_coop));
  if (timed) HIPCK(hipEventRecord(C->ev_r[1], C->cs));
  return AMBPTT_OK;
}

// after the stream finished: did every wait end in time?
ambptt_status resident_status(ambptt_ctx* C) {
  HIPCK(hipMemcpy(C->status_host, C->ws + C->L.off_status, 2 * sizeof(unsigned), hipMemcpyDeviceToHost));
  if (C->status_host[0] == 0u) return AMBPTT_OK;
  const unsigned w = C->status_host[1];
  const unsigned code = w >> 24, entry = (w & 0xffffffu);
  const char* why = code == 0 ? "a barrier wait exceeded the timeout"
                  : code == 3 ? "two prefetches without a barrier between them"
                  : code == 4 ? "unknown program entry" : "abort";
  return fail(AMBPTT_EINTERNAL, std::string("resident pass aborted: ") + why +
                                    (entry ? " (program entry " + std::to_string(entry - 1) + ")" : std::string()));
}

// T_A: one forward step (barrier included); T_T: one forward step when every
// step also moves a state over the host link (stores, then prefetches).  Each
// from the difference of a long and a short program, so that the launch and
// the weight load cancel.
ambptt_status resident_calibrate(ambptt_ctx* C, const void* x, const void* W, const float* b, const void* h0,
                                 const float* c0, double* ta_us, double* tt_us) {
  const Layout& L = C->L;
  const ambptt_problem& p = C->p;
  ambptt_status s = ensure_host(C, 2, size_t(L.r_nwg) * 1024, true);
  if (s != AMBPTT_OK) return s;
  if ((s = resident_inputs(C, h0, c0)) != AMBPTT_OK) return s;
  ResidentArgs a;
  if ((s = resident_args(C, x, W, b, &a)) != AMBPTT_OK) return s;
  const int L0 = p.fast_slots, L1 = p.fast_slots + 1;
  auto program = [&](int steps, int kind) {
    std::vector<int32_t> v;
    int cur = L0;
    for (int i = 0; i < steps; ++i) {
      // stores as in the sweep: each step's output lands in a tier slot and
      // goes to the host right away; prefetches as in the reverse sweep
      const int dst = kind == 1 ? i % 2 : (cur == L0 ? L1 : L0);
      v.insert(v.end(), {kPFwd, int32_t(i % p.n_steps), cur, dst});
      cur = dst;
      if (kind == 1) v.insert(v.end(), {kPStore | kPStaged, 0, dst, i % 2});
      // each prefetch names the next one (entry 2 i + 3), as compiled programs do
      if (kind == 2) v.insert(v.end(), {kPPref, i + 1 < steps ? 2 * i + 3 : 0, i % 2, i % 2});
    }
    return v;
  };
  double per[3] = {0, 0, 0};
  const int kinds = p.fast_slots >= 2 ? 3 : 1;  // the host tier needs two slots
  for (int kind = 0; kind < kinds; ++kind) {
    float ms[2] = {0.f, 0.f};
    const int steps[2] = {16, 80};
    for (int rep = 0; rep < 2; ++rep) {  // the first round warms up
      for (int k = 0; k < 2; ++k) {
        if ((s = resident_launch(C, a, program(steps[k], kind), true)) != AMBPTT_OK) return s;
        HIPCK(hipEventSynchronize(C->ev_r[1]));
        HIPCK(hipEventElapsedTime(&ms[k], C->ev_r[0], C->ev_r[1]));
        if ((s = resident_status(C)) != AMBPTT_OK) return s;
      }
    }
    per[kind] = 1000.0 * double(ms[1] - ms[0]) / double(steps[1] - steps[0]);
  }
  *ta_us = std::max(per[0], 1e-3);
  *tt_us = std::max(per[1], per[2]);
  return AMBPTT_OK;
}

ambptt_status resident_run(ambptt_ctx* C, const void* x_seq, const void* W, const float* b, const void* h0,
                           const float* c0, float* dW, float* db, float* dh0, float* dc0, double* loss,
                           ambptt_stats* stats) {
  const ambptt_problem& p = C->p;
  const Layout& L = C->L;
  const double t0 = now_us();
  Plan plan;
  ResidentCounts rc;
  std::vector<int32_t> prog;
  try {
    plan = pass_plan(C);
    prog = compile_resident(plan, p.fast_slots, C->elide_prefetch, &rc);
    if (C->res_test_stall) prog.insert(prog.begin(), {kPCopy, INT32_MAX, p.fast_slots, p.fast_slots + 1});
  } catch (const std::length_error& e) {
    return fail(AMBPTT_EUNSUPPORTED, e.what());
  } catch (const std::exception& e) {
    return fail(AMBPTT_EINTERNAL, e.what());
  }
  const double t1 = now_us();
  ambptt_status s;
  if (plan.async && (s = ensure_host(C, plan.host_slots_used, size_t(L.r_nwg) * 1024, true)) != AMBPTT_OK)
    return s;
  ResidentArgs a;
  if ((s = resident_args(C, x_seq, W, b, &a)) != AMBPTT_OK) return s;
  a.dh0 = dh0;
  a.dc0 = dc0;
  HIPCK(launch_fill32(C->ws + L.off_loss, (size_t)L.loss_slots * 2, 0u, C->cs));
  if ((s = resident_inputs(C, h0, c0)) != AMBPTT_OK) return s;
  const bool timed = C->timing_sample > 0;
  if ((s = resident_launch(C, a, prog, timed)) != AMBPTT_OK) return s;
  const int GH = L.G * p.hidden, K1 = p.input + p.hidden;
  HIPCK(launch_resident_reduce(a.dWp, a.dbp, L.r_mtiles, GH, K1, dW, db, C->cs));
  const double scale = p.loss == AMBPTT_LOSS_HALF_SQ_LAST ? 0.5 : 1.0 / ((double)p.batch * p.hidden);
  double* dloss = (double*)(C->ws + L.off_lossout);
  HIPCK(launch_loss_sum((const double*)(C->ws + L.off_loss), L.loss_slots, scale, dloss, C->cs));
  HIPCK(hipMemcpyAsync(C->host_loss, dloss, sizeof(double), hipMemcpyDeviceToHost, C->cs));
  const double t_enq = now_us();
  HIPCK(hipStreamSynchronize(C->cs));
  const double t2 = now_us();
  if ((s = resident_status(C)) != AMBPTT_OK) return s;
  if (loss) *loss = *C->host_loss;
  if (stats) {
    ambptt_stats st{};
    st.mode = plan.online ? 3 : plan.async ? 1 : 0;
    st.interval = int32_t(plan.interval);
    st.window = 0;
    st.path = 1;
    st.n_steps = p.n_steps;
    st.actions = (int64_t)plan.acts.size();
    st.forward_evals = rc.forward_evals;
    st.adjoints = rc.adjoints;
    st.takeshots = rc.takeshots;
    st.takeshot_copies = rc.takeshot_copies;
    st.restores = rc.restores;
    st.stores = rc.stores;
    st.prefetches = rc.prefetches;
    st.prefetches_elided = rc.prefetches_elided;
    st.bytes_d2h = rc.stores * (int64_t)L.state_bytes;
    st.bytes_h2d = (rc.prefetches - rc.prefetches_elided) * (int64_t)L.state_bytes;
    st.compute_waits = 0;
    st.kernel_launches = 6;
    st.recompute_factor = double(rc.forward_evals) / double(p.n_steps);
    st.forward_cost = plan.weighted ? C->plan_cost : double(rc.forward_evals);
    st.schedule_us = t1 - t0;
    st.run_us = t2 - t1;
    st.enqueue_us = t_enq - t1;
    if (timed) {
      float ms = 0.f;
      HIPCK(hipEventElapsedTime(&ms, C->ev_r[0], C->ev_r[1]));
      st.kernel_us[AMBPTT_K_PASS] = 1000.0 * ms;
      st.kernel_samples[AMBPTT_K_PASS] = 1;
    }
    st.kernel_calls[AMBPTT_K_PASS] = 1;
    st.kernel_calls[AMBPTT_K_OTHER] = 1;
    *stats = st;
  }
  if (rc.forward_evals != plan.evals)
    return fail(AMBPTT_EINTERNAL, "resident forward count differs from the schedule");
  C->last_plan = std::move(plan);
  return AMBPTT_OK;
}

}  // namespace

// ---------------------------------------------------------------------------

extern "C" {

const char* ambptt_version(void) { return "ambptt 0.1 (gfx950)"; }

const char* ambptt_last_error(void) { return g_err.c_str(); }

int64_t ambptt_revolve_advances(int64_t n, int32_t s) {
  if (n < 1 || s < 1) return -1;
  return revolve_advances(n, s);
}

int64_t ambptt_schedule_evals(int64_t n, int32_t s, int64_t H, int32_t interval_min, int32_t* interval_out,
                              int32_t* mode_out) {
  if (n < 1 || s < 1 || H < 0 || interval_min < 0) return -1;
  bool async = false;
  int64_t I = 0, ev = 0;
  plan_counts(n, s, H, interval_min, &async, &I, &ev);
  if (interval_out) *interval_out = int32_t(I);
  if (mode_out) *mode_out = async ? 1 : 0;
  return ev;
}

ambptt_status ambptt_schedule_text(int64_t n, int32_t s, int64_t H, int32_t interval_min, char* buf, size_t cap,
                                   size_t* needed) {
  if (n < 1 || s < 1 || H < 0 || interval_min < 0) return fail(AMBPTT_EINVAL, "schedule: bad arguments");
  try {
    const std::string t = plan_text(make_plan(n, s, H, interval_min));
    if (needed) *needed = t.size() + 1;
    if (!buf || cap < t.size() + 1) return fail(AMBPTT_EINVAL, "schedule: buffer too small");
    std::memcpy(buf, t.c_str(), t.size() + 1);
    return AMBPTT_OK;
  } catch (const std::exception& e) {
    return fail(AMBPTT_EINTERNAL, e.what());
  }
}

static bool costs_ok(const double* costs, int64_t n) {
  for (int64_t t = 0; t < n; ++t)
    if (!(costs[t] > 0.0) || !(costs[t] < 1e300)) return false;
  return true;
}

ambptt_status ambptt_set_widths(ambptt_ctx* C, const int32_t* widths, int64_t count) {
  if (!C || !widths) return fail(AMBPTT_EINVAL, "ctx/widths is NULL");
  if (!C->L.mlpv) return fail(AMBPTT_EINVAL, "layer widths belong to the MLP cell");
  if (count != C->p.n_steps + 1) return fail(AMBPTT_EINVAL, "need n + 1 widths");
  int32_t top = 0;
  for (int64_t t = 0; t < count; ++t) {
    const int32_t w = widths[t];
    if (w < 16 || w % 16 || w > C->p.hidden) return fail(AMBPTT_EINVAL, "widths must be multiples of 16 up to hidden");
    top = std::max(top, w);
  }
  if (top != C->p.hidden) return fail(AMBPTT_EINVAL, "the largest width must equal the problem's hidden size");
  set_layer_widths(C, std::vector<int32_t>(widths, widths + count));
  return AMBPTT_OK;
}

ambptt_status ambptt_set_step_costs(ambptt_ctx* C, const double* costs, int64_t n) {
  if (!C) return fail(AMBPTT_EINVAL, "ctx is NULL");
  if (!costs || n == 0) {
    C->step_costs.clear();
    C->costs_version++;
    return AMBPTT_OK;
  }
  if (n != C->p.n_steps) return fail(AMBPTT_EINVAL, "step costs: need one cost per step of the problem");
  if (!costs_ok(costs, n)) return fail(AMBPTT_EINVAL, "step costs must be positive and finite");
  if (C->online) return fail(AMBPTT_EINVAL, "online checkpointing and step costs exclude each other");
  C->step_costs.assign(costs, costs + n);
  C->costs_version++;
  return AMBPTT_OK;
}

ambptt_status ambptt_schedule_text_costs(int64_t n, int32_t s, int64_t H, int32_t interval_min, const double* costs,
                                         char* buf, size_t cap, size_t* needed) {
  if (n < 1 || s < 1 || H < 0 || interval_min < 0 || !costs) return fail(AMBPTT_EINVAL, "schedule: bad arguments");
  if (!costs_ok(costs, n)) return fail(AMBPTT_EINVAL, "step costs must be positive and finite");
  try {
    const std::string t = plan_text(make_plan_costs(n, s, H, interval_min, std::vector<double>(costs, costs + n), nullptr));
    if (needed) *needed = t.size() + 1;
    if (!buf || cap < t.size() + 1) return fail(AMBPTT_EINVAL, "schedule: buffer too small");
    std::memcpy(buf, t.c_str(), t.size() + 1);
    return AMBPTT_OK;
  } catch (const std::length_error& e) {
    return fail(AMBPTT_EUNSUPPORTED, e.what());
  } catch (const std::invalid_argument& e) {
    return fail(AMBPTT_EINVAL, e.what());
  } catch (const std::exception& e) {
    return fail(AMBPTT_EINTERNAL, e.what());
  }
}

ambptt_status ambptt_schedule_text_sized(int64_t n, int32_t s, int64_t H, int32_t interval_min, const int64_t* sizes,
                                         const double* costs, char* buf, size_t cap, size_t* needed) {
  if (n < 1 || s < 1 || H < 0 || interval_min < 0 || !sizes) return fail(AMBPTT_EINVAL, "schedule: bad arguments");
  if (costs && !costs_ok(costs, n)) return fail(AMBPTT_EINVAL, "step costs must be positive and finite");
  try {
    const std::vector<double> c = costs ? std::vector<double>(costs, costs + n) : std::vector<double>();
    const std::string t = plan_text(make_plan_sized(n, s, H, interval_min, std::vector<int64_t>(sizes, sizes + n + 1),
                                                    costs ? &c : nullptr, nullptr));
    if (needed) *needed = t.size() + 1;
    if (!buf || cap < t.size() + 1) return fail(AMBPTT_EINVAL, "schedule: buffer too small");
    std::memcpy(buf, t.c_str(), t.size() + 1);
    return AMBPTT_OK;
  } catch (const std::length_error& e) {
    return fail(AMBPTT_EUNSUPPORTED, e.what());
  } catch (const std::invalid_argument& e) {
    return fail(AMBPTT_EINVAL, e.what());
  } catch (const std::exception& e) {
    return fail(AMBPTT_EINTERNAL, e.what());
  }
}

int64_t ambptt_interval_from_timings(double t_a_us, double t_t_us, int32_t s, int32_t rule) {
  if (!(t_a_us > 0.0) || !(t_t_us >= 0.0) || s < 1 || rule < 0 || rule > 1) {
    fail(AMBPTT_EINVAL, "interval: need T_A > 0, T_T >= 0, s >= 1, rule 0 or 1");
    return -1;
  }
  return interval_from_timings(t_a_us, t_t_us, s, rule, 0.0);
}

ambptt_status ambptt_schedule_text_online(int64_t n, int32_t s, int64_t H, int32_t interval_min, char* buf,
                                          size_t cap, size_t* needed) {
  if (n < 1 || s < 1 || H < 0 || interval_min < 0) return fail(AMBPTT_EINVAL, "schedule: bad arguments");
  try {
    const std::string t = plan_text(make_plan_online(n, s, H, interval_min));
    if (needed) *needed = t.size() + 1;
    if (!buf || cap < t.size() + 1) return fail(AMBPTT_EINVAL, "schedule: buffer too small");
    std::memcpy(buf, t.c_str(), t.size() + 1);
    return AMBPTT_OK;
  } catch (const std::exception& e) {
    return fail(AMBPTT_EINTERNAL, e.what());
  }
}

ambptt_status ambptt_resident_program(int64_t n, int32_t s, int64_t H, int32_t interval_min, int32_t flags,
                                      int32_t* buf, size_t cap, size_t* entries) {
  if (n < 1 || s < 1 || H < 0 || interval_min < 0 || (flags & ~3) != 0)
    return fail(AMBPTT_EINVAL, "resident program: bad arguments");
  try {
    const int64_t I = std::max<int32_t>(interval_min, 1);
    const Plan plan = (flags & 2) ? make_plan_online(n, s, H, I) : make_plan(n, s, H, I);
    const std::vector<int32_t> prog = compile_resident(plan, s, (flags & 1) != 0, nullptr);
    const size_t m = prog.size() / 4;
    if (entries) *entries = m;
    if (!buf || cap < m) return fail(AMBPTT_EINVAL, "resident program: buffer too small");
    std::memcpy(buf, prog.data(), prog.size() * sizeof(int32_t));
    return AMBPTT_OK;
  } catch (const std::exception& e) {
    return fail(AMBPTT_EINTERNAL, e.what());
  }
}

ambptt_status ambptt_query(const ambptt_problem* p, size_t* state_bytes, size_t* slot_pool_bytes,
                           size_t* workspace_bytes) {
  ambptt_status s = validate(p);
  if (s != AMBPTT_OK) return s;
  const Layout L = make_layout(p, 0);
  if (state_bytes) *state_bytes = L.stride;
  if (slot_pool_bytes) *slot_pool_bytes = L.stride * (size_t)p->fast_slots;
  if (workspace_bytes) *workspace_bytes = L.total;
  return AMBPTT_OK;
}

ambptt_status ambptt_create(const ambptt_problem* p, void* stream, ambptt_ctx** out) {
  if (!out) return fail(AMBPTT_EINVAL, "out is NULL");
  *out = nullptr;
  ambptt_status s = validate(p);
  if (s != AMBPTT_OK) return s;
  ambptt_ctx* C = new ambptt_ctx();
  C->p = *p;
  C->L = make_layout(p, 0);
  C->interval_min = p->interval_min;
  C->cs = (hipStream_t)stream;
  auto bail = [&](const char* what, hipError_t e) {
    std::string m = std::string(what) + ": " + hipGetErrorString(e);
    ambptt_destroy(C);
    return fail(AMBPTT_EHIP, m);
  };
  hipError_t e;
  if ((e = hipGetDevice(&C->device)) != hipSuccess) return bail("hipGetDevice", e);
  if (C->device >= 0 && C->device < kMaxDevices) {  // the device is current: its copy of the scratch array
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch[C->device]) {
      void* ptr = nullptr;
      if ((e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch))) != hipSuccess) return bail("hipGetSymbolAddress", e);
      if (!ptr) return bail("hipGetSymbolAddress", hipErrorInvalidSymbol);
      g_scratch[C->device] = (char*)ptr;
    }
  }
  if ((e = hipStreamCreateWithFlags(&C->xs, hipStreamNonBlocking)) != hipSuccess) return bail("hipStreamCreate", e);
  if ((e = hipStreamCreateWithFlags(&C->ds, hipStreamNonBlocking)) != hipSuccess) return bail("hipStreamCreate", e);
  if (C->L.mlpv) set_layer_widths(C, std::vector<int32_t>(size_t(p->n_steps) + 1, p->hidden));
  C->ev_slot.resize(size_t(p->fast_slots), nullptr);
  C->pend.assign(size_t(p->fast_slots), kNone);
  if ((e = make_sync_events(C)) != hipSuccess) return bail("hipEventCreate", e);
  void* hl = nullptr;
  if ((e = hipHostMalloc(&hl, 64, hipHostMallocDefault)) != hipSuccess) return bail("hipHostMalloc", e);
  C->host_loss = (double*)hl;
  void* sh = nullptr;
  if ((e = hipHostMalloc(&sh, 64, hipHostMallocDefault)) != hipSuccess) return bail("hipHostMalloc", e);
  C->status_host = (unsigned*)sh;
  for (auto& ev : C->ev_r)
    if ((e = hipEventCreate(&ev)) != hipSuccess) return bail("hipEventCreate", e);
  *out = C;
  return AMBPTT_OK;
}

ambptt_status ambptt_bind(ambptt_ctx* C, void* slot_pool, size_t pool_bytes, void* workspace, size_t ws_bytes) {
  if (!C) return fail(AMBPTT_EINVAL, "ctx is NULL");
  if (!slot_pool) return fail(AMBPTT_EINVAL, "the slot pool is required");
  if (((uintptr_t)slot_pool % kAlign) || ((uintptr_t)workspace % kAlign))
    return fail(AMBPTT_EINVAL, "slot pool and workspace must be 256-byte aligned");
  if (pool_bytes < C->L.stride * (size_t)C->p.fast_slots) return fail(AMBPTT_EINVAL, "slot pool too small");
  if (workspace && ws_bytes < C->L.total) return fail(AMBPTT_EINVAL, "workspace too small");
  C->pool = (char*)slot_pool;
  C->ws = (char*)workspace;
  return AMBPTT_OK;
}

static ambptt_status reserve(ambptt_ctx* C);

ambptt_status ambptt_set_int(ambptt_ctx* C, const char* key, int64_t v) {
  if (!C || !key) return fail(AMBPTT_EINVAL, "ctx/key is NULL");
  const std::string k(key);
  if (k == "timing_sample") {
    if (v < 0) return fail(AMBPTT_EINVAL, "timing_sample must be >= 0");
    C->timing_sample = v;
  } else if (k == "elide_prefetch") {
    C->elide_prefetch = v != 0;
  } else if (k == "window") {
    const int wmax = auto_window(&C->p);
    if (v < 0 || v > wmax) return fail(AMBPTT_EINVAL, "window must be in [0, " + std::to_string(wmax) + "]");
    C->window_opt = int(v);
    const Layout L2 = make_layout(&C->p, int(v == 0 ? wmax : v));
    // same offsets except the rings, which only shrink
    C->L.window = L2.window;
  } else if (k == "path") {
    if (v < 0 || v > 2) return fail(AMBPTT_EINVAL, "path must be 0 (auto), 1 (per-step launches) or 2 (resident)");
    C->path_opt = int(v);
  } else if (k == "wide_batch") {
    C->wide_opt = v != 0;
  } else if (k == "event_system_fence") {
    if (C->sys_fence != (v != 0)) {
      C->sys_fence = v != 0;
      hipError_t e = hipDeviceSynchronize();
      if (e == hipSuccess) e = make_sync_events(C);
      if (e != hipSuccess) return fail(AMBPTT_EHIP, std::string("event_system_fence: ") + hipGetErrorString(e));
    }
  } else if (k == "host_waits") {
    if (v < -1 || v > 1) return fail(AMBPTT_EINVAL, "host_waits must be -1 (by path), 0 or 1");
    C->host_waits = int(v);
  } else if (k == "test_copy_delay_us") {
    if (v < 0 || v > 100000) return fail(AMBPTT_EINVAL, "test_copy_delay_us must be 0 .. 100000");
    C->test_copy_delay_us = v;
  } else if (k == "test_poison") {
    C->test_poison = v != 0;
  } else if (k == "lds_gemm") {
    if (v < 0 || v > 2) return fail(AMBPTT_EINVAL, "lds_gemm must be 0, 1 or 2");
    C->lds_gemm = int(v);
  } else if (k == "hadj_launch") {
    C->hadj_launch = v != 0;
  } else if (k == "prod_split") {
    C->prod_split = v != 0;
  } else if (k == "uniform_sizes") {
    if (v < 0 || v > 1) return fail(AMBPTT_EINVAL, "uniform_sizes must be 0 or 1");
    C->uniform_sizes = v == 1;
  } else if (k == "store_policy") {
    if (v < 0 || v > 1) return fail(AMBPTT_EINVAL, "store_policy must be 0 (every I-th state) or 1 (when the previous store completed)");
    if (v == 1 && C->path_opt == 2) return fail(AMBPTT_EUNSUPPORTED, "store_policy 1 runs on the per-step path only");
    if (v == 1 && C->online) return fail(AMBPTT_EINVAL, "store_policy 1 and online checkpointing exclude each other");
    C->store_policy = int(v);
  } else if (k == "interval_rule") {
    if (v < 0 || v > 1) return fail(AMBPTT_EINVAL, "interval_rule must be 0 (ceil(T_T / T_A)) or 1 (least modelled time)");
    C->interval_rule = int(v);
  } else if (k == "online") {
    if (v < 0 || v > 1) return fail(AMBPTT_EINVAL, "online must be 0 or 1");
    if (v == 1 && C->store_policy == 1)
      return fail(AMBPTT_EINVAL, "store_policy 1 and online checkpointing exclude each other");
    if (v == 1 && C->ftier) return fail(AMBPTT_EUNSUPPORTED, "online checkpointing does not run over a file tier");
    if (v == 1 && !C->step_costs.empty()) return fail(AMBPTT_EINVAL, "online checkpointing and step costs exclude each other");
    C->online = v != 0;
  } else if (k == "dw_stream") {
    if (v < -1 || v > 1) return fail(AMBPTT_EINVAL, "dw_stream must be -1 (by path), 0 or 1");
    C->dw_stream = int(v);
  } else if (k == "resident_cooperative") {
    C->res_coop = v != 0;
  } else if (k == "resident_test_stall") {
    C->res_test_stall = v != 0;
  } else if (k == "resident_timeout_ms") {
    if (v < 0 || v > 600000) return fail(AMBPTT_EINVAL, "resident_timeout_ms must be in [0, 600000]");
    C->res_timeout_ms = v;
  } else if (k == "reserve") {
    if (v != 1) return fail(AMBPTT_EINVAL, "reserve: 1 allocates what the current schedule needs");
    return reserve(C);
  } else if (k == "interval_min") {
    if (v < 0) return fail(AMBPTT_EINVAL, "interval_min must be >= 0");
    C->interval_min = v;
  } else {
    return fail(AMBPTT_EINVAL, "unknown key " + k);
  }
  return AMBPTT_OK;
}

static ambptt_status check_run_args(ambptt_ctx* C, const void* x_seq, const void* W, const float* b, const void* h0,
                                    const float* c0) {
  if (!C) return fail(AMBPTT_EINVAL, "ctx is NULL");
  if (!C->pool) return fail(AMBPTT_EINVAL, "ambptt_bind has not been called");
  if (!C->ws) return fail(AMBPTT_EINVAL, "no workspace is bound (only ambptt_run_noalloc runs without one)");
  if ((!x_seq && C->p.input > 0) || !W || !b || !h0) return fail(AMBPTT_EINVAL, "missing input pointer");
  if (C->L.G == 4 && !c0) return fail(AMBPTT_EINVAL, "LSTM needs c0");
  return AMBPTT_OK;
}

ambptt_status ambptt_calibrate(ambptt_ctx* C, const void* x_seq, const void* W, const float* b, const void* h0,
                               const float* c0, int32_t* interval_min_out, double* t_a_us, double* t_t_us) {
  ambptt_status s = check_run_args(C, x_seq, W, b, h0, c0);
  if (s != AMBPTT_OK) return s;
  if (C->path_opt == 2 && !resident_possible(C))
    return fail(AMBPTT_EUNSUPPORTED, "the resident kernel does not fit this problem on this device");
  if (resident_possible(C)) {
    double ta = 0.0, tt = 0.0;
    if ((s = resident_calibrate(C, x_seq, W, b, h0, c0, &ta, &tt)) != AMBPTT_OK) return s;
    // transfers that lengthen a step by less than 5% count as hidden
    const int64_t I = interval_from_timings(ta, tt, C->p.fast_slots, C->interval_rule, 0.05);
    C->interval_min = I;
    if (interval_min_out) *interval_min_out = int32_t(std::min<int64_t>(I, INT32_MAX));
    if (t_a_us) *t_a_us = ta;
    if (t_t_us) *t_t_us = tt;
    return AMBPTT_OK;
  }
  Exec E(C, x_seq, W, b);
  if ((s = prepare_inputs(C, W, h0, c0, E)) != AMBPTT_OK) return s;
  if ((s = ensure_host(C, 2, C->L.stride, true)) != AMBPTT_OK) return s;
  hipEvent_t e0, e1;
  HIPCK(hipEventCreateWithFlags(&e0, event_flags(C, true)));
  HIPCK(hipEventCreateWithFlags(&e1, event_flags(C, true)));
  const int64_t n = C->p.n_steps;
  const int reps = 16;
  float ms = 0.f;
  for (int warm = 0; warm < 2; ++warm) {
    HIPCK(hipEventRecord(e0, C->cs));
    for (int i = 0; i < reps; ++i) {
      char* dst = E.other_live();
      if ((s = E.fwd_step(i % n, E.cur, dst)) != AMBPTT_OK) return s;
      E.set_cur_live(dst);
    }
    HIPCK(hipEventRecord(e1, C->cs));
    HIPCK(hipEventSynchronize(e1));
    HIPCK(hipEventElapsedTime(&ms, e0, e1));
  }
  const double ta = 1000.0 * ms / reps;
  double tt = 0.0;
  for (int dir = 0; dir < 2; ++dir) {
    double best = 1e30;
    for (int rep = 0; rep < 3; ++rep) {
      HIPCK(hipEventRecord(e0, C->xs));
      if (dir == 0)
        HIPCK(hipMemcpyAsync(C->host, E.live(0), C->L.state_bytes, hipMemcpyDeviceToHost, C->xs));
      else
        HIPCK(hipMemcpyAsync(E.live(1), C->host, C->L.state_bytes, hipMemcpyHostToDevice, C->xs));
      HIPCK(hipEventRecord(e1, C->xs));
      HIPCK(hipEventSynchronize(e1));
      HIPCK(hipEventElapsedTime(&ms, e0, e1));
      best = std::min(best, 1000.0 * ms);
    }
    tt = std::max(tt, best);
  }
  // The sweep's view of a transfer: per step of a sweep that stores every
  // state through the two alternating fast slots (the executor's own store
  // path, copies running beside the forward steps), as the resident kernel's
  // calibration measures it.  A transfer hidden behind a step gives T_A.
  if (!C->ftier && n >= 9 && C->p.fast_slots >= 2) {
    const int64_t steps = std::min<int64_t>(n - 1, 24);
    std::vector<Action> acts;
    for (int64_t i = 0; i < steps; ++i) {
      acts.push_back({Op::Snap, i % 2, i, 0});
      acts.push_back({Op::Store, i % 2, i % 2, i});
      acts.push_back({Op::Advance, i, i + 1, 0});
    }
    const int64_t lens[2] = {steps / 3, steps};
    // The host link can be slow for a few milliseconds at a time (seen
    // right after other processes pinned and released large blocks): an
    // attempt whose sweep cost per step exceeds 1.5 times the larger of the
    // plain copy and the step is measured again after a pause, up to three
    // attempts, and the least cost counts.
    double sweep = 1e30;
    for (int attempt = 0; attempt < 3 && sweep > 1.5 * std::max(tt, ta); ++attempt) {
      if (attempt) std::this_thread::sleep_for(std::chrono::milliseconds(50));
      double per[2] = {1e30, 1e30};  // the best of three rounds after a warm-up round
      for (int rep = 0; rep < 4; ++rep) {
        for (int k = 0; k < 2; ++k) {
          std::fill(C->pend.begin(), C->pend.end(), kNone);
          HIPCK(hipStreamSynchronize(C->xs));
          HIPCK(hipStreamSynchronize(C->cs));
          HIPCK(hipEventRecord(e0, C->cs));
          const std::vector<Action> part(acts.begin(), acts.begin() + 3 * lens[k]);
          if ((s = E.run_acts(part, 0, nullptr, nullptr)) != AMBPTT_OK) return s;
          HIPCK(hipEventRecord(C->ev_c, C->xs));  // the last store
          HIPCK(hipStreamWaitEvent(C->cs, C->ev_c, 0));
          HIPCK(hipEventRecord(e1, C->cs));
          HIPCK(hipEventSynchronize(e1));
          HIPCK(hipEventElapsedTime(&ms, e0, e1));
          if (rep > 0) per[k] = std::min(per[k], 1000.0 * ms);
        }
      }
      sweep = std::min(sweep, (per[1] - per[0]) / double(lens[1] - lens[0]));
    }
    HIPCK(hipStreamSynchronize(C->xs));
    std::fill(C->pend.begin(), C->pend.end(), kNone);
    tt = std::max(tt, sweep);
  }
  if (C->ftier) {  // the file takes every stored state too: the slower of the two links sets T_T
    HIPCK(hipMemcpy(C->host, E.live(0), C->L.state_bytes, hipMemcpyDeviceToHost));
    double best = 1e30;
    for (int rep = 0; rep < 3; ++rep) {
      const double sec = C->ftier->time_write(C->host, C->L.state_bytes);
      if (sec < 0) return fail(AMBPTT_EINTERNAL, "file tier: calibration write failed");
      best = std::min(best, 1e6 * sec);
    }
    tt = std::max(tt, best);
  }
  HIPCK(hipEventDestroy(e0));
  HIPCK(hipEventDestroy(e1));
  const int64_t I = interval_from_timings(ta, tt, C->p.fast_slots, C->interval_rule, 0.0);
  C->interval_min = I;
  if (interval_min_out) *interval_min_out = int32_t(std::min<int64_t>(I, INT32_MAX));
  if (t_a_us) *t_a_us = ta;
  if (t_t_us) *t_t_us = tt;
  return AMBPTT_OK;
}

// Host slots the per-step pass of `plan` fills: the plan's, or with stores
// decided during the sweep as many as it may take; in front of a file tier
// only the pinned ring.
static int64_t host_slots_needed(const ambptt_ctx* C, const Plan& plan, bool dynamic) {
  int64_t slots = dynamic ? std::min<int64_t>(slow_capacity(C), C->p.n_steps) : plan.host_slots_used;
  if (C->ftier) slots = std::min<int64_t>(slots, C->p.slow_slots);
  return slots;
}

// Allocates now what a pass of the current schedule would otherwise allocate
// on first use (the pinned host tier and the resident program's staging), so
// that ambptt_run_noalloc can run it.  The interval is the context's I_min,
// or 1 (the most host slots any interval takes) before calibration.
static ambptt_status reserve(ambptt_ctx* C) {
  const ambptt_problem& p = C->p;
  Plan plan;
  std::vector<int32_t> prog;
  const bool res = resident_possible(C);
  try {
    plan = pass_plan(C);
    if (res) {
      ResidentCounts rc;
      prog = compile_resident(plan, p.fast_slots, C->elide_prefetch, &rc);
    }
  } catch (const std::length_error& e) {
    return fail(AMBPTT_EUNSUPPORTED, e.what());
  } catch (const std::exception& e) {
    return fail(AMBPTT_EINTERNAL, e.what());
  }
  ambptt_status s;
  if ((s = grow_slot_events(C, plan.slot_ids)) != AMBPTT_OK) return s;
  if (res) {
    if ((s = ensure_prog_host(C, prog.size() + 4)) != AMBPTT_OK) return s;
    if (plan.async) return ensure_host(C, plan.host_slots_used, size_t(C->L.r_nwg) * 1024, true);
    return AMBPTT_OK;
  }
  const bool dynamic = C->store_policy == 1 && plan.async && p.n_steps >= 2;
  if (plan.async) return ensure_host(C, host_slots_needed(C, plan, dynamic), C->L.stride, C->ftier != nullptr);
  return AMBPTT_OK;
}

// One pass on the context's bound buffers (the workspace is C->ws).
static ambptt_status run_pass(ambptt_ctx* C, const void* x_seq, const void* W, const float* b, const void* h0,
                              const float* c0, float* dW, float* db, float* dh0, float* dc0, double* loss,
                              ambptt_stats* stats) {
  ambptt_status s;
  const ambptt_problem& p = C->p;
  const Layout& L = C->L;
  if (C->path_opt == 2 && C->store_policy == 1)
    return fail(AMBPTT_EUNSUPPORTED, "store_policy 1 runs on the per-step path only");
  if (C->path_opt == 2 && !resident_possible(C))
    return fail(AMBPTT_EUNSUPPORTED, "the resident kernel does not fit this problem on this device");
  if (resident_possible(C)) return resident_run(C, x_seq, W, b, h0, c0, dW, db, dh0, dc0, loss, stats);
  if (L.mlpv && C->online)
    return fail(AMBPTT_EUNSUPPORTED, "online checkpointing is not available for states of different sizes");
  const double t0 = now_us();
  Plan plan;
  try {
    plan = pass_plan(C);
  } catch (const std::length_error& e) {
    return fail(AMBPTT_EUNSUPPORTED, e.what());
  } catch (const std::exception& e) {
    return fail(AMBPTT_EINTERNAL, e.what());
  }
  const double t1 = now_us();
  // stores decided during the sweep, where the fixed-interval policy would
  // use the host tier at all
  const bool dynamic = C->store_policy == 1 && plan.async && p.n_steps >= 2;
  if (plan.async) {
    const size_t slots = size_t(host_slots_needed(C, plan, dynamic));
    if ((s = ensure_host(C, int64_t(slots), L.stride, C->ftier != nullptr)) != AMBPTT_OK) return s;
    if (C->ftier) {
      if (!C->ftier->finish()) return fail(AMBPTT_EINTERNAL, C->ftier->error());
      while (C->ev_file.size() < slots) {
        hipEvent_t ev;
        HIPCK(hipEventCreateWithFlags(&ev, hipEventDisableTiming));
        C->ev_file.push_back(ev);
      }
      while (C->ev_file.size() > slots) {
        HIPCK(hipEventDestroy(C->ev_file.back()));
        C->ev_file.pop_back();
      }
      C->ftier->begin(C->host, int64_t(slots), L.stride, L.state_bytes);
      C->ftier->bytes_written = C->ftier->bytes_read = 0;
    }
  }
  Exec E(C, x_seq, W, b);
  if ((s = E.grow_slots(plan.slot_ids)) != AMBPTT_OK) return s;
  std::fill(C->pend.begin(), C->pend.end(), kNone);
  const size_t GH = (size_t)L.G * p.hidden;
  if (!L.mlp) {  // windows accumulate into dW; the MLP writes each layer once
    HIPCK(launch_fill32(dW, GH * (p.input + p.hidden), 0u, C->cs));
    HIPCK(launch_fill32(db, GH, 0u, C->cs));
  }
  HIPCK(launch_fill32(C->ws + L.off_loss, (size_t)L.loss_slots * 2, 0u, C->cs));
  if ((s = prepare_inputs(C, W, h0, c0, E)) != AMBPTT_OK) return s;
  if (dynamic) {
    std::vector<int64_t> starts;
    if ((s = E.dynamic_sweep(starts, dW, db)) != AMBPTT_OK) return s;
    try {
      const std::vector<double>* costs = C->step_costs.empty() ? nullptr : &C->step_costs;
      plan = L.mlpv ? make_plan_sized_starts(p.n_steps, p.fast_slots, slow_capacity(C), starts, plan_units(C), costs,
                                             &C->plan_cost)
                    : make_plan_starts(p.n_steps, p.fast_slots, slow_capacity(C), starts, costs, &C->plan_cost);
    } catch (const std::exception& e) {
      // the sweep is enqueued: let it and its stores finish before reporting
      (void)hipStreamSynchronize(C->cs);
      (void)hipStreamSynchronize(C->xs);
      (void)hipStreamSynchronize(C->ds);
      if (C->ftier) (void)C->ftier->finish();
      if (dynamic_cast<const std::length_error*>(&e)) return fail(AMBPTT_EUNSUPPORTED, e.what());
      return fail(AMBPTT_EINTERNAL, e.what());
    }
    if ((s = E.grow_slots(plan.slot_ids)) != AMBPTT_OK) return s;
    for (size_t k = 1; k <= starts.size(); ++k)  // the longest interval
      plan.interval = std::max(plan.interval, (k < starts.size() ? starts[k] : p.n_steps) - starts[k - 1]);
    // the sweep ran the plan's first 3 (K - 1) actions: snapshot, store and advance per stored start
    if ((s = E.run_acts(plan.acts, 3 * (starts.size() - 1), dW, db)) != AMBPTT_OK) return s;
  } else if ((s = E.run(plan, dW, db)) != AMBPTT_OK) {
    return s;
  }
  if ((s = E.final_step(dh0, dc0)) != AMBPTT_OK) return s;
  const double t_enq = now_us();
  double scale = 1.0;
  if (p.loss == AMBPTT_LOSS_HALF_SQ_LAST) scale = 0.5;
  else scale = 1.0 / ((double)p.batch * p.hidden);
  double* dloss = (double*)(C->ws + L.off_lossout);
  HIPCK(launch_loss_sum((const double*)(C->ws + L.off_loss), L.loss_slots, scale, dloss, C->cs));
  HIPCK(hipMemcpyAsync(C->host_loss, dloss, sizeof(double), hipMemcpyDeviceToHost, C->cs));
  HIPCK(hipStreamSynchronize(C->cs));
  HIPCK(hipStreamSynchronize(C->ds));
  HIPCK(hipStreamSynchronize(C->xs));
  if (C->ftier && plan.async && !C->ftier->finish()) return fail(AMBPTT_EINTERNAL, C->ftier->error());
  const double t2 = now_us();
  if (loss) *loss = *C->host_loss;
  ambptt_stats& st = E.st;
  if (C->ftier && plan.async) {
    st.bytes_file_w = C->ftier->bytes_written;
    st.bytes_file_r = C->ftier->bytes_read;
  }
  double sum[6] = {0, 0, 0, 0, 0, 0};
  int64_t cnt[6] = {0, 0, 0, 0, 0, 0};
  for (auto& smp : E.samples) {
    float ms = 0.f;
    HIPCK(hipEventElapsedTime(&ms, smp.a, smp.b));
    sum[smp.cls] += 1000.0 * ms;
    cnt[smp.cls]++;
  }
  if (stats) {
    st.mode = plan.online ? 3 : plan.dynamic ? 2 : plan.async ? 1 : 0;
    st.interval = int32_t(plan.interval);
    st.window = L.window;
    st.n_steps = p.n_steps;
    st.actions = (int64_t)plan.acts.size();
    st.recompute_factor = double(st.forward_evals) / double(p.n_steps);
    st.forward_cost = plan.weighted ? C->plan_cost : double(st.forward_evals);
    st.schedule_us = t1 - t0;
    st.run_us = t2 - t1;
    st.enqueue_us = t_enq - t1;
    for (int k = 0; k < 6; ++k) {
      st.kernel_us[k] = cnt[k] ? sum[k] / cnt[k] : 0.0;
      st.kernel_samples[k] = cnt[k];
      st.kernel_calls[k] = E.calls[k];
    }
    *stats = st;
  }
  if (st.forward_evals != plan.evals)
    return fail(AMBPTT_EINTERNAL, "executor forward count " + std::to_string(st.forward_evals) +
                                      " != schedule count " + std::to_string(plan.evals));
  C->last_plan = std::move(plan);
  return AMBPTT_OK;
}

ambptt_status ambptt_run(ambptt_ctx* C, const void* x_seq, const void* W, const float* b, const void* h0,
                         const float* c0, float* dW, float* db, float* dh0, float* dc0, double* loss,
                         ambptt_stats* stats) {
  ambptt_status s = check_run_args(C, x_seq, W, b, h0, c0);
  if (s != AMBPTT_OK) return s;
  if (!dW || !db || !dh0 || (C->L.G == 4 && !dc0)) return fail(AMBPTT_EINVAL, "missing gradient pointer");
  if (C->p.slow_slots > 0 && C->interval_min == 0) {
    if ((s = ambptt_calibrate(C, x_seq, W, b, h0, c0, nullptr, nullptr, nullptr)) != AMBPTT_OK) return s;
  }
  return run_pass(C, x_seq, W, b, h0, c0, dW, db, dh0, dc0, loss, stats);
}

ambptt_status ambptt_run_noalloc(ambptt_ctx* C, const void* x_seq, const void* W, const float* b, const void* h0,
                                 const float* c0, float* dW, float* db, float* dh0, float* dc0, double* loss,
                                 ambptt_stats* stats) {
  if (!C) return fail(AMBPTT_EINVAL, "ctx is NULL");
  if (!C->pool) return fail(AMBPTT_EINVAL, "ambptt_bind has not been called");
  if ((!x_seq && C->p.input > 0) || !W || !b || !h0) return fail(AMBPTT_EINVAL, "missing input pointer");
  if (C->L.G == 4 && !c0) return fail(AMBPTT_EINVAL, "LSTM needs c0");
  if (!dW || !db || !dh0 || (C->L.G == 4 && !dc0)) return fail(AMBPTT_EINVAL, "missing gradient pointer");
  if (C->L.total > kScratchBytes)
    return fail(AMBPTT_EINVAL, "the workspace of this problem (" + std::to_string(C->L.total) +
                                   " bytes) exceeds the static scratch of " + std::to_string(kScratchBytes) + " bytes");
  if (C->p.slow_slots > 0 && C->interval_min == 0)
    return fail(AMBPTT_EINVAL, "the interval is not set: call ambptt_calibrate or set \"interval_min\" first");
  if (C->ftier) return fail(AMBPTT_EUNSUPPORTED, "the file tier is not available without allocation");
  if (C->device < 0 || C->device >= kMaxDevices || !g_scratch[C->device])
    return fail(AMBPTT_EINTERNAL, "no scratch address for this context's device");
  char* const bound = C->ws;
  C->ws = g_scratch[C->device];
  C->no_alloc = true;
  const ambptt_status s = run_pass(C, x_seq, W, b, h0, c0, dW, db, dh0, dc0, loss, stats);
  C->no_alloc = false;
  C->ws = bound;
  return s;
}

ambptt_status ambptt_set_file_tier(ambptt_ctx* C, const char* dir, int64_t file_slots) {
  if (!C) return fail(AMBPTT_EINVAL, "ctx is NULL");
  if (file_slots < 0) return fail(AMBPTT_EINVAL, "file_slots must be >= 0");
  if (file_slots > 0 && (!dir || !*dir)) return fail(AMBPTT_EINVAL, "file tier: a directory is required");
  if (file_slots > 0 && C->p.slow_slots < 1)
    return fail(AMBPTT_EINVAL, "file tier: the problem needs at least one pinned host slot in front of the file");
  if (file_slots > 0 && C->online)
    return fail(AMBPTT_EUNSUPPORTED, "online checkpointing does not run over a file tier");
  if (file_slots > 0 && C->path_opt == 2) return fail(AMBPTT_EUNSUPPORTED, "the file tier runs on the per-step path only");
  if (C->ftier) {
    (void)hipStreamSynchronize(C->xs);
    (void)C->ftier->finish();
    delete C->ftier;
    C->ftier = nullptr;
  }
  if (file_slots == 0) return AMBPTT_OK;
  std::string err;
  C->ftier = FileTier::open(dir, file_slots, &err);
  if (!C->ftier) return fail(AMBPTT_EINVAL, err);
  return AMBPTT_OK;
}

ambptt_status ambptt_last_schedule_text(ambptt_ctx* C, char* buf, size_t cap, size_t* needed) {
  if (!C) return fail(AMBPTT_EINVAL, "ctx is NULL");
  if (C->last_plan.n == 0) return fail(AMBPTT_EINVAL, "no pass has run on this context");
  const std::string t = plan_text(C->last_plan);
  if (needed) *needed = t.size() + 1;
  if (!buf || cap < t.size() + 1) return fail(AMBPTT_EINVAL, "schedule: buffer too small");
  std::memcpy(buf, t.c_str(), t.size() + 1);
  return AMBPTT_OK;
}

ambptt_status ambptt_schedule_text_starts(int64_t n, int32_t s, int64_t H, const int64_t* starts, int64_t nstarts,
                                          char* buf, size_t cap, size_t* needed) {
  if (!starts || nstarts < 1) return fail(AMBPTT_EINVAL, "schedule: no interval starts");
  try {
    const std::string t = plan_text(make_plan_starts(n, s, H, std::vector<int64_t>(starts, starts + nstarts)));
    if (needed) *needed = t.size() + 1;
    if (!buf || cap < t.size() + 1) return fail(AMBPTT_EINVAL, "schedule: buffer too small");
    std::memcpy(buf, t.c_str(), t.size() + 1);
    return AMBPTT_OK;
  } catch (const std::invalid_argument& e) {
    return fail(AMBPTT_EINVAL, e.what());
  } catch (const std::exception& e) {
    return fail(AMBPTT_EINTERNAL, e.what());
  }
}

ambptt_status ambptt_schedule_text_starts_costs(int64_t n, int32_t s, int64_t H, const int64_t* starts,
                                                int64_t nstarts, const double* costs, char* buf, size_t cap,
                                                size_t* needed) {
  if (!starts || nstarts < 1) return fail(AMBPTT_EINVAL, "schedule: no interval starts");
  if (!costs || n < 1) return fail(AMBPTT_EINVAL, "schedule: need one cost per step");
  try {
    const std::vector<double> cv(costs, costs + n);
    const std::string t =
        plan_text(make_plan_starts(n, s, H, std::vector<int64_t>(starts, starts + nstarts), &cv, nullptr));
    if (needed) *needed = t.size() + 1;
    if (!buf || cap < t.size() + 1) return fail(AMBPTT_EINVAL, "schedule: buffer too small");
    std::memcpy(buf, t.c_str(), t.size() + 1);
    return AMBPTT_OK;
  } catch (const std::length_error& e) {
    return fail(AMBPTT_EUNSUPPORTED, e.what());
  } catch (const std::invalid_argument& e) {
    return fail(AMBPTT_EINVAL, e.what());
  } catch (const std::exception& e) {
    return fail(AMBPTT_EINTERNAL, e.what());
  }
}

void ambptt_destroy(ambptt_ctx* C) {
  if (!C) return;
  if (C->xs) (void)hipStreamSynchronize(C->xs);
  for (auto& ev : C->ev_slot)
    if (ev) (void)hipEventDestroy(ev);
  if (C->ev_c) (void)hipEventDestroy(C->ev_c);
  for (auto& ev : C->tpool) (void)hipEventDestroy(ev);
  if (C->ds) (void)hipStreamSynchronize(C->ds);
  for (auto& ev : C->ev_dw)
    if (ev) (void)hipEventDestroy(ev);
  if (C->ev_c2) (void)hipEventDestroy(C->ev_c2);
  for (auto& ev : C->ev_end)
    if (ev) (void)hipEventDestroy(ev);
  if (C->ftier) {
    (void)C->ftier->finish();
    delete C->ftier;
  }
  for (auto& ev : C->ev_file) (void)hipEventDestroy(ev);
  if (C->ds) (void)hipStreamDestroy(C->ds);
  if (C->xs) (void)hipStreamDestroy(C->xs);
  free_host(C);
  if (C->host_loss) (void)hipHostFree(C->host_loss);
  if (C->prog_host) {
    (void)hipStreamSynchronize(C->cs);
    (void)hipHostFree(C->prog_host);
  }
  if (C->status_host) (void)hipHostFree(C->status_host);
  for (auto& ev : C->ev_r)
    if (ev) (void)hipEventDestroy(ev);
  delete C;
}

}  // extern "C"
