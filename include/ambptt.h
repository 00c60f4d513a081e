/*
 * ambptt — backpropagation through time under asynchronous multistage
 * checkpointing, on one AMD Instinct MI355X (gfx950).
 *
 * Kukreja, Hückelheim, Gorman, "Backpropagation for long sequences: beyond
 * memory constraints with constant overheads" (arXiv 1806.01117).
 *
 * The library drives one whole forward + reverse pass over n recurrent steps
 * (Section 4: the driver calls the forward and backward operators as the
 * schedule directs).  Level 1 is a pool of s fast checkpoint slots in HBM;
 * Level 2 is pinned host DRAM (Section 2: only the relative speed and size of
 * the two levels matter).  Every I-th state is copied to Level 2 on a
 * dedicated copy stream while the forward sweep continues, and is prefetched
 * back one interval before the reverse sweep needs it; Revolve schedules the
 * recomputation inside each interval (Section 2, Fig. 2).  The interval is
 * I = ceil(T_T / T_A) (Section 3), raised if needed so the stored states fit
 * the Level-2 budget; with no Level 2, or when the two-level schedule would
 * not recompute strictly less, plain Revolve is used (Section 3, fallback).
 *
 * Conventions for every call below
 *   - Device pointers are HIP device addresses; the caller owns all device
 *     memory (inputs, parameters, gradients, the slot pool and the
 *     workspace).  The library never allocates device memory.
 *   - The library owns the pinned host tier (allocated with hipHostMalloc
 *     when a schedule first needs it), one copy stream and its events.
 *   - Every call returns a status; nothing throws across this boundary.  On
 *     failure ambptt_last_error() returns a message for the calling thread.
 *     After AMBPTT_EHIP the context must be destroyed.
 *   - Row-major layouts.  Batch rows first: a state h is [B][H].
 *   - Operand dtype (AMBPTT_F32 or AMBPTT_BF16) applies to x, W and the
 *     stored hidden state h; biases, the LSTM cell state c, every gradient
 *     and all accumulation are fp32.
 */
#ifndef AMBPTT_H
#define AMBPTT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  AMBPTT_OK = 0,
  AMBPTT_EINVAL = -1,       /* bad argument or size; nothing was enqueued */
  AMBPTT_ENOMEM = -2,       /* pinned host allocation failed; nothing leaked */
  AMBPTT_EHIP = -3,         /* a HIP runtime call failed; context unusable */
  AMBPTT_EUNSUPPORTED = -4, /* valid but not implemented (e.g. a shape constraint) */
  AMBPTT_EINTERNAL = -5     /* schedule / executor invariant broken */
} ambptt_status;

/* Recurrent cells: the per-step forward operator and its adjoint. */
enum {
  AMBPTT_CELL_TANH_RNN = 1, /* h' = tanh(W [x|h] + b), W[H][D+H] */
  AMBPTT_CELL_LSTM = 2,     /* z = W [x|h] + b, W[4H][D+H], gate blocks i,f,g,o;
                               c' = s(f) c + s(i) tanh(g); h' = s(o) tanh(c') */
  AMBPTT_CELL_RESMLP = 3,   /* depth as sequence: y' = y + relu(W_l y + b_l),
                               W[L][w][w] (output x input), b[L][w]; D = 0 */
  AMBPTT_CELL_MLP = 4       /* depth as sequence with layers of different
                               widths, states of different sizes (Sections 1.1
                               and 6): y_{l+1} = relu(W_l y_l + b_l),
                               W_l [w_{l+1}][w_l] and b_l [w_{l+1}] stored one
                               layer after the other; widths from
                               ambptt_set_widths (all = hidden by default,
                               hidden = the largest); D = 0; fp32 only */
};

enum { AMBPTT_F32 = 0, AMBPTT_BF16 = 1 };

enum {
  AMBPTT_LOSS_HALF_SQ_LAST = 0, /* L = 1/2 sum(h_n^2) */
  AMBPTT_LOSS_MEAN_SQ_ALL = 1,  /* L = sum_{t=1..n} mean(h_t^2) */
  AMBPTT_LOSS_MEAN_LAST = 2     /* L = mean(h_n) */
};

/* The problem as the paper states it (Sections 3-4): n steps, the state
 * described by the cell and its sizes, s fast slots, a slow-storage budget. */
typedef struct {
  int32_t cell;          /* AMBPTT_CELL_* */
  int32_t dtype;         /* AMBPTT_F32 | AMBPTT_BF16 */
  int32_t loss;          /* AMBPTT_LOSS_* */
  int32_t batch;         /* B >= 1 */
  int32_t input;         /* D >= 0, multiple of 16 (0 for RESMLP) */
  int32_t hidden;        /* H (or MLP width) >= 16, multiple of 16 */
  int64_t n_steps;       /* n >= 1 (layers L for RESMLP) */
  int32_t fast_slots;    /* s >= 1 HBM checkpoint slots (the first state's included) */
  int32_t interval_min;  /* I_min >= 1, or 0 to measure it (ambptt_calibrate) */
  int64_t slow_slots;    /* host slots H >= 0; 0 = single-stage Revolve */
} ambptt_problem;

/* Counters of one ambptt_run.  recompute_factor = forward_evals / n, where a
 * forward evaluation is one forward step (advances plus the first turn's). */
typedef struct {
  int32_t mode;            /* 0 = Revolve, 1 = asynchronous two-level, 2 = two-level with
                              stores decided during the sweep ("store_policy" 1),
                              3 = online checkpointing ("online" 1) */
  int32_t interval;        /* I (0 in Revolve mode; in mode 2 the longest interval;
                              in mode 3 the first interval, 0 in one level) */
  int32_t window;          /* steps per dW accumulation window (0: resident kernel) */
  int32_t path;            /* 0 = one launch per step, 1 = resident whole-pass kernel */
  int64_t n_steps;
  int64_t actions;
  int64_t forward_evals;
  int64_t adjoints;
  int64_t takeshots, takeshot_copies, restores;
  int64_t stores, prefetches, prefetches_elided;
  int64_t bytes_d2h, bytes_h2d;
  int64_t compute_waits;   /* compute-stream waits on the copy stream */
  int64_t kernel_launches;
  double recompute_factor;
  double schedule_us;      /* host time to build the schedule */
  double run_us;           /* host wall time of the forward + reverse pass */
  double enqueue_us;       /* host time spent enqueueing it (run_us minus the final wait) */
  /* average device time of sampled launches per kernel class (0 if sampling
   * is off): AMBPTT_K_* below */
  double kernel_us[6];
  int64_t kernel_samples[6];
  int64_t kernel_calls[6];
  int64_t bytes_file_w, bytes_file_r;  /* file tier traffic (ambptt_set_file_tier) */
  double forward_cost;     /* sum of the step costs of every forward evaluation
                              (ambptt_set_step_costs; without costs = forward_evals) */
} ambptt_stats;

/* Kernel classes of ambptt_stats.kernel_*: forward step, the resident
 * whole-pass kernel, adjoint step (gate recomputation and cell adjoint), the
 * adjoint's own product launch on the wide-batch bf16 path and the fp32
 * large-batch path (hbar = zbar W_h, or the MLP's ybar + zbar W_{l+1}),
 * weight-gradient window, and everything
 * else. */
enum { AMBPTT_K_FWD = 0, AMBPTT_K_PASS = 1, AMBPTT_K_ADJ = 2, AMBPTT_K_HADJ = 3,
       AMBPTT_K_DW = 4, AMBPTT_K_OTHER = 5 };

typedef struct ambptt_ctx ambptt_ctx;

/* ---- pure host calls (no GPU needed) ------------------------------------ */

const char* ambptt_version(void);

/* Least number of advanced steps that reverses n steps with s slots
 * (binomial checkpointing of Griewank and Walther, behind the paper's
 * R(n, s) in Section 3): F(n, s) = r n - C(s + r, s + 1), where r is the
 * integer with C(s + r - 1, s) < n <= C(s + r, s).  Plain Revolve then runs
 * F(n, s) + 1 forward steps.  Returns < 0 on bad arguments. */
int64_t ambptt_revolve_advances(int64_t n, int32_t s);

/* Forward evaluations of the schedule the library would run for (n, s, H,
 * I_min); writes the chosen interval (0 = Revolve) and mode (0/1) when the
 * pointers are non-NULL.  Returns < 0 on bad arguments. */
int64_t ambptt_schedule_evals(int64_t n, int32_t s, int64_t H, int32_t interval_min,
                              int32_t* interval_out, int32_t* mode_out);

/* Canonical text of that schedule: a header line
 *   "ambptt-schedule v1 n=<n> s=<s> H=<H> I=<I|0> mode=<revolve|async>"
 * then one action per line: "A t0 t1" advance, "S k t" snapshot to slot k,
 * "R k t" restore from slot k, "F t" first turn, "Y t" adjoint step,
 * "W k h t" store slot k to host slot h, "P h k t" prefetch host h to slot k.
 * Writes at most cap bytes (NUL-terminated when it fits) and sets *needed to
 * the full length + 1.  EINVAL if cap is too small (buf untouched). */
ambptt_status ambptt_schedule_text(int64_t n, int32_t s, int64_t H, int32_t interval_min,
                                   char* buf, size_t cap, size_t* needed);

/* Canonical text of the two-level schedule over interval starts decided
 * during the forward sweep, the non-uniform policy that the paper's
 * conclusions (Section 6) propose: the next state is stored whenever the
 * previous transfer has completed.  starts[0..nstarts) must be 0 = t_0 <
 * t_1 < ... < t_{K-1} < n with K - 1 <= H, and s >= 2.  Interval k is
 * [t_k, t_{k+1}) (the last one [t_{K-1}, n)); the sweep stores t_0 .. t_{K-2}
 * to host slots 0 .. K-2 through fast slots k % 2, and the reverse prefetches
 * one interval ahead and reverses each interval with Revolve on s - 1 slots,
 * as in ambptt_schedule_text (header "I=0 mode=dynamic").  Buffer rules as
 * there; EINVAL on bad starts. */
ambptt_status ambptt_schedule_text_starts(int64_t n, int32_t s, int64_t H, const int64_t* starts,
                                          int64_t nstarts, char* buf, size_t cap, size_t* needed);

/* The schedule of ambptt_schedule_text_starts with every reversal split for
 * the step costs costs[0..n) (see ambptt_set_step_costs): what a pass runs
 * with store_policy 1 and step costs (Section 6's stores decided during the
 * sweep, with the dynamic program inside each interval).  The header ends
 * with " split=cost".  Buffer rules as in ambptt_schedule_text; EINVAL on bad
 * starts or costs, EUNSUPPORTED when a reversal's table would exceed 1 Mi
 * entries. */
ambptt_status ambptt_schedule_text_starts_costs(int64_t n, int32_t s, int64_t H, const int64_t* starts,
                                                int64_t nstarts, const double* costs, char* buf, size_t cap,
                                                size_t* needed);

/* Canonical text of the schedule of ambptt_schedule_text with every
 * reversal split for the step costs costs[0..n) (see ambptt_set_step_costs);
 * the header ends with " split=cost".  Buffer rules as in
 * ambptt_schedule_text; EINVAL on bad arguments or costs, EUNSUPPORTED when a
 * reversal's table would exceed 1 Mi entries (see ambptt_set_step_costs). */
ambptt_status ambptt_schedule_text_costs(int64_t n, int32_t s, int64_t H, int32_t interval_min,
                                         const double* costs, char* buf, size_t cap, size_t* needed);

/* Canonical text of the schedule when the states differ in size (the case
 * Sections 1.1 and 6 set beside Revolve's uniform states; Section 6 would
 * run a one-level method for unequal checkpoints inside each interval).  sizes[0..n] (>= 1) are the sizes of x_0 .. x_n in units of a
 * common granule; the fast pool holds s * max(sizes) units and the
 * snapshots stack in it: the one taken at recursion depth k ("slot" k, which
 * may exceed s - 1 when states are small) lies above the states in the slots
 * below it, and in two levels slots 0 and 1 are the interval starts'
 * regions of max(sizes) units each.  Every reversal of [a, a+l) with M units
 * free above x_a splits where a dynamic program over Revolve's recursion
 * with a budget finds the least total cost of recomputed steps,
 *   T(a, l, M) = min over m with sizes[a+m] <= M of
 *                C(a, a+m) + T(a+m, l-m, M - sizes[a+m]) + T(a, m, M),
 * ties to the largest m, the chain when no snapshot fits (C: the step costs,
 * costs[0..n) > 0, or 1 each when costs is NULL).  Plain: M = s max(sizes) -
 * sizes[0]; two levels (H > 0, s >= 2, I = max(I_min, 1, ceil(n / (H+1))) <
 * n), taken when strictly cheaper: M = (s - 2) max(sizes) in every interval.
 * Unit sizes give ambptt_schedule_text's schedule.  Header suffix
 * " split=size".  Buffer rules as in ambptt_schedule_text; EINVAL on bad
 * arguments, EUNSUPPORTED when a reversal's table would exceed 1 Mi entries
 * (l (l + 1) (M + 1)). */
ambptt_status ambptt_schedule_text_sized(int64_t n, int32_t s, int64_t H, int32_t interval_min,
                                         const int64_t* sizes, const double* costs, char* buf, size_t cap,
                                         size_t* needed);

/* The interval I_min for measured times of one forward step (T_A) and of one
 * state over the host link (T_T), in microseconds, with s fast slots.
 *   rule 0: the paper's (Section 3), the smallest I whose forward sweep
 *     hides one transfer: ceil(T_T / T_A).
 *   rule 1: among I = 1 .. ceil(T_T / T_A), the one with the least
 *     modelled time per step, (max(I T_A, T_T) + F(I, s - 1) T_A) / I: an
 *     interval of the sweep takes as long as its store when the link is the
 *     bottleneck, and its reverse recomputes F(I, s - 1) steps (ties: the
 *     smaller I).  With T_T <= T_A both give 1.
 * Pure host.  Returns -1 on bad arguments (T_A <= 0, T_T < 0, s < 1). */
int64_t ambptt_interval_from_timings(double t_a_us, double t_t_us, int32_t s, int32_t rule);

/* Canonical text of the online checkpointing schedule for n steps (header
 * "mode=online", I = the first interval, 0 in one level): the variant that
 * the paper names beside Revolve (Section 1.1), where the number of steps is
 * not known while the forward sweep runs.  Every decision about state x_t is
 * taken when x_t is computed, knowing only that step t exists; n shows
 * itself when x_{n-1} is reached, so every action before the sweep gets
 * there is the same for every longer n.
 *   H = 0 (or s = 1): one level.  States are held in the s fast slots by a
 *     placement that never advances a step more often than Revolve would
 *     (the least repetition number) and equals Revolve's count for
 *     n <= C(s + 2, 2); the held segments are reversed with Revolve.
 *   H > 0, s >= 2: two levels.  Every I-th state (I = max(I_min, 1)) goes
 *     to the lowest free host slot through fast slot 0 or 1; when a start
 *     finds no host slot free, I doubles and the stored starts that are not
 *     its multiples give theirs back.  Inside each interval the one-level
 *     placement runs on s - 1 slots; the reverse prefetches one interval
 *     ahead as in the fixed-interval policy.
 * Buffer rules as in ambptt_schedule_text; EINVAL on bad arguments. */
ambptt_status ambptt_schedule_text_online(int64_t n, int32_t s, int64_t H, int32_t interval_min,
                                          char* buf, size_t cap, size_t* needed);

/* The program the resident whole-pass kernel would run for the schedule of
 * (n, s, H, I_min) (flags bit 0: skip prefetches into a slot that already
 * holds their state; bit 1: the online schedule of
 * ambptt_schedule_text_online), 4 int32 per entry {op, y, z, w}:
 *   0 end (dL/dx_0, dW, loss)      1 forward step y, buffer z -> buffer w
 *   2 adjoint step y from buffer z (w = 1: first turn)
 *   3 copy buffer z -> w, first waiting until every workgroup has read the
 *     inputs of barrier y (y = 0: no wait)
 *   4 store slot z to host slot w  5 prefetch host slot z to slot w
 *   6 barrier only
 * Buffers 0..s-1 are the HBM slots, s and s+1 the two live buffers.  Ops 0,
 * 1, 2 and 6 are the barriers of the workgroups that share batch rows.
 * Writes at most cap entries and sets *entries to the full count.  EINVAL if
 * cap is too small (buf untouched) or on bad arguments.  Pure host. */
ambptt_status ambptt_resident_program(int64_t n, int32_t s, int64_t H, int32_t interval_min,
                                      int32_t flags, int32_t* buf, size_t cap, size_t* entries);

/* Sizes the caller allocates: bytes of one state (padded slot stride), of the
 * slot pool (fast_slots * stride) and of the workspace.  The slot pool is
 * Level 1 of Section 2 at exactly the s checkpoints of the problem statement
 * of Section 3 (the number of states that fit in fast memory at once); the
 * state is what one step passes to the next (Section 1.1: the checkpoint is
 * the state of a layer or timestep).  Pure host: EINVAL / EUNSUPPORTED as for
 * ambptt_create; out pointers may be NULL. */
ambptt_status ambptt_query(const ambptt_problem* p, size_t* state_bytes,
                           size_t* slot_pool_bytes, size_t* workspace_bytes);

const char* ambptt_last_error(void);

/* ---- GPU calls ----------------------------------------------------------- */

/* Validates p, creates the copy stream and events on the current device.
 * stream is the compute stream (hipStream_t; NULL = the null stream).
 * Section 2: the compute stream runs the forward and adjoint operators while
 * a second, owned stream moves states between Level 1 and Level 2, so that
 * transfers run beside the computation.  *out is owned by the caller and
 * released with ambptt_destroy; on failure *out is untouched and nothing is
 * leaked.  EINVAL for a bad problem, EHIP if a stream or event cannot be
 * made, EUNSUPPORTED for shapes the kernels do not take. */
ambptt_status ambptt_create(const ambptt_problem* p, void* stream, ambptt_ctx** out);

/* Binds caller-owned device memory: the slot pool and the workspace, at
 * least the sizes ambptt_query reports, 256-byte aligned.  The slot pool is
 * the fixed fast-memory budget of Section 3 (s checkpoints); the library
 * keeps the pointers (it does not copy or free them) until the next bind or
 * ambptt_destroy.  The workspace may be NULL (any size): then only
 * ambptt_run_noalloc runs passes, and ambptt_run and ambptt_calibrate fail
 * with EINVAL.  EINVAL if the pool is NULL, or a pointer is misaligned or its
 * buffer too small. */
ambptt_status ambptt_bind(ambptt_ctx* ctx, void* slot_pool, size_t pool_bytes,
                          void* workspace, size_t workspace_bytes);

/* Sets a tuning / debug knob.  Keys: "timing_sample" (time every k-th
 * kernel launch with events, 0 = off), "elide_prefetch" (0/1, default 1),
 * "window" (dW window steps, 0 = automatic), "path" (0 = the resident
 * whole-pass kernel when the problem and device allow it, else one launch
 * per step; 1 = one launch per step; 2 = resident, EUNSUPPORTED at run time
 * if it does not fit), "resident_timeout_ms" (how long one barrier wait of the
 * resident kernel may take before the pass aborts with EINTERNAL; default
 * 2000), "resident_cooperative" (1, default: hipLaunchCooperativeKernel,
 * whose runtime guarantees that the whole grid is resident; 0: a plain
 * launch, about 0.5 % faster on the 512-LSTM, which the device holds at once
 * only when nothing else occupies it, else the pass ends in the barrier
 * timeout), "resident_test_stall" (1: the resident program starts with a wait
 * that is never satisfied, so the pass ends in that timeout; for tests of the
 * abort path), "wide_batch" (1, default: batches of 48 rows and more in bf16
 * run the wide-batch kernels; 0: the small-batch kernels), "dw_stream" (1:
 * weight-gradient windows run on a stream of their own, beside the steps; 0:
 * on the compute stream, after the window's last adjoint; -1, default: 0 on
 * the wide-batch bf16 path and the large-batch fp32 path, whose kernels each
 * fill the device, and for the MLP of layers of different widths, else 1),
 * "event_system_fence" (0, default: the events that order the library's
 * streams and time its kernels use device-scope fences; 1: system-scope, as
 * HIP's default events do), "store_policy" (0, default: the sweep stores
 * every I-th state; 1: it stores the next state once the previous store has
 * completed, at least ceil(n / (H + 1)) steps apart, the non-uniform policy
 * of Section 6; where the fixed-interval policy would use the host tier, on
 * the per-step path only: EUNSUPPORTED with "path" 2; stats mode 2 and
 * ambptt_last_schedule_text give the schedule that ran), "online" (0,
 * default; 1: online checkpointing, the schedule of
 * ambptt_schedule_text_online with the context's I_min, on either path;
 * stats mode 3; EINVAL together with "store_policy" 1, EUNSUPPORTED over a
 * file tier), "interval_rule" (1, default: ambptt_calibrate picks the
 * interval with the least modelled time per step; 0: ceil(T_T / T_A), see
 * ambptt_interval_from_timings), "test_copy_delay_us" (tests of the stream
 * ordering, per-step path: a host function that holds the copy stream this
 * many microseconds, at most 100000, before every store and prefetch, and
 * the weight-gradient stream before every window on it, so that the waits
 * of compute on them are taken; 0 by default), "test_poison" (1: a prefetch
 * first fills its fast slot with NaN bytes on the copy stream, so that
 * compute reading the slot before the prefetch has landed spoils the
 * gradients), "uniform_sizes" (states of different sizes: 1 plans the
 * schedule as if every state had the size of the largest, i.e. slots of the
 * largest size in the same byte budget, for comparison with the sized
 * schedule; 0 by default), "lds_gemm" (fp32 path for large batches: 1, default, runs the gate
 * product with its cell epilogue and the h-adjoint product on LDS-tiled
 * kernels (128 x 128 and 64 x 64 tiles, two workgroups per CU) where they
 * have at least 256 tiles; 2 wherever their shape constraints hold; 0 never:
 * the direct-load kernels), "hadj_launch" (1,
 * default: on the fp32 path for large batches the adjoint's h-adjoint
 * product zbar_{t+1} W_h runs as a launch of its own, kernel class
 * AMBPTT_K_HADJ; 0: fused into the adjoint step's launch), "prod_split" (1,
 * default: where both LDS-tiled kernels run and the 64 x 64 tiles would move
 * twice the operand rows per MFMA, that launch uses 128 x 128 tiles with the
 * reduction split in up to 4 parts, which the adjoint adds in order; 0: the
 * 64 x 64 tiles), "reserve" (1: allocate now the pinned host
 * tier and resident-program staging that the current schedule needs, with
 * the interval I_min, or 1 before calibration, which takes the most host
 * slots; see ambptt_run_noalloc), "host_waits"
 * (when compute must wait for a host-tier copy still in flight: 1 the host
 * waits before enqueueing the dependent work, 0 a stream wait on the compute
 * stream; -1, default: 1 on the wide-batch bf16 and large-batch fp32 paths,
 * whose queued kernels keep the device busy while the host waits, else 0).
 * EINVAL for unknown keys or values out of range. */
ambptt_status ambptt_set_int(ambptt_ctx* ctx, const char* key, int64_t value);

/* Puts a file below the pinned host tier: a third storage level for states
 * that do not fit in pinned host memory (the paper's platforms store to DRAM
 * or SSD, Section 5).  The schedule then has file_slots slow slots; the
 * problem's slow_slots pinned buffers (>= 1) become a ring in front of the
 * file: slot h is stored through buffer h % slow_slots and written behind to
 * the file by a host I/O thread; in the reverse, which takes the slots in
 * decreasing order, slot h - slow_slots is read back into the buffer as soon
 * as slot h has left it.  The file is created in `dir` and removed from it at
 * once (it lives until the tier is replaced or the context destroyed).
 * file_slots = 0 removes the tier.  Per-step path only (EUNSUPPORTED with
 * "path" 2; "path" 0 then runs per step).  ambptt_calibrate takes the file's
 * write time per state into T_T.  EINVAL if the file cannot be created. */
ambptt_status ambptt_set_file_tier(ambptt_ctx* ctx, const char* dir, int64_t file_slots);

/* Layer widths w_0 .. w_n of an AMBPTT_CELL_MLP problem (count = n + 1):
 * multiples of 16 from 16 up to the problem's hidden size, which one of them
 * must equal.  State x_t is y_t [B][w_t] (fp32); the slot pool of
 * fast_slots states of the largest size is then byte-addressed and every
 * schedule is the sized one of ambptt_schedule_text_sized, with the sizes of
 * the states (rounded up to 256 bytes) in units of their greatest common
 * divisor: small states stack more snapshots into the same HBM budget, and
 * with stores decided during the sweep ("store_policy" 1) every interval is
 * reversed by the same sized recursion, the pairing Section 6 proposes.
 * Online checkpointing is not available for it (EUNSUPPORTED at run time).
 * EINVAL for another cell, a wrong count or width. */
ambptt_status ambptt_set_widths(ambptt_ctx* ctx, const int32_t* widths, int64_t count);

/* Relative forward costs of the n steps (costs[t] > 0 for step t; NULL or
 * n = 0 removes them): layers or steps of unequal cost, which the paper's
 * Sections 1.1 and 6 point to.  Every reversal of two or more steps on two
 * or more fast slots is then split where a dynamic program over Revolve's
 * recursion finds the least total cost of recomputed forward steps
 * (ambptt_schedule_text_costs); the mode, interval and slots stay those of
 * the uniform schedule, and equal costs give it exactly.  The costs are
 * copied; with "store_policy" 1 the reversals of the intervals the sweep
 * chose are split for them too.  EINVAL if n differs from the problem's, a
 * cost is not positive and finite, or "online" is set.  The dynamic program
 * of a reversal of l steps on k slots keeps l (l + 1) (k + 1) entries and
 * takes about l^3 k / 6 operations; a pass whose schedule holds a reversal
 * over 1 Mi entries (single-level Revolve over ~300 steps with 10 slots;
 * in the two-level policy the intervals are the reversals) fails in
 * ambptt_run with EUNSUPPORTED. */
ambptt_status ambptt_set_step_costs(ambptt_ctx* ctx, const double* costs, int64_t n);

/* Measures T_A (one forward step) and T_T (one state over the host link,
 * the slower direction) and sets the context's I_min from them with the
 * context's "interval_rule" (ambptt_interval_from_timings; on the resident
 * kernel rule 0 lets a transfer lengthen a step by 5 % before counting it).
 * Uses the same inputs as ambptt_run; writes nothing the caller owns.  Any
 * out pointer may be NULL. */
ambptt_status ambptt_calibrate(ambptt_ctx* ctx, const void* x_seq, const void* W,
                               const float* b, const void* h0, const float* c0,
                               int32_t* interval_min_out, double* t_a_us, double* t_t_us);

/* One forward + reverse pass (blocks until the compute stream is done):
 * Section 4's driver, which runs the forward and backward operators as the
 * schedule directs and returns the parameter and initial-state gradients;
 * the schedule is the two-level one of Sections 2-3 (or plain Revolve).
 * Fails with EINVAL before enqueueing anything if a pointer is NULL (other
 * than those marked optional) or nothing is bound; with EHIP if a HIP call
 * fails (the context is then unusable); with EINTERNAL if an executor
 * invariant breaks (a resident-kernel barrier timed out), after which the
 * context stays usable.
 *   x_seq  [n][B][D] operand dtype (NULL for RESMLP)
 *   W      TANH_RNN/LSTM: [G*H][D+H]; RESMLP: [L][w][w]; MLP: the layers'
 *          [w_{l+1}][w_l] one after the other; operand dtype
 *   b      fp32 [G*H] (RESMLP: [L][w]; MLP: the layers' [w_{l+1}])
 *   h0     [B][H] operand dtype (MLP: [B][w_0]); c0 fp32 [B][H] for LSTM, else NULL
 *   dW, db fp32, same layouts as W, b (overwritten)
 *   dh0    fp32 [B][H] (MLP: [B][w_0]); dc0 fp32 [B][H] for LSTM, else NULL
 *   loss   host double (may be NULL); stats host (may be NULL)
 * The inputs must not be written while the call runs. */
ambptt_status ambptt_run(ambptt_ctx* ctx, const void* x_seq, const void* W, const float* b,
                         const void* h0, const float* c0, float* dW, float* db,
                         float* dh0, float* dc0, double* loss, ambptt_stats* stats);

/* ambptt_run without allocation, for callers that cannot allocate memory
 * while they run: code under HIP graph capture, tight serving loops, hosts
 * that forbid hipMalloc.  The same pass, kernels and results as ambptt_run on
 * the same context, but the workspace is the library's own static device
 * array of 64 MiB (one per GPU, held until the process ends) instead of the
 * bound one; the bound slot pool, the inputs and the outputs are the
 * caller's as there.  It calls no hipMalloc, hipHostMalloc, hipFree or other
 * allocating HIP or torch routine (the schedule is built on the host heap,
 * as in ambptt_run), takes no timing samples beyond events already created,
 * and therefore refuses, with EINVAL and nothing enqueued, what would need an
 * allocation:
 *   - a workspace (ambptt_query) larger than 64 MiB;
 *   - a host-tier schedule before its interval is known (ambptt_calibrate,
 *     or "interval_min" set);
 *   - a pinned host tier or resident-program staging buffer that the pass
 *     needs and that is not yet allocated: ambptt_set_int(ctx, "reserve", 1)
 *     allocates them for the current schedule (an earlier ambptt_run of the
 *     same schedule leaves them allocated too);
 *   - a file tier (EUNSUPPORTED).
 * Every call on one GPU shares the scratch array and leaves its contents
 * behind; the pass clears what must start at zero.  Calls that overlap on
 * one GPU (two threads, or two streams in flight) race on it: serialise them. */
ambptt_status ambptt_run_noalloc(ambptt_ctx* ctx, const void* x_seq, const void* W, const float* b,
                                 const void* h0, const float* c0, float* dW, float* db,
                                 float* dh0, float* dc0, double* loss, ambptt_stats* stats);

/* Canonical text (as ambptt_schedule_text) of the schedule the last
 * ambptt_run on this context executed; with "store_policy" 1 it holds the
 * interval starts the sweep chose.  Buffer rules as there; EINVAL before the
 * first pass.  Host only. */
ambptt_status ambptt_last_schedule_text(ambptt_ctx* ctx, char* buf, size_t cap, size_t* needed);

/* Frees the host tier, the copy stream and events.  NULL-safe. */
void ambptt_destroy(ambptt_ctx* ctx);

#ifdef __cplusplus
}
#endif

#endif /* AMBPTT_H */
