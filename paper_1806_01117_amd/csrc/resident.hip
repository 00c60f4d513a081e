// Resident whole-pass kernel for small recurrent states (fp32 tanh RNN and
// LSTM, gfx950).
//
// For a batch of 64 and hidden size 512 one step is a 64 x 2048 x 768 GEMM:
// 1.3 us of MFMA work for the whole chip, while a launch per step pays the
// launch itself plus a fresh fetch of W (6.3 MB) into every CU, because L2 is
// invalidated between kernels.  Here one cooperative launch runs the whole
// forward + reverse pass, as a program of actions compiled on the host from
// the checkpoint schedule, and every workgroup keeps its slice of the weights
// in registers for the whole pass.
//
// Decomposition.  Workgroup (mt, ug) owns batch rows 16 mt .. 16 mt + 15 and
// hidden units U ug .. U ug + U - 1 (U = 8 for the LSTM, i.e. 32 gate
// columns; 16 for the RNN): the gate rows of W for those units, the rows of
// the weight gradient, and the (row, unit) slice of every state (h and c).
// The ng = H / U workgroups of one row tile form a group: a step needs the
// whole h_t of its 16 rows, so the members exchange h through HBM and meet at
// a flag barrier once per step.  Rows are independent, so groups never wait
// for each other.
//
// Coherence.  The L2 caches of the 8 XCDs are not coherent with each other.
// Everything that another workgroup reads (state slices, partial h-adjoints)
// is written and read with device-scope (sc1) buffer accesses, which bypass
// the non-coherent caches; a workgroup drains its stores (s_waitcnt) before
// it raises its progress flag, and readers load only after seeing the flag.
//
// Adjoint.  The adjoint of step t needs hbar = zbar_{t+1} W_h for its units.
// Instead of gathering all of zbar (16 x 4H per row tile) into every
// workgroup, each workgroup multiplies its own zbar columns by its own rows
// of W_h (held in registers) and writes a 16 x H partial; the owner of a
// unit then sums the ng partials of its units in a fixed order.  The weight
// gradient of the workgroup's gate rows over its 16 batch rows is
// accumulated in MFMA accumulators for the whole pass (the adjoint steps come
// in the order t = n-1 .. 0 under every schedule, so the sums are
// bit-identical across schedules) and summed over row tiles by a small
// kernel afterwards.
//
// Two-level checkpoints (Section 2).  Each workgroup moves its own 1 KiB
// slice of a state between an HBM slot and the pinned host tier, so the host
// tier needs no synchronisation between workgroups.  One wave issues those
// transfers: a store loads the slice at the action and writes it to host
// memory after the next barrier; a prefetch loads from host memory at the
// action and writes the slot after the next barrier, when every member has
// left the steps that read the slot's previous contents.  That wave does not
// stage step inputs, so the host link's latency delays only its own
// instructions, and only when the next step starts before the data arrived.
//
// Every wait is bounded: a workgroup that waits longer than the timeout sets
// a device-wide abort flag, and every other wait watches that flag, so the
// grid always drains.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "ambptt.h"
#include "kernels.hpp"
#include "mfma.hpp"

namespace ambptt {
namespace {

constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kCopyWave = kWaves - 1;        // issues the host-tier transfers
constexpr int kStageThreads = 64 * kCopyWave;  // waves that stage step inputs
constexpr int kKch = 6;                      // most 16-wide reduction chunks per wave: D + H <= 768
constexpr int kHmax = 512;                   // H <= 512
constexpr int kSmax = 8;                     // workgroups per octet (the first level of the h-adjoint sum)
constexpr int kUMmax = 64;                   // hidden units per octet member in that sum: H / S <= 64
constexpr int kKmax = 16 * kWaves * kKch;
constexpr int kXld = kKmax + 4;              // LDS row stride of the staged [x | h] rows
constexpr int kDev = 16;                     // sc1: coherent across the device
constexpr int kSys = 17;                     // sc0 sc1: system scope (host memory)

typedef unsigned int u4v __attribute__((ext_vector_type(4)));

// Every buffer this kernel addresses is the same for all lanes of a wave;
// readfirstlane states that, so the descriptor lives in scalar registers even
// where the compiler cannot prove it (otherwise it emits a loop over lanes).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base, unsigned bytes) {
  const unsigned long long p = (unsigned long long)base;
  const unsigned lo = __builtin_amdgcn_readfirstlane(unsigned(p)), hi = __builtin_amdgcn_readfirstlane(unsigned(p >> 32));
  void* ub = (void*)(((unsigned long long)hi << 32) | lo);
  return __builtin_amdgcn_make_buffer_rsrc(ub, 0, __builtin_amdgcn_readfirstlane(bytes), 0x00020000);
}
template <int AUX>
__device__ __forceinline__ f4 ld4(__amdgpu_buffer_rsrc_t r, unsigned off) {
  return __builtin_bit_cast(f4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, AUX));
}
template <int AUX>
__device__ __forceinline__ void st4(__amdgpu_buffer_rsrc_t r, unsigned off, f4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u4v, v), r, off, 0, AUX);
}
template <int AUX>
__device__ __forceinline__ float ld1(__amdgpu_buffer_rsrc_t r, unsigned off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, AUX));
}
template <int AUX>
__device__ __forceinline__ void st1(__amdgpu_buffer_rsrc_t r, unsigned off, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, v), r, off, 0, AUX);
}
__device__ __forceinline__ unsigned ld_flag(const unsigned* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_flag(unsigned* p, unsigned v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ f4 mma4(const f4& a, const f4& b, f4 c) {
  c = mfma_f32_16x16x4(a.x, b.x, c);
  c = mfma_f32_16x16x4(a.y, b.y, c);
  c = mfma_f32_16x16x4(a.z, b.z, c);
  return mfma_f32_16x16x4(a.w, b.w, c);
}

// Gate nonlinearities on the hardware exp2 and reciprocal (about 1 ulp each):
// sigma(z) = 1 / (1 + e^-z), tanh(z) = 2 sigma(2z) - 1.  Both saturate
// correctly for |z| -> inf (e^-z -> inf gives 0, -> 0 gives 1).
__device__ __forceinline__ float sigm(float z) { return __builtin_amdgcn_rcpf(1.0f + __expf(-z)); }
__device__ __forceinline__ float tanh_f(float z) { return 2.0f * sigm(2.0f * z) - 1.0f; }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// KCH: 16-wide reduction chunks per wave (the reduction is zero-padded to
// 8 KCH chunks, so no loop over chunks has a bound that varies by wave).
// Wave w holds chunks w, w + 8, w + 16, ...: every wave then has its share of
// the x columns and of the h columns, and the x part of a step's gate GEMM
// (which depends on no other workgroup) runs while the h_t rows are loaded.
template <int G, int KCH>
__global__ __launch_bounds__(kThreads) void resident_pass(ResidentArgs a) {
  constexpr int U = (G == 4) ? 8 : 16;
  constexpr int NC = G * U;            // gate columns of the workgroup (32 | 16)
  constexpr int NB = NC / 16;          // 16-column MFMA blocks of the gate GEMM
  constexpr int KW = NC / 16;          // 16-wide chunks of the partial product's reduction
  constexpr int NS = 16 * U;           // (row, unit) pairs of the slice (128 | 256)
  constexpr int NG4 = NS / 4;          // float4s of one slice of partial sums (32 | 64)
  constexpr int PER = U / 4;           // float4s per slice row
  constexpr int OK = kSmax * NC;       // gate columns of an octet (reduction of its partial product)
  constexpr int OLD = OK + 4;          // LDS row stride of the octet's zbar and of W_h^T

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = lane & 15, q = lane >> 4;
  const int B = a.B, D = a.D, H = a.H, K1 = D + H, GH = G * H;
  const int ng = a.ng, nwg = a.mtiles * a.ng;
  int mt, ug;
  if (a.xcd_map) {
    // ids are dealt to the 8 XCDs round-robin: a row tile takes 8 / mtiles
    // XCDs, and consecutive unit groups (so whole octets) share one
    const int per = 8 / a.mtiles, x = int(blockIdx.x % 8);
    mt = x / per;
    ug = (x % per) * (ng / per) + int(blockIdx.x / 8);
  } else {
    mt = int(blockIdx.x) / ng;
    ug = int(blockIdx.x) % ng;
  }
  const int me = mt * ng + ug;
  // octets: S consecutive unit groups of a row tile (S = min(8, ng))
  const int S = a.S, nO = ng / S, oc = ug / S, op_ = ug % S;
  const int UM = H / S;                 // units whose octet partial this workgroup forms
  const int ub0 = op_ * UM;
  const int m0 = 16 * mt, j0 = U * ug;
  const int nch = K1 / 16;
  const int nxc = D / 16;     // chunks of the x columns
  auto chunk = [&](int i) { return wave + kWaves * i; };  // slot i of this wave; chunks >= nch are zero
  const unsigned hbytes = unsigned(B) * unsigned(H) * 4u;
  const unsigned sbytes = G == 4 ? unsigned(a.c_off) + hbytes : hbytes;
  auto wrow = [&](int n) { return (n / U) * H + j0 + (n % U); };  // W row of gate column n
  auto buf = [&](int id) -> char* {
    return id < a.nslots ? a.pool + (size_t)id * a.stride : (id == a.nslots ? a.live0 : a.live1);
  };

  __shared__ __attribute__((aligned(16))) float xs[16][kXld];  // [x_t | h_t] rows of the tile
  __shared__ float zs[kWaves][16][NC + 1];                     // per-wave gate partial sums
  __shared__ __attribute__((aligned(16))) float zb[16][NC + 4];  // zbar_t of the workgroup
  __shared__ float hp[kSmax][NS];                              // octet partials of the slice's h-adjoint
  __shared__ float cbs[NS];                                    // cbar carried between adjoints
  __shared__ __attribute__((aligned(16))) float zbo[16][OLD];   // zbar of the octet's gate columns
  __shared__ __attribute__((aligned(16))) float whs[kUMmax * OLD];  // W_h^T: octet's columns x own units
  __shared__ __attribute__((aligned(16))) float stg[2 * NS];  // the last forward step's output slice (h, c)
  __shared__ double wsum[kWaves];
  __shared__ int stop;

  // ---- weights into registers ---------------------------------------------
  f4 Wr[KCH][NB];  // B operands of the gate GEMM: W[col][16 ch + 4 q + e]
#pragma unroll
  for (int i = 0; i < KCH; ++i) {
    const int ch = chunk(i);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
      Wr[i][nb] = ch < nch ? *(const f4*)(a.W + (size_t)wrow(nb * 16 + r) * K1 + ch * 16 + 4 * q)
                           : f4{0.f, 0.f, 0.f, 0.f};
  }
  // W_h^T for the octet's partial product (its B operand): whs[u][k] =
  // W[row of octet column k][D + ub0 + u], k = m NC + n for member m's gate
  // column n, so that a lane's four reduction indices are one 16-byte read.
  // Columns of absent members and units beyond UM stay zero, as do the
  // octet-zbar columns beyond S NC.
  for (int idx = tid; idx < kUMmax * OK; idx += kThreads) {
    const int u = idx / OK, k = idx % OK, m = k / NC, n = k % NC;
    float v = 0.f;
    if (u < UM && m < S) v = a.W[(size_t)((n / U) * H + U * (oc * S + m) + n % U) * K1 + D + ub0 + u];
    whs[u * OLD + k] = v;
  }
  for (int idx = tid; idx < 16 * OLD; idx += kThreads) zbo[idx / OLD][idx % OLD] = 0.f;
  // reduction columns K1 .. 16 * 8 KCH of the staged rows stay zero
  for (int idx = tid; idx < 16 * (16 * kWaves * KCH - K1); idx += kThreads) {
    const int w = 16 * kWaves * KCH - K1;
    xs[idx / w][K1 + idx % w] = 0.f;
  }
  f4 dacc[KCH][NB];  // dW blocks (gate block nb, reduction chunk chunk(i))
#pragma unroll
  for (int i = 0; i < KCH; ++i)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) dacc[i][nb] = f4{0.f, 0.f, 0.f, 0.f};
  float dbacc = 0.f;
  double lacc = 0.0;  // loss terms of this thread's (row, unit), summed over the adjoint steps in order

  // epilogue thread (ml, u) of the slice
  const bool epi = tid < NS;
  const int ml = tid / U, u = tid % U;
  const int em = m0 + ml, ej = j0 + u;
  const bool erow = epi && em < B;
  const unsigned eoff = unsigned(em * H + ej) * 4u;
  float bias[G];
#pragma unroll
  for (int g = 0; g < G; ++g) bias[g] = erow ? a.bias[g * H + ej] : 0.f;
  if (epi) cbs[tid] = 0.f;

  // copy-wave lane -> 16 bytes of the slice (h part, then c part)
  const int cl_i = lane < 16 * PER ? lane : lane - 16 * PER;
  const bool cl_h = lane < 16 * PER;
  const bool cl_c = (G == 4) && !cl_h && lane < 32 * PER;
  const int cl_row = cl_i / PER;
  const bool cl_ok = wave == kCopyWave && (cl_h || cl_c) && m0 + cl_row < B;
  const unsigned cl_off = unsigned(((m0 + cl_row) * H + j0 + 4 * (cl_i % PER)) * 4) + (cl_c ? unsigned(a.c_off) : 0u);
  auto host_rsrc = [&](int hslot) { return rsrc(a.host + ((size_t)hslot * nwg + me) * 1024, 1024); };

  if (tid == 0) stop = 0;
  __syncthreads();

  unsigned sc = 0;     // group barriers passed
  int na = 0;          // adjoint steps done
  int pend_pref = -1;  // slot of the prefetch whose data the copy wave holds
  int pref_next = -1;  // program entry of the next prefetch (its host read may start early)
  int early_pc = -1;   // entry whose host read was started at the last prefetch's landing
  bool pcie_st = false;  // host-tier stores issued since the copy wave last waited
  bool early_after_st = false;  // an early host read was issued after the slot store being drained
  int pend_store = -1; // host slot of the store whose data the copy wave holds
  bool dirty = false;  // the copy wave wrote a slot since its last drain
  f4 pv = f4{0.f, 0.f, 0.f, 0.f}, sv = f4{0.f, 0.f, 0.f, 0.f};
  int pc = 0;
  // the program is read-only for the whole launch: reading it through the
  // constant address space makes every entry a scalar load, which no wave
  // waits for behind its own vector memory traffic (host-link reads and
  // writes of the copy wave in particular)
  const __attribute__((address_space(4))) int* prog = (const __attribute__((address_space(4))) int*)a.prog;

  // all stores of this workgroup that others may read are complete
  auto drain = [&]() {
    if (wave != kCopyWave) {
      __builtin_amdgcn_s_waitcnt(0);
    } else if (dirty) {
      // the slot store issued by the last flush must land; an early host read
      // issued after it may stay in flight (vector memory counts retire in order)
      if (early_after_st) __builtin_amdgcn_s_waitcnt(0x0F71);  // vmcnt(1)
      else __builtin_amdgcn_s_waitcnt(0x0F70);                 // vmcnt(0)
      pcie_st = pcie_st && early_after_st;
    }
    dirty = false;
    early_after_st = false;
    __syncthreads();
  };
  // copy wave: host read of the slice of host slot h into pv.  The data are
  // first used by the slot store at the next flush, so the read stays in
  // flight across everything the wave does until then.
  auto host_read = [&](int h) {
    if (pcie_st) {  // a store to the host tier may target the same slot: let it land first
      __builtin_amdgcn_s_waitcnt(0x0F70);
      pcie_st = false;
    }
    if (cl_ok) pv = ld4<kSys>(host_rsrc(h), unsigned(lane) * 16u);
  };
  // wave 0 waits until flags[0 .. cnt) all reach target
  auto wait_flags = [&](const unsigned* flags, int cnt, unsigned target) -> bool {
    if (wave == 0) {
      const unsigned long long t0 = __builtin_amdgcn_s_memrealtime();
      int st = 0;
      for (unsigned it = 0;; ++it) {
        bool ok = true;
        for (int j = lane; j < cnt; j += 64) ok = ok && ld_flag(flags + j) >= target;
        if (__all(ok)) break;
        if ((it & 31) == 31) {
          if (ld_flag(a.status) != 0u) {
            st = 1;
            break;
          }
          if ((long long)(__builtin_amdgcn_s_memrealtime() - t0) > a.timeout) {
            st = 2;
            break;
          }
        }
        __builtin_amdgcn_s_sleep(1);
      }
      if (lane == 0) {
        if (st == 2) {
          st_flag(a.status + 1, unsigned(pc + 1));
          st_flag(a.status, 1u);
        }
        stop = st;
      }
    }
    __syncthreads();
    return stop == 0;
  };
  auto wait_group = [&](const unsigned* flags, unsigned target) -> bool {
    return wait_flags(flags + mt * ng, ng, target);
  };
  // the nO octet partials of this workgroup's units from the last adjoint
  // step, P[octet][unit][row] -> hp[octet][u 16 + row] (staging threads)
  auto stage_partials = [&]() {
    const float* pin = a.P + (((size_t)((na + 1) & 1) * a.mtiles + mt) * nO) * H * 16;
    const __amdgpu_buffer_rsrc_t prs = rsrc(pin, unsigned(nO * H * 16 * 4));
    for (int idx = tid; idx < nO * NG4; idx += kStageThreads) {
      const int o2 = idx / NG4, v4 = idx % NG4;
      *(f4*)&hp[o2][4 * v4] = ld4<kDev>(prs, unsigned(((o2 * H + j0) * 16 + 4 * v4) * 4));
    }
  };
  // weight gradient of the workgroup's gate rows for the last adjoint step,
  // dW += zbar^T [x | h], on the wave's own reduction chunks (block (nb,
  // chunk chunk(i)) of 16 x 16).  It feeds nothing the other workgroups wait
  // for, so it runs after this workgroup has raised its flag for the next
  // barrier, while the flags of the others are on their way.
  bool pend_dw = false;
  auto deferred_dw = [&]() {
    // operands of batch rows 4 c4 + q, read one group ahead of the MFMAs
    float av[2][NB], bv[2][KCH];
    auto load = [&](int c4, int buf_) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) av[buf_][nb] = zb[4 * c4 + q][nb * 16 + r];
#pragma unroll
      for (int i = 0; i < KCH; ++i) bv[buf_][i] = xs[4 * c4 + q][chunk(i) * 16 + r];
    };
    load(0, 0);
#pragma unroll
    for (int c4 = 0; c4 < 4; ++c4) {
      if (c4 < 3) load(c4 + 1, (c4 + 1) & 1);
      __builtin_amdgcn_sched_barrier(0);  // keep the reads ahead of the MFMAs that hide them
#pragma unroll
      for (int i = 0; i < KCH; ++i)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          dacc[i][nb] = mfma_f32_16x16x4(av[c4 & 1][nb], bv[c4 & 1][i], dacc[i][nb]);
    }
    if (tid < NC) {
      float s = 0.f;
#pragma unroll
      for (int row = 0; row < 16; ++row) s += zb[row][tid];
      dbacc += s;
    }
    pend_dw = false;
  };
  // group barrier number sc + 1, in two halves (the caller drained first)
  auto raise = [&]() {
    if (tid == 0) st_flag(a.ready + me, sc + 1);
    if (pend_dw) {
      deferred_dw();
      __syncthreads();  // its reads of the staged rows come before new rows are staged
    }
  };
  auto enter = [&]() -> bool {
    if (!wait_group(a.ready, sc + 1)) return false;
    ++sc;
    return true;
  };
  auto flush = [&]() {  // complete the held transfers (after a barrier; the copy wave's lanes move data)
    if (pend_pref >= 0) {
      if (cl_ok) st4<kDev>(rsrc(buf(pend_pref), sbytes), cl_off, pv);
      dirty = true;
      pend_pref = -1;
      if (pref_next >= 0) {  // start the next prefetch's host read now (pv is free again)
        if (wave == kCopyWave) host_read(prog[4 * pref_next + 2]);
        early_pc = pref_next;
        early_after_st = true;
        pref_next = -1;
      }
    }
    if (pend_store >= 0) {
      if (cl_ok) st4<kSys>(host_rsrc(pend_store), unsigned(lane) * 16u, sv);
      pcie_st = true;
      pend_store = -1;
    }
  };
  auto abort_op = [&](unsigned code) {
    if (tid == 0) {
      st_flag(a.status + 1, unsigned(pc + 1) | (code << 24));
      st_flag(a.status, 1u);
    }
  };

  // one forward (adj = false) or adjoint step t from buffer src
  auto step = [&](int t, int src, int dst, bool adj, bool first) -> bool {
    drain();
    raise();
    const char* sb = buf(src);
    const __amdgpu_buffer_rsrc_t srs = rsrc(sb, sbytes);
    // inputs that do not depend on the other members, staged while wave 0
    // polls: x_t rows (waves 1 .. 6) and the own c_t (epilogue threads)
    if (wave > 0 && wave < kCopyWave) {
      const int nx4 = 4 * D;  // float4s of 16 rows of x
      for (int idx = tid - 64; idx < nx4; idx += kStageThreads - 64) {
        const int row = idx / (D / 4), col = 4 * (idx % (D / 4));
        f4 v = f4{0.f, 0.f, 0.f, 0.f};
        if (m0 + row < B) v = *(const f4*)(a.x + ((size_t)t * B + m0 + row) * D + col);
        *(f4*)&xs[row][col] = v;
      }
    }
    float cold = 0.f;
    if (G == 4 && erow) cold = ld1<kDev>(srs, unsigned(a.c_off) + eoff);
    f4 acc[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[nb] = f4{0.f, 0.f, 0.f, 0.f};
    auto gemm_part = [&](bool xpart) {
      f4 av[KCH];
#pragma unroll
      for (int i = 0; i < KCH; ++i) {
        const int ch = chunk(i);
        if (xpart ? ch < nxc : (ch >= nxc && ch < nch)) av[i] = *(const f4*)&xs[r][ch * 16 + 4 * q];
      }
#pragma unroll
      for (int i = 0; i < KCH; ++i) {
        const int ch = chunk(i);
        if (xpart ? ch < nxc : (ch >= nxc && ch < nch)) {
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) acc[nb] = mma4(av[i], Wr[i][nb], acc[nb]);
        }
      }
    };
    if (!enter()) return false;
    // stage h_t next to x_t (and, in an adjoint step, the octet partials of
    // step t + 1): the loads are issued first, the x part of the gate GEMM
    // z[16][NC] = [x|h] W^T runs while they travel, then they go to LDS
    constexpr int NHV = (4 * kHmax + kStageThreads - 1) / kStageThreads;
    f4 hv[NHV], qv[2];
    const int nh4 = 4 * H;
    if (tid < kStageThreads) {
#pragma unroll
      for (int j = 0; j < NHV; ++j) {
        const int idx = tid + j * kStageThreads, row = idx / (H / 4), col = 4 * (idx % (H / 4));
        hv[j] = f4{0.f, 0.f, 0.f, 0.f};
        if (idx < nh4 && m0 + row < B) hv[j] = ld4<kDev>(srs, unsigned(((m0 + row) * H + col) * 4));
      }
      if (adj && !first) {
        const float* pin = a.P + (((size_t)((na + 1) & 1) * a.mtiles + mt) * nO) * H * 16;
        const __amdgpu_buffer_rsrc_t prs = rsrc(pin, unsigned(nO * H * 16 * 4));
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int idx = tid + j * kStageThreads, o2 = idx / NG4, v4 = idx % NG4;
          if (idx < nO * NG4) qv[j] = ld4<kDev>(prs, unsigned(((o2 * H + j0) * 16 + 4 * v4) * 4));
        }
      }
    }
    gemm_part(true);
    if (tid < kStageThreads) {
#pragma unroll
      for (int j = 0; j < NHV; ++j) {
        const int idx = tid + j * kStageThreads, row = idx / (H / 4), col = 4 * (idx % (H / 4));
        if (idx < nh4) *(f4*)&xs[row][D + col] = hv[j];
      }
      if (adj && !first) {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int idx = tid + j * kStageThreads, o2 = idx / NG4, v4 = idx % NG4;
          if (idx < nO * NG4) *(f4*)&hp[o2][4 * v4] = qv[j];
        }
      }
    }
    __syncthreads();
    if (tid == 0) st_flag(a.consumed + me, sc);
    flush();

    // the h part of the gate GEMM
    gemm_part(false);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int v = 0; v < 4; ++v) zs[wave][4 * q + v][nb * 16 + r] = acc[nb][v];
    __syncthreads();

    float lterm = 0.f;
    if (epi) {
      float z[G];
#pragma unroll
      for (int g = 0; g < G; ++g) {
        float s = 0.f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) s += zs[w][ml][g * U + u];
        z[g] = s + bias[g];
      }
      float h1, c1 = 0.f, tc = 0.f, ig = 0.f, fg = 0.f, gg = 0.f, og = 0.f;
      if (G == 4) {
        ig = sigm(z[0]);
        fg = sigm(z[1 % G]);
        gg = tanh_f(z[2 % G]);
        og = sigm(z[3 % G]);
        c1 = fg * cold + ig * gg;
        tc = tanh_f(c1);
        h1 = og * tc;
      } else {
        h1 = tanh_f(z[0]);
      }
      if (!adj) {
        if (erow) {
          const __amdgpu_buffer_rsrc_t drs = rsrc(buf(dst), sbytes);
          st1<kDev>(drs, eoff, h1);
          if (G == 4) st1<kDev>(drs, unsigned(a.c_off) + eoff, c1);
        }
        stg[tid] = h1;  // host-slice order: h [16][U], then c [16][U]
        if (G == 4) stg[NS + tid] = c1;
      } else {
        float hbar = 0.f;
        if (!first) {
#pragma unroll
          for (int g = 0; g < kSmax; ++g)
            if (g < nO) hbar += hp[g][u * 16 + ml];
        }
        float sd = 0.f;
        if (a.loss == AMBPTT_LOSS_MEAN_SQ_ALL) {
          sd = 2.f * h1 * a.inv_bh;
          lterm = h1 * h1;
        } else if (first) {
          if (a.loss == AMBPTT_LOSS_HALF_SQ_LAST) {
            sd = h1;
            lterm = h1 * h1;
          } else {
            sd = a.inv_bh;
            lterm = h1;
          }
        }
        const float hb = hbar + sd;
        if (G == 4) {
          const float cb = first ? 0.f : cbs[tid];
          const float ob = hb * tc;
          const float ch = cb + hb * og * (1.f - tc * tc);
          zb[ml][u] = erow ? ch * gg * ig * (1.f - ig) : 0.f;
          zb[ml][U + u] = erow ? ch * cold * fg * (1.f - fg) : 0.f;
          zb[ml][2 * U + u] = erow ? ch * ig * (1.f - gg * gg) : 0.f;
          zb[ml][3 * U + u] = erow ? ob * og * (1.f - og) : 0.f;
          cbs[tid] = erow ? ch * fg : 0.f;
        } else {
          zb[ml][u] = erow ? hb * (1.f - h1 * h1) : 0.f;
        }
        if (!erow) lterm = 0.f;
        lacc += (double)lterm;
      }
    }
    if (!adj) return true;
    __syncthreads();
    // h-adjoint, first level: the octet's zbar columns times W_h for this
    // workgroup's share of units, summed at the owners at the next barrier
    {
      float* zout = a.Z + (((size_t)(na & 1) * a.mtiles + mt) * ng + ug) * (16 * NC);
      if (tid < 4 * NC) {  // 16 rows x NC columns
        const int row = tid / (NC / 4), c = 4 * (tid % (NC / 4));
        st4<kDev>(rsrc(zout, 16 * NC * 4), unsigned((row * NC + c) * 4), *(const f4*)&zb[row][c]);
      }
    }
    pend_dw = true;
    drain();
    if (tid == 0) st_flag(a.oflag + me, unsigned(na + 1));
    deferred_dw();  // while the octet's flags travel
    if (!wait_flags(a.oflag + mt * ng + oc * S, S, unsigned(na + 1))) return false;
    if (tid < kStageThreads) {
      const float* zin = a.Z + (((size_t)(na & 1) * a.mtiles + mt) * ng + oc * S) * (16 * NC);
      const __amdgpu_buffer_rsrc_t zrs = rsrc(zin, unsigned(S * 16 * NC * 4));
      for (int idx = tid; idx < S * 4 * NC; idx += kStageThreads) {
        const int m = idx / (4 * NC), w = idx % (4 * NC), row = w / (NC / 4), c = 4 * (w % (NC / 4));
        *(f4*)&zbo[row][m * NC + c] = ld4<kDev>(zrs, unsigned(idx * 16));
      }
    }
    __syncthreads();
    if (wave < 4) {  // one 16-unit block of the share per wave (UM <= 64)
      const int jb = wave;
      if (jb * 16 < UM) {
        // two accumulators over even and odd chunks, operands one pair ahead
        const float* wb = &whs[(jb * 16 + r) * OLD + 4 * q];
        const float* zr = &zbo[r][4 * q];
        f4 acc0 = f4{0.f, 0.f, 0.f, 0.f}, acc1 = f4{0.f, 0.f, 0.f, 0.f};
        f4 a0 = *(const f4*)zr, b0 = *(const f4*)wb, a1 = *(const f4*)(zr + 16), b1 = *(const f4*)(wb + 16);
#pragma unroll
        for (int ch = 0; ch < OK / 16; ch += 2) {
          f4 na0 = a0, nb0 = b0, na1 = a1, nb1 = b1;
          if (ch + 2 < OK / 16) {
            na0 = *(const f4*)(zr + 16 * (ch + 2));
            nb0 = *(const f4*)(wb + 16 * (ch + 2));
            na1 = *(const f4*)(zr + 16 * (ch + 3));
            nb1 = *(const f4*)(wb + 16 * (ch + 3));
          }
          __builtin_amdgcn_sched_barrier(0);
          acc0 = mma4(a0, b0, acc0);
          acc1 = mma4(a1, b1, acc1);
          a0 = na0, b0 = nb0, a1 = na1, b1 = nb1;
        }
        const f4 acc = acc0 + acc1;
        const int u = jb * 16 + r;
        if (u < UM) {
          float* pout = a.P + ((((size_t)(na & 1) * a.mtiles + mt) * nO + oc) * H) * 16;
          st4<kDev>(rsrc(pout, unsigned(H * 16 * 4)), unsigned(((ub0 + u) * 16 + 4 * q) * 4), acc);
        }
      }
    }
    ++na;
    return true;
  };

  bool ok = true, ended = false;
  for (pc = 0; pc < a.nprog && ok; ++pc) {
    const __attribute__((address_space(4))) int* op = prog + 4 * pc;
    const int code = op[0] & 0xff;
    if (code == kPFwd || code == kPAdj) {
      ok = step(op[1], op[2], op[3], code == kPAdj, code == kPAdj && op[3] != 0);
    } else if (code == kPCopy) {
      drain();
      if (op[1] > 0 && !wait_group(a.consumed, unsigned(op[1]))) {
        ok = false;
        break;
      }
      if (erow) {
        const __amdgpu_buffer_rsrc_t s = rsrc(buf(op[2]), sbytes), d = rsrc(buf(op[3]), sbytes);
        st1<kDev>(d, eoff, ld1<kDev>(s, eoff));
        if (G == 4) st1<kDev>(d, unsigned(a.c_off) + eoff, ld1<kDev>(s, unsigned(a.c_off) + eoff));
      }
    } else if (code == kPStore) {
      const bool staged = (op[0] & kPStaged) != 0;
      if (staged) __syncthreads();  // the step's output slice is in LDS
      else drain();
      if (wave == kCopyWave) {
        if (pend_store >= 0) {
          if (cl_ok) st4<kSys>(host_rsrc(pend_store), unsigned(lane) * 16u, sv);
        }
        if (staged) {
          sv = *(const f4*)&stg[4 * lane];
        } else {
          if (cl_ok) sv = ld4<kDev>(rsrc(buf(op[2]), sbytes), cl_off);
          dirty = true;  // the slot may be rewritten after the next barrier: land the load first
        }
      }
      pend_store = op[3];
    } else if (code == kPPref) {
      drain();
      if (pend_pref >= 0) {  // the host compiler separates prefetches by a barrier
        abort_op(3);
        ok = false;
        break;
      }
      if (pend_store >= 0) {  // the host slot may be the one being stored
        if (cl_ok) st4<kSys>(host_rsrc(pend_store), unsigned(lane) * 16u, sv);
        pcie_st = true;
      }
      if (early_pc != pc && wave == kCopyWave) host_read(op[2]);  // else it started at the last landing
      early_pc = -1;
      pend_store = -1;
      pend_pref = op[3];
      pref_next = op[1] > 0 ? op[1] : -1;
    } else if (code == kPSync) {
      drain();
      raise();
      ok = enter();
      if (ok) flush();
    } else if (code == kPEnd) {
      drain();
      raise();
      ok = enter();
      if (ok) flush();
      ended = ok;
      break;
    } else {
      abort_op(4);
      ok = false;
    }
  }
  if (!ended) return;

  // dL/dh_0 = sum of the partials of the adjoint of step 0; dL/dc_0 = cbar_0.
  // (after the loop, so that none of these addresses stays live through it)
  if (tid < kStageThreads) stage_partials();
  __syncthreads();
  if (erow) {
    float hbar = 0.f;
#pragma unroll
    for (int g = 0; g < kSmax; ++g)
      if (g < nO) hbar += hp[g][u * 16 + ml];
    a.dh0[em * H + ej] = hbar;
    if (G == 4) a.dc0[em * H + ej] = cbs[tid];
  }
#pragma unroll
  for (int i = 0; i < KCH; ++i) {
    const int ch = chunk(i);
    if (ch < nch) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int v = 0; v < 4; ++v)
          a.dWp[((size_t)mt * GH + wrow(nb * 16 + 4 * q + v)) * K1 + ch * 16 + r] = dacc[i][nb][v];
    }
  }
  if (tid < NC) a.dbp[(size_t)mt * GH + wrow(tid)] = dbacc;
  {
    double v = lacc;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
    if (lane == 0) wsum[wave] = v;
    __syncthreads();
    if (tid == 0) {
      double t = 0.0;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) t += wsum[w];
      a.loss_acc[me] = t;
    }
  }
}

__global__ void resident_reduce(const float* __restrict__ dWp, const float* __restrict__ dbp, int mtiles, int GH,
                                int K1, float* __restrict__ dW, float* __restrict__ db) {
  const size_t n = (size_t)GH * K1;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    float s = 0.f;
    for (int m = 0; m < mtiles; ++m) s += dWp[(size_t)m * n + i];
    dW[i] = s;
    if (i < (size_t)GH) {
      float t = 0.f;
      for (int m = 0; m < mtiles; ++m) t += dbp[(size_t)m * GH + i];
      db[i] = t;
    }
  }
}

}  // namespace

int resident_units(int G) { return G == 4 ? 8 : 16; }
int resident_max_k(int) { return kKmax; }
int resident_max_h(int) { return kHmax; }
int resident_octet(int ng, int H) {
  const int S = ng < kSmax ? ng : kSmax;
  return (ng % S == 0 && H % S == 0 && H / S <= kUMmax) ? S : 0;
}

// The kernel variant a problem runs: its reduction chunks per wave (the
// register-held weight slice) decide the template instance.
static const void* resident_fn(int G, int D, int H) {
  const int nch = (D + H) / 16, kch = (nch + kWaves - 1) / kWaves;
  if (kch <= 1) return G == 4 ? (const void*)resident_pass<4, 1> : (const void*)resident_pass<1, 1>;
  if (kch <= 2) return G == 4 ? (const void*)resident_pass<4, 2> : (const void*)resident_pass<1, 2>;
  if (kch <= 3) return G == 4 ? (const void*)resident_pass<4, 3> : (const void*)resident_pass<1, 3>;
  return G == 4 ? (const void*)resident_pass<4, kKch> : (const void*)resident_pass<1, kKch>;
}

hipError_t resident_capacity(int G, int D, int H, int* blocks) {
  int dev = 0, per = 0;
  hipDeviceProp_t prop;
  hipError_t e;
  if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
  if ((e = hipGetDeviceProperties(&prop, dev)) != hipSuccess) return e;
  // occupancy of the variant that launch_resident will launch for (G, D, H)
  if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, resident_fn(G, D, H), kThreads, 0)) != hipSuccess)
    return e;
  *blocks = prop.cooperativeLaunch ? per * prop.multiProcessorCount : 0;
  return hipSuccess;
}

hipError_t launch_resident(int G, const ResidentArgs& a, hipStream_t s, bool cooperative) {
  ResidentArgs arg = a;
  void* args[] = {&arg};
  const dim3 grid(unsigned(a.mtiles * a.ng)), block(kThreads);
  const void* fn = resident_fn(G, a.D, a.H);
  if (cooperative) return hipLaunchCooperativeKernel(fn, grid, block, args, 0, s);
  // plain launch: the caller checked that the grid fits the device at once;
  // if other work keeps some workgroups out, the bounded waits end the pass
  return hipLaunchKernel(fn, grid, block, args, 0, s);
}

hipError_t launch_resident_reduce(const float* dWp, const float* dbp, int mtiles, int GH, int K1, float* dW,
                                  float* db, hipStream_t s) {
  const size_t n = (size_t)GH * K1;
  const unsigned blocks = unsigned(std::min<size_t>((n + 255) / 256, 4096));
  hipLaunchKernelGGL(resident_reduce, dim3(blocks), dim3(256), 0, s, dWp, dbp, mtiles, GH, K1, dW, db);
  return hipGetLastError();
}

}  // namespace ambptt
