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
constexpr int kKch = 6;                      // 16-wide reduction chunks per wave: D + H <= 768
constexpr int kNbw = 5;                      // 16-column blocks of the partial product per wave: H <= 560
constexpr int kHmax = 16 * (kWaves - 1) * kNbw;
constexpr int kKmax = 16 * kWaves * kKch;
constexpr int kXld = kKmax + 4;              // LDS row stride of the staged [x | h] rows
constexpr int kDev = 16;                     // sc1: coherent across the device
constexpr int kSys = 17;                     // sc0 sc1: system scope (host memory)

typedef unsigned int u4v __attribute__((ext_vector_type(4)));

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base, unsigned bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, 0x00020000);
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

__device__ __forceinline__ float sigm(float z) { return 1.0f / (1.0f + __expf(-z)); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

template <int G>
__global__ __launch_bounds__(kThreads) void resident_pass(ResidentArgs a) {
  constexpr int U = (G == 4) ? 8 : 16;
  constexpr int NC = G * U;            // gate columns of the workgroup (32 | 16)
  constexpr int NB = NC / 16;          // 16-column MFMA blocks of the gate GEMM
  constexpr int KW = NC / 16;          // 16-wide chunks of the partial product's reduction
  constexpr int NS = 16 * U;           // (row, unit) pairs of the slice (128 | 256)
  constexpr int NG4 = NS / 4;          // float4s of one partial slab (32 | 64)
  constexpr int NGRP = kStageThreads / NG4;  // thread groups summing partials (14 | 7)
  constexpr int PER = U / 4;           // float4s per slice row
  static_assert(kStageThreads % NG4 == 0, "partial-sum groups");

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = lane & 15, q = lane >> 4;
  const int B = a.B, D = a.D, H = a.H, K1 = D + H, GH = G * H;
  const int ng = a.ng, nwg = a.mtiles * a.ng;
  int mt, ug;
  if (a.xcd_map) {  // ids are dealt to the 8 XCDs round-robin: keep a row tile on 8 / mtiles of them
    const int per = 8 / a.mtiles, x = int(blockIdx.x % 8);
    mt = x / per;
    ug = int(blockIdx.x / 8) * per + x % per;
  } else {
    mt = int(blockIdx.x) / ng;
    ug = int(blockIdx.x) % ng;
  }
  const int me = mt * ng + ug;
  const int m0 = 16 * mt, j0 = U * ug;
  const int nch = K1 / 16;
  const int c0 = (nch * wave) / kWaves, c1 = (nch * (wave + 1)) / kWaves;
  const int hb16 = H / 16;
  const unsigned hbytes = unsigned(B) * unsigned(H) * 4u;
  const unsigned sbytes = G == 4 ? unsigned(a.c_off) + hbytes : hbytes;
  auto wrow = [&](int n) { return (n / U) * H + j0 + (n % U); };  // W row of gate column n
  auto buf = [&](int id) -> char* {
    return id < a.nslots ? a.pool + (size_t)id * a.stride : (id == a.nslots ? a.live0 : a.live1);
  };

  __shared__ __attribute__((aligned(16))) float xs[16][kXld];  // [x_t | h_t] rows of the tile
  __shared__ float zs[kWaves][16][NC + 1];                     // per-wave gate partial sums
  __shared__ __attribute__((aligned(16))) float zb[16][NC + 4];  // zbar_t of the workgroup
  __shared__ float hp[NGRP][NS];                               // partial h-adjoint sums
  __shared__ float cbs[NS];                                    // cbar carried between adjoints
  __shared__ __attribute__((aligned(16))) float whs[NC * (kHmax + 4)];  // W_h rows of the gate columns
  __shared__ float wsum[kWaves];
  __shared__ int stop;

  // ---- weights into registers ---------------------------------------------
  f4 Wr[kKch][NB];  // B operands of the gate GEMM: W[col][16 ch + 4 q + e]
#pragma unroll
  for (int i = 0; i < kKch; ++i) {
    const int ch = c0 + i;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
      Wr[i][nb] = ch < c1 ? *(const f4*)(a.W + (size_t)wrow(nb * 16 + r) * K1 + ch * 16 + 4 * q)
                          : f4{0.f, 0.f, 0.f, 0.f};
  }
  // rows of W_h for the workgroup's gate columns (the partial product's B
  // operand), whs[n][j] = W[wrow(n)][D + j]; the row stride H + 4 keeps the
  // four row groups of a wave's read on different banks
  const int whld = H + 4;
  for (int idx = tid; idx < NC * (H / 4); idx += kThreads) {
    const int n = idx / (H / 4), col = 4 * (idx % (H / 4));
    *(f4*)&whs[n * whld + col] = *(const f4*)(a.W + (size_t)wrow(n) * K1 + D + col);
  }
  f4 dacc[kKch][NB];  // dW blocks (gate block nb, reduction chunk c0 + i)
#pragma unroll
  for (int i = 0; i < kKch; ++i)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) dacc[i][nb] = f4{0.f, 0.f, 0.f, 0.f};
  float dbacc = 0.f;
  double lacc = 0.0;

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
  int pend_store = -1; // host slot of the store whose data the copy wave holds
  bool dirty = false;  // the copy wave wrote a slot since its last drain
  f4 pv = f4{0.f, 0.f, 0.f, 0.f}, sv = f4{0.f, 0.f, 0.f, 0.f};
  int pc = 0;

  // all stores of this workgroup that others may read are complete
  auto drain = [&]() {
    if (wave != kCopyWave || dirty) __builtin_amdgcn_s_waitcnt(0);
    dirty = false;
    __syncthreads();
  };
  // wave 0 waits until every member's flag reaches target
  auto wait_group = [&](const unsigned* flags, unsigned target) -> bool {
    if (wave == 0) {
      const unsigned long long t0 = __builtin_amdgcn_s_memrealtime();
      int st = 0;
      for (unsigned it = 0;; ++it) {
        bool ok = true;
        for (int j = lane; j < ng; j += 64) ok = ok && ld_flag(flags + mt * ng + j) >= target;
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
  auto enter = [&]() -> bool {  // group barrier number sc + 1 (caller drained)
    if (tid == 0) st_flag(a.ready + me, sc + 1);
    if (!wait_group(a.ready, sc + 1)) return false;
    ++sc;
    return true;
  };
  auto flush = [&]() {  // complete the held transfers (after a barrier; the copy wave's lanes move data)
    if (pend_pref >= 0) {
      if (cl_ok) st4<kDev>(rsrc(buf(pend_pref), sbytes), cl_off, pv);
      dirty = true;
      pend_pref = -1;
    }
    if (pend_store >= 0) {
      if (cl_ok) st4<kSys>(host_rsrc(pend_store), unsigned(lane) * 16u, sv);
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
    if (!enter()) return false;
    // stage [x_t | h_t]; the adjoint also sums the partial h-adjoints of step t + 1
    if (tid < kStageThreads) {
      const int nh4 = 4 * H;
      for (int idx = tid; idx < nh4; idx += kStageThreads) {
        const int row = idx / (H / 4), col = 4 * (idx % (H / 4));
        f4 v = f4{0.f, 0.f, 0.f, 0.f};
        if (m0 + row < B) v = ld4<kDev>(srs, unsigned(((m0 + row) * H + col) * 4));
        *(f4*)&xs[row][D + col] = v;
      }
      if (adj && !first) {
        const int v4 = tid % NG4, grp = tid / NG4;
        const float* slab = a.P + ((((size_t)((na + 1) & 1) * a.mtiles + mt) * ng + ug) * ng) * NS;
        const __amdgpu_buffer_rsrc_t prs = rsrc(slab, unsigned(ng * NS * 4));
        f4 s = f4{0.f, 0.f, 0.f, 0.f};
        for (int srcw = grp; srcw < ng; srcw += NGRP) s += ld4<kDev>(prs, unsigned((srcw * NS + 4 * v4) * 4));
        *(f4*)&hp[grp][4 * v4] = s;
      }
    }
    __syncthreads();
    if (tid == 0) st_flag(a.consumed + me, sc);
    flush();

    // gate GEMM: z[16][NC] = [x|h] W^T over this wave's chunks
    {
      f4 acc[NB];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) acc[nb] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < kKch; ++i) {
        const int ch = c0 + i;
        if (ch < c1) {
          const f4 av = *(const f4*)&xs[r][ch * 16 + 4 * q];
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) acc[nb] = mma4(av, Wr[i][nb], acc[nb]);
        }
      }
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int v = 0; v < 4; ++v) zs[wave][4 * q + v][nb * 16 + r] = acc[nb][v];
    }
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
        gg = tanhf(z[2 % G]);
        og = sigm(z[3 % G]);
        c1 = fg * cold + ig * gg;
        tc = tanhf(c1);
        h1 = og * tc;
      } else {
        h1 = tanhf(z[0]);
      }
      if (!adj) {
        if (erow) {
          const __amdgpu_buffer_rsrc_t drs = rsrc(buf(dst), sbytes);
          st1<kDev>(drs, eoff, h1);
          if (G == 4) st1<kDev>(drs, unsigned(a.c_off) + eoff, c1);
        }
      } else {
        float hbar = 0.f;
        if (!first) {
#pragma unroll
          for (int g = 0; g < NGRP; ++g) hbar += hp[g][u * 16 + ml];
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
      }
    }
    if (!adj) return true;

    const float ls = wave_sum(lterm);
    if (lane == 0) wsum[wave] = ls;
    __syncthreads();
    if (tid == 0) {
      float s = 0.f;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) s += wsum[w];
      lacc += (double)s;
    }
    // partial h-adjoint of the workgroup's gate columns, to the owners of the units
    if (wave < kCopyWave) {
      float* pbase = a.P + (((size_t)(na & 1) * a.mtiles + mt) * ng) * ng * NS;
      const __amdgpu_buffer_rsrc_t prs = rsrc(pbase, unsigned(ng * ng * NS * 4));
#pragma unroll
      for (int i = 0; i < kNbw; ++i) {
        const int jb = wave + kCopyWave * i;
        if (jb < hb16) {
          f4 acc = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int ch = 0; ch < KW; ++ch) {
            const f4 av = *(const f4*)&zb[r][16 * ch + 4 * q];
            const float* wb = &whs[(16 * ch + 4 * q) * whld + jb * 16 + r];
            const f4 bv = f4{wb[0], wb[whld], wb[2 * whld], wb[3 * whld]};
            acc = mma4(av, bv, acc);
          }
          const int col = jb * 16 + r, dsw = col / U, du = col % U;
          st4<kDev>(prs, unsigned(((dsw * ng + ug) * NS + du * 16 + 4 * q) * 4), acc);
        }
      }
    }
    // weight gradient of the workgroup's gate rows, dW += zbar^T [x | h], on
    // the wave's own reduction chunks (block (nb, chunk) of 16 x 16)
#pragma unroll
    for (int c4 = 0; c4 < 4; ++c4) {
      float av[NB];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) av[nb] = zb[4 * c4 + q][nb * 16 + r];
#pragma unroll
      for (int i = 0; i < kKch; ++i) {
        const int ch = c0 + i;
        if (ch < c1) {
          const float bv = xs[4 * c4 + q][ch * 16 + r];
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) dacc[i][nb] = mfma_f32_16x16x4(av[nb], bv, dacc[i][nb]);
        }
      }
    }
    if (tid < NC) {
      float s = 0.f;
#pragma unroll
      for (int row = 0; row < 16; ++row) s += zb[row][tid];
      dbacc += s;
    }
    ++na;
    return true;
  };

  bool ok = true, ended = false;
  for (pc = 0; pc < a.nprog && ok; ++pc) {
    const int* op = a.prog + 4 * pc;
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
      drain();
      if (wave == kCopyWave) {
        if (pend_store >= 0) {
          if (cl_ok) st4<kSys>(host_rsrc(pend_store), unsigned(lane) * 16u, sv);
        }
        if (cl_ok) sv = ld4<kDev>(rsrc(buf(op[2]), sbytes), cl_off);
        dirty = true;  // the slot may be rewritten after the next barrier: land the load first
      }
      pend_store = op[3];
    } else if (code == kPPref) {
      drain();
      if (pend_pref >= 0) {  // the host compiler separates prefetches by a barrier
        abort_op(3);
        ok = false;
        break;
      }
      if (wave == kCopyWave) {
        if (pend_store >= 0) {  // the host slot may be the one being stored
          if (cl_ok) st4<kSys>(host_rsrc(pend_store), unsigned(lane) * 16u, sv);
          __builtin_amdgcn_s_waitcnt(0);
        }
        if (cl_ok) pv = ld4<kSys>(host_rsrc(op[2]), unsigned(lane) * 16u);
      }
      pend_store = -1;
      pend_pref = op[3];
    } else if (code == kPSync) {
      drain();
      ok = enter();
      if (ok) flush();
    } else if (code == kPEnd) {
      drain();
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
  if (tid < kStageThreads) {
    const int v4 = tid % NG4, grp = tid / NG4;
    const float* slab = a.P + ((((size_t)((na + 1) & 1) * a.mtiles + mt) * ng + ug) * ng) * NS;
    const __amdgpu_buffer_rsrc_t prs = rsrc(slab, unsigned(ng * NS * 4));
    f4 s = f4{0.f, 0.f, 0.f, 0.f};
    for (int srcw = grp; srcw < ng; srcw += NGRP) s += ld4<kDev>(prs, unsigned((srcw * NS + 4 * v4) * 4));
    *(f4*)&hp[grp][4 * v4] = s;
  }
  __syncthreads();
  if (erow) {
    float hbar = 0.f;
#pragma unroll
    for (int g = 0; g < NGRP; ++g) hbar += hp[g][u * 16 + ml];
    a.dh0[em * H + ej] = hbar;
    if (G == 4) a.dc0[em * H + ej] = cbs[tid];
  }
#pragma unroll
  for (int i = 0; i < kKch; ++i) {
    const int ch = c0 + i;
    if (ch < c1) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int v = 0; v < 4; ++v)
          a.dWp[((size_t)mt * GH + wrow(nb * 16 + 4 * q + v)) * K1 + ch * 16 + r] = dacc[i][nb][v];
    }
  }
  if (tid < NC) a.dbp[(size_t)mt * GH + wrow(tid)] = dbacc;
  if (tid == 0) a.loss_acc[me] = lacc;
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

hipError_t resident_capacity(int G, int* blocks) {
  int dev = 0, per = 0;
  hipDeviceProp_t prop;
  hipError_t e;
  if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
  if ((e = hipGetDeviceProperties(&prop, dev)) != hipSuccess) return e;
  if (G == 4) e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, resident_pass<4>, kThreads, 0);
  else e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, resident_pass<1>, kThreads, 0);
  if (e != hipSuccess) return e;
  *blocks = prop.cooperativeLaunch ? per * prop.multiProcessorCount : 0;
  return hipSuccess;
}

hipError_t launch_resident(int G, const ResidentArgs& a, hipStream_t s, bool cooperative) {
  ResidentArgs arg = a;
  void* args[] = {&arg};
  const dim3 grid(unsigned(a.mtiles * a.ng)), block(kThreads);
  const void* fn = G == 4 ? (const void*)resident_pass<4> : (const void*)resident_pass<1>;
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
