// Wide-batch bf16 step kernels (gfx950): the LSTM / tanh-RNN cell and the
// residual MLP when the batch has 48 rows or more.
//
// At these shapes a step is a short, fat GEMM (the 2048-wide LSTM: 128 x 8192
// x 3072 with a 50 MB weight matrix; the 4096-wide MLP layer: 256 x 4096 x
// 4096).  What bounds it is how fast every CU pulls its operands through L2,
// not the MFMA rate.  Two choices follow from that:
//   * Tiles move the fewest bytes per CU: a 64 x 64 output tile per
//     workgroup for the cell's gate GEMM (64 batch rows x 16 LSTM units, all
//     four gates) and for the MLP layer, 32 x 32 for the h-adjoint product.
//     The adjoint's products hbar = zbar W_h (cell) and zbar W_{l+1} (MLP)
//     are launches of their own: each reads the whole zbar of its rows, and
//     fused into the cell kernel's tile they would move twice the bytes.
//   * Loads cover whole 128-byte lines.  The activation operand is read as
//     rows, one load instruction covering 8 rows x 128 bytes (lane l: row
//     l >> 3, bytes 16 (l & 7) ..), which pulls about twice the bandwidth of
//     the MFMA operand layout (16 rows x 64 bytes per instruction); each wave
//     turns its rows into MFMA fragments through LDS scratch tiles of its own
//     (swizzled 16 x 128-byte tiles), so no workgroup barrier sits in the
//     main loop.  The recurrent cell's weights, fixed for a pass, are read
//     from a copy in fragment order (pack_nt below): one load instruction
//     reads a fragment's 1 KiB contiguously into the lanes that multiply it,
//     with no trip through LDS.
// Inside a workgroup the 8 waves split the reduction in 64-wide blocks, so no
// byte is loaded twice; the loads of the next block(s) are in flight while
// the current one is multiplied.  The partial products meet in LDS and are
// summed in wave order (bit-reproducible).
//
// Operands are bf16 on v_mfma_f32_16x16x32_bf16 (lane l: row or column
// l & 15, reduction indices 8 (l >> 4) .. +7 of a 32-wide chunk; result:
// column l & 15, rows 4 (l >> 4) .. +3).  Stored h / y, zbar and the copies
// kept for the weight gradient are bf16 (nearest even); accumulation, the
// LSTM cell state, its adjoint and the carried MLP adjoint stay fp32.
#include <hip/hip_runtime.h>

#include "ambptt.h"
#include "kernels.hpp"
#include "mfma.hpp"

namespace ambptt {
namespace {

constexpr int kWaves = 8;  // waves per workgroup of the launched kernels
constexpr int kSlot = 2048;  // one 16-row x 128-byte scratch tile

typedef unsigned int u4v __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float sigm(float z) { return 1.0f / (1.0f + __expf(-z)); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// Workgroup id -> tile, XCD-aware: ids are dealt to the 8 XCDs round-robin,
// and each XCD takes a contiguous run of tiles numbered column-group major,
// so the row groups that share weight rows share one L2.
__device__ __forceinline__ int tile_of(int ntile) {
  const int per = (ntile + 7) / 8;
  return int(blockIdx.x % 8) * per + int(blockIdx.x / 8);
}

// Buffer descriptor of a whole operand.  Every buffer here is the same for
// all lanes of a wave; readfirstlane states that, so the descriptor sits in
// scalar registers.  Reads at or past `bytes` return zero (rows beyond the
// batch).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base, unsigned bytes) {
  const unsigned long long p = (unsigned long long)base;
  const unsigned lo = __builtin_amdgcn_readfirstlane(unsigned(p)), hi = __builtin_amdgcn_readfirstlane(unsigned(p >> 32));
  void* ub = (void*)(((unsigned long long)hi << 32) | lo);
  return __builtin_amdgcn_make_buffer_rsrc(ub, 0, __builtin_amdgcn_readfirstlane(bytes), 0x00020000);
}
__device__ __forceinline__ u4v bload(__amdgpu_buffer_rsrc_t r, unsigned voff, unsigned soff) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
}

// Rows of a row-major operand, read in 16-row groups and 64-wide reduction
// blocks (128 bytes of a bf16 row).  Instruction h of group g covers rows
// row0 + 16 g + 8 h + (lane >> 3), bytes 16 (lane & 7) .. +15 of the block.
struct Rows {
  __amdgpu_buffer_rsrc_t r;
  unsigned voff;    // lane part: (lane >> 3) stride + 16 (lane & 7)
  unsigned base;    // row0 stride (the same for the wave)
  unsigned stride;  // row stride in bytes
  __device__ __forceinline__ u4v load(int g, int h, int blk) const {
    return bload(r, voff, base + unsigned(16 * g + 8 * h) * stride + unsigned(blk) * 128u);
  }
  // instruction h of the 16 rows starting at row `first` (an absolute row)
  __device__ __forceinline__ u4v load_at(int first, int h, int blk) const {
    return bload(r, voff, unsigned(first + 8 * h) * stride + unsigned(blk) * 128u);
  }
};
__device__ __forceinline__ Rows rows_of(const void* p, unsigned bytes, int row0, int stride_bytes) {
  const int lane = threadIdx.x & 63;
  Rows s;
  s.r = rsrc(p, bytes);
  s.voff = unsigned((lane >> 3) * stride_bytes + 16 * (lane & 7));
  s.base = unsigned(row0) * unsigned(stride_bytes);
  s.stride = unsigned(stride_bytes);
  return s;
}

// An NT operand Bm(k, n) = B[n][k] in fragment order: the fragment of n tile
// jt (columns 16 jt ..) and 32-wide reduction step ks is 1 KiB, lane l's 16
// bytes being B[16 jt + (l & 15)][32 ks + 8 (l >> 4) .. +7], the operand
// layout of v_mfma_f32_16x16x32_bf16; the K / 32 fragments of an n tile are
// consecutive (n tile major).
struct Frags {
  __amdgpu_buffer_rsrc_t r;
  unsigned voff;  // 16 lane
  unsigned tile;  // bytes of one n tile: K / 32 fragments
  __device__ __forceinline__ u4v load(int jt, int ks) const {
    return bload(r, voff, unsigned(jt) * tile + unsigned(ks) * 1024u);
  }
};
__device__ __forceinline__ Frags frags_of(const void* p, int N, int K) {
  Frags f;
  f.r = rsrc(p, unsigned(N) * unsigned(K) * 2u);
  f.voff = unsigned(threadIdx.x & 63) * 16u;
  f.tile = unsigned(K / 32) * 1024u;
  return f;
}

// Per-lane LDS offsets within one 16 x 128-byte scratch tile.  Row t's
// 16-byte group k sits at slot k ^ (t & 7): the 8 lanes that write one row hit
// 8 different slots, and the reads of one fragment column spread over the
// banks (measured free of bank conflicts on gfx950, where an extra flip for
// rows 8..15 was not).
struct Xpose {
  unsigned w0, w1;  // writes of the rows-0..7 and rows-8..15 instructions
  unsigned r0, r1;  // fragment reads: reduction indices 0..31 and 32..63 of the block
  __device__ __forceinline__ void init() {
    const int lane = threadIdx.x & 63;
    auto sw = [](int t) { return t & 7; };
    const int t0 = lane >> 3, t1 = 8 + (lane >> 3), k = lane & 7;
    w0 = unsigned(t0 * 128 + 16 * (k ^ sw(t0)));
    w1 = unsigned(t1 * 128 + 16 * (k ^ sw(t1)));
    const int r = lane & 15, q = lane >> 4;
    r0 = unsigned(r * 128 + 16 * (q ^ sw(r)));
    r1 = unsigned(r * 128 + 16 * ((q + 4) ^ sw(r)));
  }
  __device__ __forceinline__ void put(char* tile, const u4v& v0, const u4v& v1) const {
    *(u4v*)(tile + w0) = v0;
    *(u4v*)(tile + w1) = v1;
  }
  // the MFMA fragment of the block's 32-wide chunk c
  __device__ __forceinline__ bf16x8 get(const char* tile, int c) const {
    return __builtin_bit_cast(bf16x8, *(const u4v*)(tile + (c ? r1 : r0)));
  }
};

// Software pipeline over reduction blocks [c0, c1): ld(blk, s) issues the
// loads of block blk into register buffer s, use(s) consumes buffer s.  The
// loads of S - 1 blocks are in flight while one is used.  c0 and c1 are the
// same for the whole wave, so every branch is scalar; the steady-state body
// has no branch and the stages keep their order, so the wait before each use
// leaves the younger blocks' loads outstanding.
template <int S, class LD, class USE>
__device__ __forceinline__ void pipeline(int c0, int c1, LD ld, USE use) {
  if (c1 <= c0) return;
  // unconditional prologue (a short range loads its last block again) in
  // stage order: the wait at the loop head is the worst case over the loop's
  // entry and its back edge
#pragma unroll
  for (int s = 0; s < S; ++s) {
    ld(min(c0 + s, c1 - 1), s);
    __builtin_amdgcn_sched_barrier(0);
  }
  int ch = c0;
  for (; ch + 2 * S <= c1; ch += S) {  // blocks ch .. ch + S - 1 are in buffers 0 .. S - 1
#pragma unroll
    for (int s = 0; s < S; ++s) {
      use(s);
      ld(ch + S + s, s);
      // keep the stages in order: the compiler would otherwise gather every
      // MFMA of the body ahead of every load and wait for all loads at once
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  // the last S .. 2S - 1 blocks
#pragma unroll
  for (int s = 0; s < S; ++s) {
    if (ch + s < c1) {
      use(s);
      if (ch + S + s < c1) ld(ch + S + s, s);
    }
  }
  ch += S;
#pragma unroll
  for (int s = 0; s < S; ++s)
    if (ch + s < c1) use(s);
}

// acc[i][nb] += A_i . B_nb over the wave's blocks [c0, c1); la(g, h, blk) and
// lb(g, h, blk) load instruction h of 16-row group g of block blk.  The wave's
// scratch `scr` holds NB + RT tiles.  With PB, lb(g, c, blk) loads the
// fragment of B's group g for the block's 32-wide chunk c (Frags), which the
// MFMAs take as loaded.
template <int RT, int NB, int S, bool PB = false, class LA, class LB>
__device__ __forceinline__ void nt_rows(int c0, int c1, char* scr, const Xpose& X, f4 (&acc)[RT][NB], LA la, LB lb) {
  u4v va[S][RT][2], vb[S][NB][2];
  pipeline<S>(
      c0, c1,
      [&](int blk, int s) {
#pragma unroll
        for (int g = 0; g < RT; ++g)
#pragma unroll
          for (int h = 0; h < 2; ++h) va[s][g][h] = la(g, h, blk);
#pragma unroll
        for (int g = 0; g < NB; ++g)
#pragma unroll
          for (int h = 0; h < 2; ++h) vb[s][g][h] = lb(g, h, blk);
      },
      [&](int s) {
        if constexpr (!PB) {
#pragma unroll
          for (int g = 0; g < NB; ++g) X.put(scr + g * kSlot, vb[s][g][0], vb[s][g][1]);
        }
#pragma unroll
        for (int i = 0; i < RT; ++i) X.put(scr + (NB + i) * kSlot, va[s][i][0], va[s][i][1]);
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          bf16x8 fb[NB];
#pragma unroll
          for (int g = 0; g < NB; ++g) fb[g] = PB ? __builtin_bit_cast(bf16x8, vb[s][g][c]) : X.get(scr + g * kSlot, c);
#pragma unroll
          for (int i = 0; i < RT; ++i) {
            const bf16x8 fa = X.get(scr + (NB + i) * kSlot, c);
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) acc[i][nb] = mfma_bf16_16x16x32(fa, fb[nb], acc[i][nb]);
          }
        }
        __builtin_amdgcn_wave_barrier();  // the tiles are read before the next block is stored
      });
}

// The wave's partial products -> ps[wave][row][col] (LDS, after every wave
// has left its main loop); the workgroup-wide sum runs in wave order.
template <int RT, int NB>
__device__ __forceinline__ void put_partials(float* ps, int wave, const f4 (&acc)[RT][NB]) {
  constexpr int LD = 16 * NB + 1;
  const int lane = threadIdx.x & 63, r = lane & 15, q = lane >> 4;
  float* p = ps + wave * (16 * RT) * LD;
#pragma unroll
  for (int i = 0; i < RT; ++i)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int v = 0; v < 4; ++v) p[(16 * i + 4 * q + v) * LD + nb * 16 + r] = acc[i][nb][v];
}
template <int RT, int NB, int NW>
__device__ __forceinline__ float sum_partials(const float* ps, int row, int col) {
  constexpr int LD = 16 * NB + 1, W = 16 * RT * LD;
  float s = 0.f;
#pragma unroll
  for (int wv = 0; wv < NW; ++wv) s += ps[wv * W + row * LD + col];
  return s;
}

// LDS of a kernel: the partial sums, or the waves' scratch, whichever is larger
template <int RT, int NB, int SCR, int NW>
constexpr int lds_bytes() {
  constexpr int ps = NW * 16 * RT * (16 * NB + 1) * 4;
  constexpr int sc = NW * SCR;
  return ps > sc ? ps : sc;
}

// ---- the recurrent cell: gate GEMM + cell update ----------------------------
//
// Workgroup tile: 64 batch rows x UN hidden units, all G gates (64 gate
// columns: UN = 16 for the LSTM, 64 for the tanh RNN).  Gate column n =
// g UN + u is weight row g H + j0 + u; a 16-column group is 16 consecutive
// weight rows, one n tile of the fragment-order copy of W (a.W: pack_nt of
// the [G H][D + H] weights).  Forward: h_{t+1}, c_{t+1}.  Adjoint (gate recomputation of
// step t): with hbar_{t+1} from the product launch before it (absent for the
// first turn) it forms zbar_t, cbar_t, the loss term and the copy of h_t for
// the weight-gradient window.
template <int G, int MODE, int NW = kWaves, int S = 2>
__global__ __launch_bounds__(64 * NW) void cell_wide(StepArgs a) {
  constexpr int RT = 4, NB = 4, TM = 64;
  constexpr int UN = 64 / G;  // hidden units of the tile
  constexpr int SCR = (RT + NB) * kSlot;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int B = a.B, D = a.D, H = a.H, GH = G * H, K1 = D + H;
  const int mg = (B + TM - 1) / TM, ntile = mg * (H / UN);
  const int w = tile_of(ntile);
  if (w >= ntile) return;  // grid padding (the whole workgroup leaves together)
  const int m0 = (w % mg) * TM, j0 = (w / mg) * UN;

  __shared__ __attribute__((aligned(16))) char lds[lds_bytes<RT, NB, SCR, NW>()];
  float* ps = (float*)lds;
  {
    f4 acc[RT][NB];
#pragma unroll
    for (int i = 0; i < RT; ++i)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) acc[i][nb] = f4{0.f, 0.f, 0.f, 0.f};
    Xpose X;
    X.init();
    const int nbk = K1 / 64, nbx = D / 64;
    const int c0 = (nbk * wave) / NW, c1 = (nbk * (wave + 1)) / NW;
    const Rows xs = rows_of(a.x, unsigned(size_t(B) * D * 2), m0, 2 * D);  // < 4 GiB: cell_wide_fits
    const Rows hs = rows_of(a.h, unsigned(size_t(B) * H * 2), m0, 2 * H);
    const Frags wf = frags_of(a.W, GH, K1);
    nt_rows<RT, NB, S, true>(
        c0, c1, lds + wave * SCR, X, acc,
        [&](int g, int h, int blk) -> u4v {  // an x or an h block: the same choice for the whole wave
          return blk < nbx ? xs.load(g, h, blk) : hs.load(g, h, blk - nbx);
        },
        [&](int g, int c, int blk) -> u4v { return wf.load(((16 * g / UN) * H + j0 + (16 * g) % UN) / 16, 2 * blk + c); });
    __syncthreads();  // every wave has left its scratch
    put_partials<RT, NB>(ps, wave, acc);
  }
  __syncthreads();

  // epilogue: pair (row ml, unit u), consecutive threads on consecutive units
  float lterm = 0.f;
  for (int pi = tid; pi < TM * UN; pi += 64 * NW) {
    const int ml = pi / UN, u = pi % UN;
    const int m = m0 + ml, j = j0 + u;
    if (m >= B) continue;
    const int o = m * H + j;
    float z[G];
#pragma unroll
    for (int g = 0; g < G; ++g) z[g] = sum_partials<RT, NB, NW>(ps, ml, g * UN + u) + a.bias[g * H + j];
    float h1, c1 = 0.f, tc = 0.f, ig = 0.f, fg = 0.f, gg = 0.f, og = 0.f, cold = 0.f;
    if (G == 4) {
      ig = sigm(z[0]);
      fg = sigm(z[1 % G]);
      gg = tanhf(z[2 % G]);
      og = sigm(z[3 % G]);
      cold = a.c[o];
      c1 = fg * cold + ig * gg;
      tc = tanhf(c1);
      h1 = og * tc;
    } else {
      h1 = tanhf(z[0]);
    }
    const __bf16 h1s = (__bf16)h1;  // the stored state (nearest even)
    if (MODE == kForward) {
      ((__bf16*)a.h_out)[o] = h1s;
      if (G == 4) a.c_out[o] = c1;
    } else {
      const float hl = (float)h1s;  // loss and seed read the stored h_{t+1}
      float sd = 0.f, lt = 0.f;
      if (a.loss == AMBPTT_LOSS_MEAN_SQ_ALL) {
        sd = 2.f * hl * a.inv_bh;
        lt = hl * hl;
      } else if (a.last) {
        if (a.loss == AMBPTT_LOSS_HALF_SQ_LAST) {
          sd = hl;
          lt = hl * hl;
        } else {
          sd = a.inv_bh;
          lt = hl;
        }
      }
      lterm += lt;
      const float hb = (a.first ? 0.f : a.hbar_in[o]) + sd;
      __bf16* zo = (__bf16*)a.zbar_out + (size_t)m * GH + j;
      if (G == 4) {
        const float cb = a.first ? 0.f : a.cbar_in[o];
        const float ob = hb * tc;
        const float ch = cb + hb * og * (1.f - tc * tc);
        zo[0] = (__bf16)(ch * gg * ig * (1.f - ig));
        zo[H] = (__bf16)(ch * cold * fg * (1.f - fg));
        zo[2 * H] = (__bf16)(ch * ig * (1.f - gg * gg));
        zo[3 * H] = (__bf16)(ob * og * (1.f - og));
        a.cbar_out[o] = ch * fg;
      } else {
        zo[0] = (__bf16)(hb * (1.f - h1 * h1));
      }
      ((__bf16*)a.hwin_out)[o] = ((const __bf16*)a.h)[o];
    }
  }
  if (MODE == kAdjoint) {
    const float s = wave_sum(lterm);
    __shared__ float wsum[NW];
    if (lane == 0) wsum[wave] = s;
    __syncthreads();
    if (tid == 0) {
      float t = 0.f;
#pragma unroll
      for (int wv = 0; wv < NW; ++wv) t += wsum[wv];
      a.loss_acc[w] += (double)t;
    }
  }
}

// The NN product's B block in LDS: row t (one k, 64 columns n) is 128 bytes,
// its 32-byte segments (16 columns each) permuted by nn_swz(t) so that the
// 16 rows one transposing read touches (rows kb + 8 g + 0..3, g = 0..3) fall
// on distinct banks within each half wave.
__device__ __forceinline__ int nn_swz(int t) { return ((t >> 1) & 1) | (((t >> 3) & 1) << 1); }

// Fragment of the block's 16 x 32 piece (columns 16 nb .., rows kb .. kb + 31):
// lane l receives rows kb + 8 (l >> 4) .. +7 of column l & 15.  Each
// ds_read_b64_tr_b16 gives lane j of a 16-lane group rows r .. r + 3 of
// column j, the group's lane i naming 4 consecutive values (row r + (i >> 2),
// columns 4 (i & 3) ..) of that 16-column segment.
__device__ __forceinline__ bf16x8 nn_frag(const char* bt, int kb, int nb) {
  const int lane = threadIdx.x & 63, g = lane >> 4, i = lane & 15;
  const int r0 = kb + 8 * g + (i >> 2), r1 = r0 + 4;
  typedef short s4 __attribute__((ext_vector_type(4)));
  typedef short s8 __attribute__((ext_vector_type(8)));
  typedef __attribute__((address_space(3))) s4 lds_s4;
  const s4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4*)(bt + r0 * 128 + 32 * (nb ^ nn_swz(r0)) + 8 * (i & 3)));
  const s4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4*)(bt + r1 * 128 + 32 * (nb ^ nn_swz(r1)) + 8 * (i & 3)));
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

// ---- products of the adjoint ------------------------------------------------
//
// out[m][n] = add[m][n] (if given) + sum_k A[m][k] Bm(k, n), A [M][K] bf16,
// over a TM x TN tile (TM = 16 RT, TN = 16 NB) per workgroup.
//   NN = false: Bm(k, n) = B[n][k] (the cell's W_h^T), B in fragment order
//     (pack_nt of the [N][K] rows);
//   NN = true:  Bm(k, n) = B[k][n] (the MLP's W_{l+1}, contiguous in n; TN =
//     64): each block's 64 x 64 elements of B go to the wave's scratch as
//     loaded (rows k of 128 bytes) and come back as fragments through
//     gfx950's transposing LDS read, so no transposed copy of the weights
//     is kept.
template <int RT, int NB, bool NN, int NW = kWaves, int S = NN ? 2 : (RT * NB >= 4 ? 3 : 4)>
__global__ __launch_bounds__(64 * NW) void prod_wide(ProdArgs a) {
  constexpr int TM = 16 * RT, TN = 16 * NB;
  constexpr int SCR = NN ? RT * kSlot + 64 * 128 : (RT + NB) * kSlot;
  static_assert(!NN || TN == 64, "the NN product takes 64-column tiles");
  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int M = a.M, N = a.N, K = a.K;
  const int mg = (M + TM - 1) / TM, ntile = mg * (N / TN);
  const int w = tile_of(ntile);
  if (w >= ntile) return;
  const int m0 = (w % mg) * TM, n0 = (w / mg) * TN;

  __shared__ __attribute__((aligned(16))) char lds[lds_bytes<RT, NB, SCR, NW>()];
  f4 acc[RT][NB];
#pragma unroll
  for (int i = 0; i < RT; ++i)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[i][nb] = f4{0.f, 0.f, 0.f, 0.f};
  const int nbk = K / 64;
  const int c0 = (nbk * wave) / NW, c1 = (nbk * (wave + 1)) / NW;
  Xpose X;
  X.init();
  char* scr = lds + wave * SCR;
  const Rows as = rows_of(a.A, unsigned(size_t(M) * K * 2), m0, 2 * K);  // < 4 GiB: the fits checks
  if constexpr (!NN) {
    const Frags bf = frags_of(a.B, N, K);
    nt_rows<RT, NB, S, true>(
        c0, c1, scr, X, acc, [&](int g, int h, int blk) -> u4v { return as.load(g, h, blk); },
        [&](int g, int c, int blk) -> u4v { return bf.load(n0 / 16 + g, 2 * blk + c); });
  } else {
    // B block: instruction p covers k rows 8 p + (lane >> 3) of the block, columns n0 + 8 (lane & 7) .. +7.
    // Row t of the block is stored as 128 bytes, its four 32-byte segments (16 columns each) permuted by
    // nn_swz(t), and a fragment (column l & 15 of a 16-column segment, 8 consecutive k) comes back with two
    // transposing reads (nn_frag).
    const int lane = tid & 63;
    const Rows bs = rows_of(a.B, unsigned(size_t(K) * N * 2), 0, 2 * N);
    const unsigned bcol = unsigned(n0) * 2u;
    char* bt = scr + RT * kSlot;
    const int lr = lane >> 3, lp = lane & 7;  // row within the instruction, 16-byte piece of the row
    u4v va[S][RT][2], vb[S][8];
    pipeline<S>(
        c0, c1,
        [&](int blk, int s) {
#pragma unroll
          for (int g = 0; g < RT; ++g)
#pragma unroll
            for (int h = 0; h < 2; ++h) va[s][g][h] = as.load(g, h, blk);
#pragma unroll
          for (int p = 0; p < 8; ++p) vb[s][p] = bload(bs.r, bs.voff, bcol + unsigned(blk * 64 + 8 * p) * bs.stride);
        },
        [&](int s) {
#pragma unroll
          for (int i = 0; i < RT; ++i) X.put(scr + i * kSlot, va[s][i][0], va[s][i][1]);
#pragma unroll
          for (int p = 0; p < 8; ++p) {
            const int t = 8 * p + lr;
            *(u4v*)(bt + t * 128 + 32 * ((lp >> 1) ^ nn_swz(t)) + 16 * (lp & 1)) = vb[s][p];
          }
          __builtin_amdgcn_wave_barrier();
#pragma unroll
          for (int c = 0; c < 2; ++c) {
            bf16x8 fb[NB];
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) fb[nb] = nn_frag(bt, 32 * c, nb);
#pragma unroll
            for (int i = 0; i < RT; ++i) {
              const bf16x8 fa = X.get(scr + i * kSlot, c);
#pragma unroll
              for (int nb = 0; nb < NB; ++nb) acc[i][nb] = mfma_bf16_16x16x32(fa, fb[nb], acc[i][nb]);
            }
          }
          __builtin_amdgcn_wave_barrier();  // the tiles are read before the next block is stored
        });
  }
  __syncthreads();  // every wave has left its scratch
  float* ps = (float*)lds;
  put_partials<RT, NB>(ps, wave, acc);
  __syncthreads();
  for (int pi = tid; pi < TM * TN; pi += 64 * NW) {
    const int ml = pi / TN, nl = pi % TN;
    const int m = m0 + ml;
    if (m >= M) continue;
    const float s = sum_partials<RT, NB, NW>(ps, ml, nl);
    const size_t o = (size_t)m * N + n0 + nl;
    a.out[o] = a.add ? a.add[o] + s : s;
  }
}

// ---- the residual MLP layer -------------------------------------------------
//
// z_l = y_l W_l^T + b_l over a 64 x 64 tile (rows x output columns).
// Forward: y_{l+1} = y_l + relu(z_l).  Adjoint (recomputation of layer l):
// ybar_{l+1} = nn_in (= ybar_{l+2} + zbar_{l+1} W_{l+1}, from the product
// launch before it) plus the loss seed; zbar_l = ybar_{l+1} 1[z_l > 0].
template <int MODE, int NW = kWaves, int S = 2>
__global__ __launch_bounds__(64 * NW) void mlp_wide(MlpArgs a) {
  constexpr int RT = 4, NB = 4, TM = 64, TN = 64;
  constexpr int SCR = (RT + NB) * kSlot;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int B = a.B, w = a.w;
  const int mg = (B + TM - 1) / TM, ntile = mg * (w / TN);
  const int tile = tile_of(ntile);
  if (tile >= ntile) return;
  const int m0 = (tile % mg) * TM, n0 = (tile / mg) * TN;

  __shared__ __attribute__((aligned(16))) char lds[lds_bytes<RT, NB, SCR, NW>()];
  float* ps = (float*)lds;
  {
    f4 acc[RT][NB];
#pragma unroll
    for (int i = 0; i < RT; ++i)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) acc[i][nb] = f4{0.f, 0.f, 0.f, 0.f};
    Xpose X;
    X.init();
    const int nbk = w / 64;
    const int c0 = (nbk * wave) / NW, c1 = (nbk * (wave + 1)) / NW;
    const Rows ys = rows_of(a.y, unsigned(size_t(B) * w * 2), m0, 2 * w);  // < 4 GiB: mlp_wide_fits
    const Rows ws = rows_of(a.W, unsigned(size_t(w) * w * 2), n0, 2 * w);
    nt_rows<RT, NB, S>(
        c0, c1, lds + wave * SCR, X, acc, [&](int g, int h, int blk) -> u4v { return ys.load(g, h, blk); },
        [&](int g, int h, int blk) -> u4v { return ws.load(g, h, blk); });
    __syncthreads();  // every wave has left its scratch
    put_partials<RT, NB>(ps, wave, acc);
  }
  __syncthreads();

  float lterm = 0.f;
  for (int pi = tid; pi < TM * TN; pi += 64 * NW) {
    const int ml = pi / TN, nl = pi % TN;
    const int m = m0 + ml, c = n0 + nl;
    if (m >= B) continue;
    const size_t o = (size_t)m * w + c;
    const float z = sum_partials<RT, NB, NW>(ps, ml, nl) + a.bias[c];
    const float yv = (float)((const __bf16*)a.y)[o];
    const __bf16 y1s = (__bf16)(yv + fmaxf(z, 0.f));
    if (MODE == kForward) {
      ((__bf16*)a.y_out)[o] = y1s;
    } else {
      const float hl = (float)y1s;  // the loss reads the stored y_{l+1}
      float yb;
      if (a.first) {
        if (a.loss == AMBPTT_LOSS_HALF_SQ_LAST) {
          yb = hl;
          lterm += hl * hl;
        } else if (a.loss == AMBPTT_LOSS_MEAN_LAST) {
          yb = a.inv_bw;
          lterm += hl;
        } else {
          yb = 2.f * hl * a.inv_bw;
          lterm += hl * hl;
        }
      } else {
        yb = a.nn_in[o];
        if (a.loss == AMBPTT_LOSS_MEAN_SQ_ALL) {
          yb += 2.f * hl * a.inv_bw;
          lterm += hl * hl;
        }
      }
      a.ybar_out[o] = yb;
      ((__bf16*)a.zbar_out)[o] = (__bf16)(z > 0.f ? yb : 0.f);
      ((__bf16*)a.ywin_out)[o] = ((const __bf16*)a.y)[o];
    }
  }
  if (MODE == kAdjoint) {
    const float s = wave_sum(lterm);
    __shared__ float wsum[NW];
    if (lane == 0) wsum[wave] = s;
    __syncthreads();
    if (tid == 0) {
      float t = 0.f;
#pragma unroll
      for (int wv = 0; wv < NW; ++wv) t += wsum[wv];
      a.loss_acc[tile] += (double)t;
    }
  }
}

unsigned grid_for(int ntile) { return unsigned(8 * ((ntile + 7) / 8)); }

// dst (fragment order, Frags) <- the [N][K] rows of src (row stride ld): one
// thread per 16-byte lane chunk, written in order.
__global__ __launch_bounds__(256) void pack_nt(const char* __restrict__ src, int K, int ld, size_t chunks,
                                               char* __restrict__ dst) {
  const size_t t = size_t(blockIdx.x) * 256 + threadIdx.x;
  if (t >= chunks) return;
  const int l = int(t & 63);
  const size_t f = t >> 6, kf = size_t(K / 32);
  const size_t jt = f / kf, ks = f % kf;
  const size_t row = 16 * jt + size_t(l & 15), col = 32 * ks + 8 * size_t(l >> 4);
  *(u4v*)(dst + 16 * t) = *(const u4v*)(src + 2 * (row * size_t(ld) + col));
}

}  // namespace

hipError_t launch_pack_nt_bf16(const void* src, int N, int K, int ld, void* dst, hipStream_t s) {
  if (N < 16 || N % 16 != 0 || K < 32 || K % 32 != 0 || ld < K || ld % 8 != 0 ||
      size_t(N) * size_t(K) * 2 > 0xFFFFFFFFull)  // Frags addresses the copy with 32-bit offsets
    return hipErrorInvalidValue;
  const size_t chunks = size_t(N) * size_t(K) / 8;
  hipLaunchKernelGGL(pack_nt, dim3(unsigned((chunks + 255) / 256)), dim3(256), 0, s, (const char*)src, K, ld, chunks,
                     (char*)dst);
  return hipGetLastError();
}

// Every operand is addressed with 32-bit buffer offsets: each must stay under 4 GiB.
static bool under_4g(size_t rows, size_t cols) { return rows * cols * 2 <= 0xFFFFFFFFull; }

bool cell_wide_fits(int G, int B, int D, int H) {
  return D % 64 == 0 && H % 64 == 0 && H > 0 && B > 0 && under_4g(size_t(B), size_t(D) + size_t(H)) &&
         under_4g(size_t(G) * H, size_t(D) + size_t(H)) && under_4g(size_t(B), size_t(G) * H);
}

bool mlp_wide_fits(int B, int w) { return w % 64 == 0 && w > 0 && B > 0 && under_4g(size_t(w), size_t(w)) && under_4g(size_t(B), size_t(w)); }

int cell_wide_tiles(int G, int B, int H) { return ((B + 63) / 64) * (H / (64 / G)); }

hipError_t launch_cell_wide(int G, int mode, const StepArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if ((mode != kForward && mode != kAdjoint) || !cell_wide_fits(G, a.B, a.D, a.H)) return hipErrorInvalidValue;
  const dim3 grid(grid_for(cell_wide_tiles(G, a.B, a.H))), block(64 * kWaves);
  if (G == 4) {
    if (mode == kForward) hipExtLaunchKernelGGL((cell_wide<4, kForward>), grid, block, 0, s, e0, e1, 0, a);
    else hipExtLaunchKernelGGL((cell_wide<4, kAdjoint>), grid, block, 0, s, e0, e1, 0, a);
  } else {
    if (mode == kForward) hipExtLaunchKernelGGL((cell_wide<1, kForward>), grid, block, 0, s, e0, e1, 0, a);
    else hipExtLaunchKernelGGL((cell_wide<1, kAdjoint>), grid, block, 0, s, e0, e1, 0, a);
  }
  return hipGetLastError();
}

bool prod_wide_big(int M, int N) { return N % 32 == 0 && ((M + 31) / 32) * (N / 32) >= 192; }

hipError_t launch_prod_nt(const ProdArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if (a.K % 64 != 0 || a.N % 16 != 0 || a.M < 1) return hipErrorInvalidValue;
  const dim3 block(64 * kWaves);
  if (prod_wide_big(a.M, a.N)) {
    const dim3 grid(grid_for(((a.M + 31) / 32) * (a.N / 32)));
    hipExtLaunchKernelGGL((prod_wide<2, 2, false>), grid, block, 0, s, e0, e1, 0, a);
  } else {
    const dim3 grid(grid_for(((a.M + 15) / 16) * (a.N / 16)));
    hipExtLaunchKernelGGL((prod_wide<1, 1, false>), grid, block, 0, s, e0, e1, 0, a);
  }
  return hipGetLastError();
}

hipError_t launch_prod_nn(const ProdArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if (a.K % 64 != 0 || a.N % 64 != 0 || a.M < 1) return hipErrorInvalidValue;
  const dim3 grid(grid_for(((a.M + 63) / 64) * (a.N / 64))), block(64 * kWaves);
  hipExtLaunchKernelGGL((prod_wide<4, 4, true>), grid, block, 0, s, e0, e1, 0, a);
  return hipGetLastError();
}

int mlp_wide_tiles(int B, int w) { return ((B + 63) / 64) * (w / 64); }

hipError_t launch_mlp_wide(int mode, const MlpArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if (!mlp_wide_fits(a.B, a.w)) return hipErrorInvalidValue;
  const dim3 grid(grid_for(mlp_wide_tiles(a.B, a.w))), block(64 * kWaves);
  if (mode == kForward) hipExtLaunchKernelGGL((mlp_wide<kForward>), grid, block, 0, s, e0, e1, 0, a);
  else if (mode == kAdjoint) hipExtLaunchKernelGGL((mlp_wide<kAdjoint>), grid, block, 0, s, e0, e1, 0, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace ambptt
