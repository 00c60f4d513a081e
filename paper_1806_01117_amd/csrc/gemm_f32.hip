// LDS-tiled fp32 kernels for the large-batch recurrent cells on gfx950
// (v_mfma_f32_16x16x4_f32): the forward step and the adjoint's gate
// recomputation of a tanh RNN (G = 1) or LSTM (G = 4) with the cell epilogue
// fused, and the adjoint's h-adjoint product hbar = zbar W_h.
//
// Both are "NT" products whose operands are contiguous in the reduction
// index k:
//   gate product  z[m][n] = sum_k [x | h][m][k] W[n][k]       (K = D + H)
//   h-adjoint     hbar[m][j] = sum_k zbar[m][k] WhT[j][k]     (K = G H)
// A workgroup of 4 waves owns one output tile, and two workgroups share a
// CU (each holds one LDS buffer of 64-wide stages, under 80 KB), so that
// while one workgroup waits at a barrier or on LDS the other keeps the
// matrix cores busy.  A stage is loaded into registers while the previous
// one is multiplied, written to LDS between the stage's two barriers, and
// multiplied from there.  Reduction indices past K read as zero.  LDS rows
// are padded by 4 floats, so that the 16 rows one MFMA operand read touches
// (16 bytes each, at one column) fall on distinct banks.
//
// Fragments: lane l reads 4 consecutive k of row l & 15 at column 4 (l >> 4)
// of a 16-wide chunk, and its 4 components feed 4 MFMAs; A and B use the
// same mapping, so the 4 MFMAs together cover the chunk.
//
// Tiles are placed XCD-aware: workgroup i runs on XCD i % 8, and the row
// tiles that read the same weight rows are given consecutive slots of one
// XCD, so the weights stream from HBM once per launch and are shared through
// that XCD's L2.
#include <hip/hip_runtime.h>

#include "ambptt.h"
#include "kernels.hpp"

namespace ambptt {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f4 mfma4(float a, float b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float sigm(float z) { return 1.0f / (1.0f + __expf(-z)); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// (row tile, column tile) of workgroup i: the mt row tiles of one column tile
// share an XCD when the column tiles divide evenly over the 8 XCDs.
__device__ __forceinline__ void tile_of(int i, int mt, int nt, int* tm, int* tn) {
  if (nt % 8 == 0) {
    const int xcd = i & 7, k = i >> 3;
    *tn = xcd * (nt >> 3) + k / mt;
    *tm = k % mt;
  } else {
    *tm = i % mt;
    *tn = i / mt;
  }
}

// ---- epilogue of the gate product: one wave's 64 x 64 accumulators ----------
// Accumulator element v of lane l is row 4 (l >> 4) + v, column l & 15 of its
// 16 x 16 block.  Forward: the cell update; adjoint: loss term (returned),
// seed, cell adjoint, zbar_t, cbar_t and the copy of h_t.
template <int G, int MODE>
__device__ __forceinline__ float cell_epilogue(const StepArgs& a, const f4 (&acc)[4][4], int m0, int j0, int wm,
                                               int wn, int r, int q) {
  const int B = a.B, H = a.H, GH = G * H;
  float lterm = 0.f;
  constexpr int NU = G == 4 ? 1 : 4;  // unit blocks per wave
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int u = 0; u < NU; ++u)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int m = m0 + wm * 64 + 16 * i + 4 * q + v;
        const int j = G == 4 ? j0 + wn * 16 + r : j0 + wn * 64 + 16 * u + r;
        if (m >= B) continue;
        const size_t o = (size_t)m * H + j;
        float h1, c1 = 0.f, tc = 0.f, ig = 0.f, fg = 0.f, gg = 0.f, og = 0.f, cold = 0.f;
        if (G == 4) {
          ig = sigm(acc[i][0][v] + a.bias[j]);
          fg = sigm(acc[i][1][v] + a.bias[H + j]);
          gg = tanhf(acc[i][2][v] + a.bias[2 * H + j]);
          og = sigm(acc[i][3][v] + a.bias[3 * H + j]);
          cold = a.c[o];
          c1 = fg * cold + ig * gg;
          tc = tanhf(c1);
          h1 = og * tc;
        } else {
          h1 = tanhf(acc[i][u][v] + a.bias[j]);
        }
        if (MODE == kForward) {
          ((float*)a.h_out)[o] = h1;
          if (G == 4) a.c_out[o] = c1;
          continue;
        }
        // adjoint: loss term of h_{t+1} and its seed dL/dh_{t+1}
        float sd = 0.f;
        if (a.loss == AMBPTT_LOSS_MEAN_SQ_ALL) {
          sd = 2.f * h1 * a.inv_bh;
          lterm += h1 * h1;
        } else if (a.last) {
          if (a.loss == AMBPTT_LOSS_HALF_SQ_LAST) {
            sd = h1;
            lterm += h1 * h1;
          } else {
            sd = a.inv_bh;
            lterm += h1;
          }
        }
        float hin = 0.f;
        if (!a.first) {  // the product's partial sums, in order
          hin = a.hbar_in[o];
          for (int ps = 1; ps < a.hbar_parts; ++ps) hin += a.hbar_in[o + (size_t)ps * B * H];
        }
        const float hb = hin + sd;
        float* zo = (float*)a.zbar_out + (size_t)m * GH + j;
        if (G == 4) {
          const float cb = a.first ? 0.f : a.cbar_in[o];
          const float ob = hb * tc;
          const float ch = cb + hb * og * (1.f - tc * tc);
          zo[0] = ch * gg * ig * (1.f - ig);
          zo[H] = ch * cold * fg * (1.f - fg);
          zo[2 * H] = ch * ig * (1.f - gg * gg);
          zo[3 * H] = ob * og * (1.f - og);
          a.cbar_out[o] = ch * fg;
        } else {
          zo[0] = hb * (1.f - h1 * h1);
        }
        ((float*)a.hwin_out)[o] = ((const float*)a.h)[o];
      }
  return lterm;
}

// ---- gate product with the cell epilogue ------------------------------------
// Tile: 128 batch rows x 128 gate columns (LSTM: 32 units x 4 gates; RNN:
// 128 units), 4 waves.  Wave (wm, wn), wm, wn < 2, computes rows
// 64 wm .. + 63 and, for the LSTM, units 16 wn .. + 15 of all four gates
// (block g of its 4 x 4 blocks of 16 x 16 is gate g), so a lane holds the
// four gates of its (row, unit) pairs in the same accumulator element; for
// the RNN units 64 wn .. + 63.
constexpr int kCM = 128, kCN = 128, kKT = 64, kLd = kKT + 4, kCW = 4;

template <int G, int MODE>
__global__ __launch_bounds__(64 * kCW, 2) void cell_gemm_f32(StepArgs a) {
  __shared__ float As[kCM][kLd];
  __shared__ float Bs[kCN][kLd];
  __shared__ float red[kCW];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int r = lane & 15, q = lane >> 4;
  const int B = a.B, D = a.D, H = a.H, K1 = D + H;
  const int mt = (B + kCM - 1) / kCM, nt = G * H / kCN;
  int tm, tn;
  tile_of(blockIdx.x, mt, nt, &tm, &tn);
  const int m0 = tm * kCM;
  const int j0 = tn * (kCN / G);  // first unit of the tile

  // loader: thread t moves rows t / 16 + 16 p, float4 column t % 16 of a
  // stage; a float4 lies wholly in x or in h (D, H multiples of 4)
  const int lr = tid >> 4, lc = 4 * (tid & 15);
  const float* x = (const float*)a.x;
  const float* h = (const float*)a.h;
  const float* W = (const float*)a.W;
  int arow[8];
#pragma unroll
  for (int p = 0; p < 8; ++p) arow[p] = min(m0 + lr + 16 * p, B - 1);  // rows >= B: clamped, discarded
  const float* brow[8];
#pragma unroll
  for (int p = 0; p < 8; ++p) {
    const int c = lr + 16 * p;
    const int n = G == 4 ? (c >> 5) * H + j0 + (c & 31) : j0 + c;
    brow[p] = W + (size_t)n * K1;
  }
  // Every load is unconditional (a lane past K reads column 0 of its row),
  // so that no branch splits the stage's loads; past K the values are
  // replaced by zero when they are written to LDS.
  f4 ra[8], rb[8];
  bool kin = true;
  auto load = [&](int st) {
    const int k = st * kKT + lc;
    kin = k < K1;
    const int kc = kin ? k : 0;
    const bool inx = kc < D;
#pragma unroll
    for (int p = 0; p < 8; ++p) {
      const float* src = inx ? x + (size_t)arow[p] * D + kc : h + (size_t)arow[p] * H + (kc - D);
      ra[p] = *(const f4*)src;
    }
#pragma unroll
    for (int p = 0; p < 8; ++p) rb[p] = *(const f4*)(brow[p] + kc);
  };
  auto store = [&]() {
    const f4 zero = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int p = 0; p < 8; ++p) *(f4*)&As[lr + 16 * p][lc] = kin ? ra[p] : zero;
#pragma unroll
    for (int p = 0; p < 8; ++p) *(f4*)&Bs[lr + 16 * p][lc] = kin ? rb[p] : zero;
  };

  f4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) acc[i][nb] = f4{0.f, 0.f, 0.f, 0.f};
  // LDS row of B block nb of this wave
  int bcol[4];
#pragma unroll
  for (int nb = 0; nb < 4; ++nb) bcol[nb] = G == 4 ? nb * 32 + wn * 16 : wn * 64 + 16 * nb;

  auto compute = [&]() {
#pragma unroll
    for (int kk = 0; kk < kKT / 16; ++kk) {
      f4 af[4], bf[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) af[i] = *(const f4*)&As[wm * 64 + 16 * i + r][16 * kk + 4 * q];
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) bf[nb] = *(const f4*)&Bs[bcol[nb] + r][16 * kk + 4 * q];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) {
          acc[i][nb] = mfma4(af[i].x, bf[nb].x, acc[i][nb]);
          acc[i][nb] = mfma4(af[i].y, bf[nb].y, acc[i][nb]);
          acc[i][nb] = mfma4(af[i].z, bf[nb].z, acc[i][nb]);
          acc[i][nb] = mfma4(af[i].w, bf[nb].w, acc[i][nb]);
        }
    }
  };
  // The next stage's global loads are issued before the multiplications
  // start (the scheduling barriers keep the compiler from sinking them below
  // the MFMAs); the first barrier of a stage waits for every wave to finish
  // reading the previous one.
  const int nst = (K1 + kKT - 1) / kKT;
  load(0);
  for (int st = 0; st < nst; ++st) {
    if (st) __syncthreads();
    store();
    if (st + 1 < nst) load(st + 1);
    __syncthreads();
    __builtin_amdgcn_sched_barrier(0);
    compute();
    __builtin_amdgcn_sched_barrier(0);
  }

  const float lterm = cell_epilogue<G, MODE>(a, acc, m0, j0, wm, wn, r, q);
  if (MODE == kAdjoint) {  // the waves' loss terms, summed in wave order
    const float s = wave_sum(lterm);
    if (lane == 0) red[wave] = s;
    __syncthreads();
    if (tid == 0) {
      double t = 0.0;
      for (int w = 0; w < kCW; ++w) t += (double)red[w];
      a.loss_acc[blockIdx.x] += t;
    }
  }
}

// ---- h-adjoint product: out = A B^T (+ add) -----------------------------------
// Tile: 64 rows x 64 columns; wave (wm, wn) computes rows 32 wm .. + 31 and
// columns 32 wn .. + 31 (2 x 2 blocks); stages of kPT = 64 reduction indices.
// The 4 MFMAs of one k-component run over all 4 blocks before the next
// component, so consecutive MFMAs never share an accumulator.
constexpr int kPM = 64, kPN = 64, kPT = 64, kPLd = kPT + 4;

__global__ __launch_bounds__(256, 2) void prod_gemm_f32(ProdArgs a) {
  __shared__ float As[kPM][kPLd];
  __shared__ float Bs[kPN][kPLd];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int r = lane & 15, q = lane >> 4;
  const int M = a.M, N = a.N, K = a.K;
  const int mt = (M + kPM - 1) / kPM, nt = N / kPN;
  int tm, tn;
  tile_of(blockIdx.x, mt, nt, &tm, &tn);
  const int m0 = tm * kPM, n0 = tn * kPN;

  // loader: thread t moves rows t / 16 + 16 p, float4 column t % 16 of a stage
  const int lr = tid >> 4, lc = 4 * (tid & 15);
  const float* arow[4];
  const float* brow[4];
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    arow[p] = (const float*)a.A + (size_t)min(m0 + lr + 16 * p, M - 1) * K;  // rows >= M: clamped, discarded
    brow[p] = (const float*)a.B + (size_t)(n0 + lr + 16 * p) * (a.ldb ? a.ldb : K);
  }
  f4 ra[4], rb[4];
  bool kin = true;
  auto load = [&](int st) {  // unconditional loads, as in the gate product
    const int k = st * kPT + lc;
    kin = k < K;
    const int kc = kin ? k : 0;
#pragma unroll
    for (int p = 0; p < 4; ++p) ra[p] = *(const f4*)(arow[p] + kc);
#pragma unroll
    for (int p = 0; p < 4; ++p) rb[p] = *(const f4*)(brow[p] + kc);
  };
  auto store = [&]() {
    const f4 zero = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int p = 0; p < 4; ++p) *(f4*)&As[lr + 16 * p][lc] = kin ? ra[p] : zero;
#pragma unroll
    for (int p = 0; p < 4; ++p) *(f4*)&Bs[lr + 16 * p][lc] = kin ? rb[p] : zero;
  };

  f4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
  auto compute = [&]() {
#pragma unroll
    for (int kk = 0; kk < kPT / 16; ++kk) {
      f4 af[2], bf[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) af[i] = *(const f4*)&As[wm * 32 + 16 * i + r][16 * kk + 4 * q];
#pragma unroll
      for (int j = 0; j < 2; ++j) bf[j] = *(const f4*)&Bs[wn * 32 + 16 * j + r][16 * kk + 4 * q];
#pragma unroll
      for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j) acc[i][j] = mfma4(af[i][c], bf[j][c], acc[i][j]);
    }
  };
  const int nst = (K + kPT - 1) / kPT;
  load(0);
  for (int st = 0; st < nst; ++st) {
    if (st) __syncthreads();
    store();
    if (st + 1 < nst) load(st + 1);
    __syncthreads();
    __builtin_amdgcn_sched_barrier(0);
    compute();
    __builtin_amdgcn_sched_barrier(0);
  }
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int m = m0 + wm * 32 + 16 * i + 4 * q + v;
      if (m >= M) continue;
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const size_t o = (size_t)m * N + n0 + wn * 32 + 16 * j + r;
        a.out[o] = a.add ? a.add[o] + acc[i][j][v] : acc[i][j][v];
      }
    }
}

// ---- h-adjoint product on the gate product's tiles, the reduction split ---------
// The 64 x 64 tiles above give the 4096-LSTM's product (512 x 4096 outputs)
// 512 workgroups, but move twice the operand rows per MFMA of the 128 x 128
// tiles.  Here each of the 128 x 128 tiles takes `parts` workgroups, one per
// contiguous run of stages, so the grid keeps two workgroups per CU; part s
// is written whole to out + s M N and the adjoint adds the parts in order.
// Loader, LDS layout, fragments and stage loop are the gate product's (wave
// (wm, wn): rows 64 wm .., columns 64 wn ..).  The row tiles of one
// (column tile, part) share an XCD, as the gate product's do.
__global__ __launch_bounds__(64 * kCW, 2) void prod_split_f32(ProdArgs a, int parts) {
  __shared__ float As[kCM][kLd];
  __shared__ float Bs[kCN][kLd];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int r = lane & 15, q = lane >> 4;
  const int M = a.M, N = a.N, K = a.K;
  const int mt = (M + kCM - 1) / kCM, nt = N / kCN;
  int tm, tc;
  tile_of(blockIdx.x, mt, nt * parts, &tm, &tc);
  const int tn = tc / parts, part = tc % parts;
  const int m0 = tm * kCM, n0 = tn * kCN;
  const int nall = (K + kKT - 1) / kKT;
  const int st0 = part * nall / parts, st1 = (part + 1) * nall / parts;

  const int lr = tid >> 4, lc = 4 * (tid & 15);
  const float* arow[8];
  const float* brow[8];
#pragma unroll
  for (int p = 0; p < 8; ++p) {
    arow[p] = (const float*)a.A + (size_t)min(m0 + lr + 16 * p, M - 1) * K;  // rows >= M: clamped, discarded
    brow[p] = (const float*)a.B + (size_t)(n0 + lr + 16 * p) * (a.ldb ? a.ldb : K);
  }
  f4 ra[8], rb[8];
  bool kin = true;
  auto load = [&](int st) {  // unconditional loads, as in the gate product
    const int k = st * kKT + lc;
    kin = k < K;
    const int kc = kin ? k : 0;
#pragma unroll
    for (int p = 0; p < 8; ++p) ra[p] = *(const f4*)(arow[p] + kc);
#pragma unroll
    for (int p = 0; p < 8; ++p) rb[p] = *(const f4*)(brow[p] + kc);
  };
  auto store = [&]() {
    const f4 zero = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int p = 0; p < 8; ++p) *(f4*)&As[lr + 16 * p][lc] = kin ? ra[p] : zero;
#pragma unroll
    for (int p = 0; p < 8; ++p) *(f4*)&Bs[lr + 16 * p][lc] = kin ? rb[p] : zero;
  };
  f4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) acc[i][nb] = f4{0.f, 0.f, 0.f, 0.f};
  auto compute = [&]() {
#pragma unroll
    for (int kk = 0; kk < kKT / 16; ++kk) {
      f4 af[4], bf[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) af[i] = *(const f4*)&As[wm * 64 + 16 * i + r][16 * kk + 4 * q];
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) bf[nb] = *(const f4*)&Bs[wn * 64 + 16 * nb + r][16 * kk + 4 * q];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) {
          acc[i][nb] = mfma4(af[i].x, bf[nb].x, acc[i][nb]);
          acc[i][nb] = mfma4(af[i].y, bf[nb].y, acc[i][nb]);
          acc[i][nb] = mfma4(af[i].z, bf[nb].z, acc[i][nb]);
          acc[i][nb] = mfma4(af[i].w, bf[nb].w, acc[i][nb]);
        }
    }
  };
  if (st0 < st1) load(st0);
  for (int st = st0; st < st1; ++st) {
    if (st > st0) __syncthreads();
    store();
    if (st + 1 < st1) load(st + 1);
    __syncthreads();
    __builtin_amdgcn_sched_barrier(0);
    compute();
    __builtin_amdgcn_sched_barrier(0);
  }
  float* out = a.out + (size_t)part * M * N;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int m = m0 + wm * 64 + 16 * i + 4 * q + v;
      if (m >= M) continue;
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) out[(size_t)m * N + n0 + wn * 64 + 16 * nb + r] = acc[i][nb][v];
    }
}

}  // namespace

bool cell_gemm_f32_fits(int G, int B, int D, int H) {
  return (G == 1 || G == 4) && B >= 1 && D >= 0 && D % 4 == 0 && H >= 1 && H % 4 == 0 && (G * H) % kCN == 0;
}

int cell_gemm_f32_tiles(int G, int B, int H) { return ((B + kCM - 1) / kCM) * (G * H / kCN); }

hipError_t launch_cell_gemm_f32(int G, int mode, const StepArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if (!cell_gemm_f32_fits(G, a.B, a.D, a.H) || (mode == kAdjoint && !a.first && !a.hbar_in)) return hipErrorInvalidValue;
  const dim3 grid(cell_gemm_f32_tiles(G, a.B, a.H)), block(64 * kCW);
  if (G == 4) {
    if (mode == kForward) hipExtLaunchKernelGGL((cell_gemm_f32<4, kForward>), grid, block, 0, s, e0, e1, 0, a);
    else if (mode == kAdjoint) hipExtLaunchKernelGGL((cell_gemm_f32<4, kAdjoint>), grid, block, 0, s, e0, e1, 0, a);
    else return hipErrorInvalidValue;
  } else {
    if (mode == kForward) hipExtLaunchKernelGGL((cell_gemm_f32<1, kForward>), grid, block, 0, s, e0, e1, 0, a);
    else if (mode == kAdjoint) hipExtLaunchKernelGGL((cell_gemm_f32<1, kAdjoint>), grid, block, 0, s, e0, e1, 0, a);
    else return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

bool prod_gemm_f32_fits(int M, int N, int K) { return M >= 1 && K >= 4 && K % 4 == 0 && N >= kPN && N % kPN == 0; }

int prod_gemm_f32_tiles(int M, int N) { return ((M + kPM - 1) / kPM) * (N / kPN); }

hipError_t launch_prod_gemm_f32(const ProdArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if (!prod_gemm_f32_fits(a.M, a.N, a.K)) return hipErrorInvalidValue;
  const dim3 grid(prod_gemm_f32_tiles(a.M, a.N)), block(256);
  hipExtLaunchKernelGGL(prod_gemm_f32, grid, block, 0, s, e0, e1, 0, a);
  return hipGetLastError();
}

int prod_split_f32_parts(int M, int N, int K) {
  if (M < 1 || K < 4 || K % 4 || N < kCN || N % kCN) return 1;
  const int tiles = ((M + kCM - 1) / kCM) * (N / kCN);
  int parts = 1;  // two workgroups per CU, each with at least 16 stages
  while (parts < kProdSplitMax && tiles * parts < 512 && (K / kKT) / (2 * parts) >= 16) parts *= 2;
  return parts;
}

hipError_t launch_prod_split_f32(const ProdArgs& a, int parts, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if (parts < 1 || parts > kProdSplitMax || a.add || a.M < 1 || a.K < 4 || a.K % 4 || a.N < kCN || a.N % kCN)
    return hipErrorInvalidValue;
  const dim3 grid(((a.M + kCM - 1) / kCM) * (a.N / kCN) * parts), block(64 * kCW);
  hipExtLaunchKernelGGL(prod_split_f32, grid, block, 0, s, e0, e1, 0, a, parts);
  return hipGetLastError();
}

}  // namespace ambptt
