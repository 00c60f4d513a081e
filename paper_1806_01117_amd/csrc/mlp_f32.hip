// An MLP whose layers change width, treated as a sequence (depth = steps):
// the states y_l [B][w_l] differ in size from layer to layer, the case the
// paper's Sections 1.1 and 6 set beside Revolve's uniform states.  fp32 on
// gfx950 (v_mfma_f32_16x16x4_f32).
//
//   forward   y_{l+1} = relu(z_l),  z_l = y_l W_l^T + b_l,  W_l[w_{l+1}][w_l]
//   adjoint   ybar_{l+1} = u + dL/dy_{l+1},  u = zbar_{l+1} W_{l+1} (0 for the last layer)
//             zbar_l = ybar_{l+1} * 1[z_l > 0]   (relu'(0) = 0)
//   product   u = zbar W  (an "NN" product: W[k][c] is contiguous in c)
//   gradient  dW_l = zbar_l^T y_l,  db_l = column sums of zbar_l (mlpv_dw, a window of layers per launch)
//
// One launch per step: the forward, the NN product alone (dL/dy_0), and the
// adjoint, which also forms u for its own tile.  A workgroup of 16 waves owns
// 32 x 32 outputs, its waves split the reduction, and the partial tiles meet
// in LDS in wave order (deterministic).  Widths are multiples of 16; a tile's
// second column block may fall past N and then idles.  The loss terms of a
// workgroup are summed in a fixed order by its first thread.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "ambptt.h"
#include "kernels.hpp"

namespace ambptt {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f4 mfma4(float a, float b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

enum { kMlpvFwd = 0, kMlpvAdj = 1, kMlpvNN = 2, kMlpvAdjU = 3 };

constexpr int kVW = 16;  // waves per workgroup

struct MlpvTile {
  int tid, lane, wave, r, q, m0, n0;
};

// TileProduct: acc[i][j] = the wave's share of A[m0 + 16 i ..][:] . B[:][n0 + 16 j ..], i < RT, for
// A [M][K] row-major and B = W^T (NT: W [N][K]) or B = W (NN: W [K][N]).
// Wave w takes chunks w, w + 16, ... of 16 reduction indices in groups of ND
// whose loads all issue before the group's first MFMA; past the last chunk
// the operands read the last one and are zeroed before use, so every wave
// issues the same loads in straight line.  Lane l reads 4 consecutive k of
// row l & 15 at 4 (l >> 4) and its components feed 4 MFMAs (A and the NT B
// the same way).  The NN B chunk (16 reduction rows x 32 columns) is read as
// whole 128-byte rows, 8 lanes a row, and turned into fragments through the
// wave's own tile bt in LDS (rows of 36 floats: the column reads of a
// fragment fall in 64 distinct banks).  With ywin, the first column of
// workgroups also writes a copy of its A rows there.
template <bool NN, int ND, int RT>
struct TileProduct {
  const float* arow[RT];
  const float* brow[2];
  const float* wnn;
  int M, N, K, nch, ngrp, nrow, ncol;
  __device__ __forceinline__ TileProduct(const MlpvTile& t, const float* __restrict__ A, const float* __restrict__ W,
                                         int M_, int N_, int K_)
      : M(M_), N(N_), K(K_) {
    nch = K / 16;
    ngrp = (nch + kVW * ND - 1) / (kVW * ND);  // groups of ND chunks per wave
#pragma unroll
    for (int i = 0; i < RT; ++i) arow[i] = A + (size_t)min(t.m0 + 16 * i + t.r, M - 1) * K + 4 * t.q;  // rows >= M: clamped, discarded
#pragma unroll
    for (int j = 0; j < 2; ++j) brow[j] = W + (size_t)min(t.n0 + 16 * j + t.r, N - 1) * K + 4 * t.q;  // NT; past N: clamped, discarded
    nrow = t.lane >> 3;
    ncol = 4 * (t.lane & 7);
    wnn = W + min(t.n0 + ncol, N - 4);  // NN: a float4 past N: clamped, discarded
  }
  // the loads of group g of the wave's chunks
  __device__ __forceinline__ void load(const MlpvTile& t, int g, f4 (&xa)[ND][RT], f4 (&xb)[ND][2]) const {
#pragma unroll
    for (int u = 0; u < ND; ++u) {
      const int k0 = 16 * min(t.wave + kVW * (ND * g + u), nch - 1);
#pragma unroll
      for (int i = 0; i < RT; ++i) xa[u][i] = *(const f4*)(arow[i] + k0);
#pragma unroll
      for (int j = 0; j < 2; ++j)
        xb[u][j] = NN ? *(const f4*)(wnn + (size_t)(k0 + nrow + 8 * j) * N) : *(const f4*)(brow[j] + k0);
    }
  }
  // group g's MFMAs into acc (and the copy of A's rows into ywin)
  __device__ __forceinline__ void mma(const MlpvTile& t, int g, f4 (&xa)[ND][RT], f4 (&xb)[ND][2],
                                      float (&bt)[16][36], float* ywin, f4 (&acc)[RT][2]) const {
    const int r = t.r, q = t.q;
#pragma unroll
    for (int u = 0; u < ND; ++u) {
      const int c = t.wave + kVW * (ND * g + u);
      if (NN) {  // raw rows nrow, nrow + 8 -> fragments of columns n0 + 16 j + r, rows 4 q .. 4 q + 3
#pragma unroll
        for (int h = 0; h < 2; ++h) *(f4*)&bt[nrow + 8 * h][ncol] = xb[u][h];
#pragma unroll
        for (int j = 0; j < 2; ++j)
          xb[u][j] = f4{bt[4 * q][16 * j + r], bt[4 * q + 1][16 * j + r], bt[4 * q + 2][16 * j + r], bt[4 * q + 3][16 * j + r]};
      }
      if (c >= nch) {  // uniform: a chunk past the reduction adds nothing
#pragma unroll
        for (int i = 0; i < RT; ++i) xa[u][i] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int j = 0; j < 2; ++j) xb[u][j] = f4{0.f, 0.f, 0.f, 0.f};
      }
#pragma unroll
      for (int k = 0; k < 4; ++k)
#pragma unroll
        for (int i = 0; i < RT; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j) acc[i][j] = mfma4(xa[u][i][k], xb[u][j][k], acc[i][j]);
      if (ywin && blockIdx.y == 0) {
#pragma unroll
        for (int i = 0; i < RT; ++i)
          if (c < nch && t.m0 + 16 * i + r < M) *(f4*)(ywin + (size_t)(t.m0 + 16 * i + r) * K + 16 * c + 4 * q) = xa[u][i];
      }
    }
  }
  // the whole product; with pre, group 0's loads were issued already into xa0, xb0
  __device__ __forceinline__ void run(const MlpvTile& t, float (&bt)[16][36], float* ywin, f4 (&acc)[RT][2],
                                      f4 (*xa0)[RT] = nullptr, f4 (*xb0)[2] = nullptr) const {
#pragma unroll
    for (int i = 0; i < RT; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
    for (int g = 0; g < ngrp; ++g) {
      f4 xa[ND][RT], xb[ND][2];
      if (g == 0 && xa0) {
#pragma unroll
        for (int u = 0; u < ND; ++u) {
#pragma unroll
          for (int i = 0; i < RT; ++i) xa[u][i] = xa0[u][i];
#pragma unroll
          for (int j = 0; j < 2; ++j) xb[u][j] = xb0[u][j];
        }
      } else {
        load(t, g, xa, xb);
      }
      __builtin_amdgcn_sched_barrier(0);  // every load of the group issues before its first MFMA
      mma(t, g, xa, xb, bt, ywin, acc);
    }
  }
};

// The 16 waves' partial tiles summed in wave order: thread tid < 512 RT gets
// element (tid >> 5, tid & 31) of the 16 RT x 32 tile (the others get 0).
// Accumulator element v of lane l is row 4 (l >> 4) + v, column l & 15 of its
// 16 x 16 block.
template <int RT>
__device__ __forceinline__ float tile_sum(const MlpvTile& t, float (&part)[kVW][32][36], const f4 (&acc)[RT][2]) {
#pragma unroll
  for (int i = 0; i < RT; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) part[t.wave][16 * i + 4 * t.q + v][16 * j + t.r] = acc[i][j][v];
  __syncthreads();
  float sum = 0.f;
  if (t.tid < 512 * RT) {
#pragma unroll
    for (int w = 0; w < kVW; ++w) sum += part[w][t.tid >> 5][t.tid & 31];
  }
  return sum;
}

// One launch per step.  A workgroup of 16 waves owns 16 RT rows x 32 columns
// of the step's output (RT = 1 where 32-row tiles would leave the device
// short of workgroups); its first 512 RT threads run the epilogue, 32
// consecutive columns per half wave.  kMlpvAdjU runs the adjoint's two products in one launch:
// first u = zbar_{l+1} W_{l+1} (NN, reduction over w_{l+2}, with ND2), then
// z_l (NT, with ND), the LDS tiles reused in between.  Its u is summed in
// the same order as the NN launch's.
template <int MODE, int ND, int ND2, int RT>
__global__ __launch_bounds__(64 * kVW) void mlpv_gemm(MlpvArgs a) {
  __shared__ float part[kVW][32][36];  // partial tiles; rows of 36: the stores of a wave spread over the banks
  __shared__ __attribute__((aligned(16))) float bt[(MODE == kMlpvNN || MODE == kMlpvAdjU) ? kVW : 1][16][36];
  __shared__ float lpart[kVW];
  MlpvTile t;
  t.tid = threadIdx.x;
  t.lane = t.tid & 63;
  t.wave = __builtin_amdgcn_readfirstlane(t.tid >> 6);
  t.r = t.lane & 15;
  t.q = t.lane >> 4;
  t.m0 = blockIdx.x * 16 * RT;
  t.n0 = blockIdx.y * 32;
  const int M = a.M, N = a.N;
  const bool adj = MODE == kMlpvAdj || MODE == kMlpvAdjU;
  float u = 0.f;
  const TileProduct<MODE == kMlpvNN, ND, RT> main(t, a.A, a.W, M, N, a.K);
  f4 acc[RT][2];
  if (MODE == kMlpvAdjU) {
    f4 acc2[RT][2];
    TileProduct<true, ND2, RT>(t, a.A2, a.W2, M, N, a.K2).run(t, bt[t.wave], nullptr, acc2);
    // the main product's first loads go out before the reduction of u
    f4 xa0[ND][RT], xb0[ND][2];
    main.load(t, 0, xa0, xb0);
    u = tile_sum(t, part, acc2);
    __syncthreads();  // part is written again below
    main.run(t, bt[0], a.ywin_out, acc, xa0, xb0);
  } else {
    main.run(t, bt[MODE == kMlpvNN ? t.wave : 0], adj ? a.ywin_out : nullptr, acc);
  }
  const float sum = tile_sum(t, part, acc);

  const int m = t.m0 + (t.tid >> 5), n = t.n0 + (t.tid & 31);
  float lterm = 0.f;
  if (t.tid < 512 * RT && m < M && n < N) {
    const size_t o = (size_t)m * N + n;
    if (MODE == kMlpvNN) {
      a.out[o] = a.add ? a.add[o] + sum : sum;
    } else {
      const float z = sum + a.bias[n];
      const float y1 = fmaxf(z, 0.f);
      if (MODE == kMlpvFwd) {
        a.out[o] = y1;
      } else {
        // the loss term of y_{l+1} (already scaled by its own 1 / (B w_{l+1}))
        // and its seed dL/dy_{l+1}
        float sd = 0.f;
        if (a.loss == AMBPTT_LOSS_MEAN_SQ_ALL) {
          sd = 2.f * y1 * a.inv;
          lterm = y1 * y1 * a.inv;
        } else if (a.last) {
          if (a.loss == AMBPTT_LOSS_HALF_SQ_LAST) {
            sd = y1;
            lterm = y1 * y1;
          } else {
            sd = a.inv;
            lterm = y1 * a.inv;
          }
        }
        const float yb1 = (MODE == kMlpvAdjU ? u : a.nn_in ? a.nn_in[o] : 0.f) + sd;
        a.zbar_out[o] = z > 0.f ? yb1 : 0.f;
      }
    }
  }
  if (adj) {
    const float s = wave_sum(lterm);
    if (t.lane == 0) lpart[t.wave] = s;
    __syncthreads();
    if (t.tid == 0) {
      float tot = 0.f;
#pragma unroll
      for (int w = 0; w < kVW; ++w) tot += lpart[w];
      a.loss_acc[blockIdx.y * gridDim.x + blockIdx.x] += (double)tot;
    }
  }
}

struct MlpvDwGroup {
  DwArgs g[kMlpvDwGroup];
};

// dW_l[n][c] = sum_m zbar_l[m][n] y_l[m][c] and db_l[n] = sum_m zbar_l[m][n]
// over the R = B rows of the layer, for the layers of a window in one launch
// (blockIdx.z: the member; tiles past its own dW return at once).  The same
// 16-wave layout: a 32 x 32 tile of dW_l, the rows m in chunks of 16 spread
// over the waves (up to ND in flight), partial tiles summed in wave order
// through LDS.  Both operands are read along m, so a lane reads its 4 rows of
// one column as 4 words, coalesced across the 16 lanes of a quarter wave;
// rows past R read row R - 1 and are zeroed.  The first column of workgroups
// also sums db.
template <int ND>
__global__ __launch_bounds__(64 * kVW) void mlpv_dw(MlpvDwGroup grp) {
  __shared__ float part[kVW][32][33];
  __shared__ float bpart[kVW][4][32];
  const DwArgs& a = grp.g[blockIdx.z];
  if (int(blockIdx.x) * 32 >= a.GH || int(blockIdx.y) * 32 >= a.H) return;  // the whole workgroup, before any barrier
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r = lane & 15, q = lane >> 4;
  const int NW = a.GH, CW = a.H, R = a.R;
  const float* Z = (const float*)a.zbar;
  const float* Y = (const float*)a.hwin;
  const int n0 = blockIdx.x * 32, c0 = blockIdx.y * 32;
  const int nch = (R + 15) / 16;
  const int ngrp = (nch + kVW * ND - 1) / (kVW * ND);
  int zc[2], yc[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    zc[i] = min(n0 + 16 * i + r, NW - 1);  // past the tile's edge: clamped, discarded
    yc[i] = min(c0 + 16 * i + r, CW - 1);
  }
  f4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
  float bs[2] = {0.f, 0.f};
  for (int g = 0; g < ngrp; ++g) {
    f4 xa[ND][2], xb[ND][2];
#pragma unroll
    for (int u = 0; u < ND; ++u) {
      const int mb = 16 * min(wave + kVW * (ND * g + u), nch - 1) + 4 * q;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const size_t m = (size_t)min(mb + k, R - 1);
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          xa[u][i][k] = Z[m * NW + zc[i]];
          xb[u][i][k] = Y[m * CW + yc[i]];
        }
      }
    }
    __builtin_amdgcn_sched_barrier(0);  // every load of the group issues before its first MFMA
#pragma unroll
    for (int u = 0; u < ND; ++u) {
      const int c = wave + kVW * (ND * g + u);
      const int mb = 16 * c + 4 * q;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const bool ok = c < nch && mb + k < R;
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          xa[u][i][k] = ok ? xa[u][i][k] : 0.f;
          xb[u][i][k] = ok ? xb[u][i][k] : 0.f;
        }
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          bs[i] += xa[u][i][k];
#pragma unroll
          for (int j = 0; j < 2; ++j) acc[i][j] = mfma4(xa[u][i][k], xb[u][j][k], acc[i][j]);
        }
      }
    }
  }
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    bpart[wave][q][16 * i + r] = bs[i];
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) part[wave][16 * i + 4 * q + v][16 * j + r] = acc[i][j][v];
  }
  __syncthreads();
  const int nl = tid >> 5, cl = tid & 31;
  const int n = n0 + nl, c = c0 + cl;
  float sum = 0.f;
#pragma unroll
  for (int w = 0; w < kVW; ++w) sum += part[w][nl][cl];
  if (n < NW && c < CW) {
    float* o = a.dW + (size_t)n * CW + c;
    *o = a.accumulate ? *o + sum : sum;
  }
  if (blockIdx.y == 0 && tid < 32 && n0 + tid < NW) {
    float b = 0.f;
#pragma unroll
    for (int w = 0; w < kVW; ++w)
#pragma unroll
      for (int qq = 0; qq < 4; ++qq) b += bpart[w][qq][tid];
    float* o = a.db + n0 + tid;
    *o = a.accumulate ? *o + b : b;
  }
}

}  // namespace

hipError_t launch_mlpv_dw(const DwArgs* a, int count, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if (count < 1 || count > kMlpvDwGroup) return hipErrorInvalidValue;
  MlpvDwGroup grp{};
  int tx = 0, ty = 0;
  for (int i = 0; i < count; ++i) {
    const DwArgs& d = a[i];
    if (d.R < 1 || d.H < 1 || d.GH < 1 || d.D != 0 || d.R != a[0].R) return hipErrorInvalidValue;
    grp.g[i] = d;
    tx = std::max(tx, (d.GH + 31) / 32);
    ty = std::max(ty, (d.H + 31) / 32);
  }
  const dim3 grid(tx, ty, count), block(64 * kVW);
  if ((a[0].R + 15) / 16 <= kVW) hipExtLaunchKernelGGL(mlpv_dw<1>, grid, block, 0, s, e0, e1, 0, grp);
  else hipExtLaunchKernelGGL(mlpv_dw<2>, grid, block, 0, s, e0, e1, 0, grp);
  return hipGetLastError();
}

int mlpv_tiles(int M, int N) { return ((M + 15) / 16) * ((N + 31) / 32); }  // the most tiles any launch has

// chunks of 16 per wave in flight: ceil(K / 256), up to 4 (longer reductions loop)
static int mlpv_nd(int K) { return std::min(4, std::max(1, (K / 16 + kVW - 1) / kVW)); }

// rows per tile: 32, or 16 where 32-row tiles give fewer workgroups than CUs
static int mlpv_rows(int M, int N) { return ((M + 31) / 32) * ((N + 31) / 32) < 256 ? 16 : 32; }

template <int MODE, int ND2, int RT>
static hipError_t launch_mlpv_rt(const MlpvArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  const dim3 grid((a.M + 16 * RT - 1) / (16 * RT), (a.N + 31) / 32), block(64 * kVW);
  switch (mlpv_nd(a.K)) {
    case 1: hipExtLaunchKernelGGL((mlpv_gemm<MODE, 1, ND2, RT>), grid, block, 0, s, e0, e1, 0, a); break;
    case 2: hipExtLaunchKernelGGL((mlpv_gemm<MODE, 2, ND2, RT>), grid, block, 0, s, e0, e1, 0, a); break;
    case 3: hipExtLaunchKernelGGL((mlpv_gemm<MODE, 3, ND2, RT>), grid, block, 0, s, e0, e1, 0, a); break;
    default: hipExtLaunchKernelGGL((mlpv_gemm<MODE, 4, ND2, RT>), grid, block, 0, s, e0, e1, 0, a); break;
  }
  return hipGetLastError();
}

template <int MODE, int ND2>
static hipError_t launch_mlpv_nd(const MlpvArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  return mlpv_rows(a.M, a.N) == 16 ? launch_mlpv_rt<MODE, ND2, 1>(a, s, e0, e1) : launch_mlpv_rt<MODE, ND2, 2>(a, s, e0, e1);
}

hipError_t launch_mlpv(int mode, const MlpvArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if (a.M < 1 || a.N < 16 || a.K < 16 || a.N % 16 || a.K % 16) return hipErrorInvalidValue;
  if (mode == kForward) return launch_mlpv_nd<kMlpvFwd, 1>(a, s, e0, e1);
  if (mode == kFinal) return launch_mlpv_nd<kMlpvNN, 1>(a, s, e0, e1);
  if (!a.A2) return launch_mlpv_nd<kMlpvAdj, 1>(a, s, e0, e1);
  if (a.K2 < 16 || a.K2 % 16 || !a.W2 || a.nn_in) return hipErrorInvalidValue;
  switch (mlpv_nd(a.K2)) {
    case 1: return launch_mlpv_nd<kMlpvAdjU, 1>(a, s, e0, e1);
    case 2: return launch_mlpv_nd<kMlpvAdjU, 2>(a, s, e0, e1);
    case 3: return launch_mlpv_nd<kMlpvAdjU, 3>(a, s, e0, e1);
    default: return launch_mlpv_nd<kMlpvAdjU, 4>(a, s, e0, e1);
  }
}

}  // namespace ambptt
