// An MLP whose layers change width, treated as a sequence (depth = steps):
// the states y_l [B][w_l] differ in size from layer to layer, the case the
// paper's Sections 1.1 and 6 set beside Revolve's uniform states.  fp32 on
// gfx950 (v_mfma_f32_16x16x4_f32).
//
//   forward   y_{l+1} = relu(z_l),  z_l = y_l W_l^T + b_l,  W_l[w_{l+1}][w_l]
//   adjoint   ybar_{l+1} = u + dL/dy_{l+1},  u = zbar_{l+1} W_{l+1} (0 for the last layer)
//             zbar_l = ybar_{l+1} * 1[z_l > 0]   (relu'(0) = 0)
//   product   u = zbar W  (an "NN" product: W[k][c] is contiguous in c)
// dW_l = zbar_l^T y_l and db_l run on the weight-gradient kernels.
//
// One launch per step.  A workgroup of 16 waves owns 32 rows x 32 columns.
// The reduction runs in chunks of 16; wave w takes chunks w, w + 16, ... in
// groups of up to four whose loads all issue before the group's first MFMA,
// so that a launch of a few hundred workgroups waits about one memory latency
// per group (one in all for K <= 1024) instead of one per chunk.  Each wave computes the whole tile (2 x 2 blocks of
// 16 x 16) over its chunks; the 16 partial tiles go to LDS and every thread
// then sums one output over the waves in wave order (deterministic) and runs
// the epilogue for it, 32 consecutive columns per half wave.  Lane l reads 4
// consecutive k of row l & 15 at 4 (l >> 4) and its components feed 4 MFMAs
// (A and the "NT" B the same way; the "NN" B is read as whole rows and turned
// into fragments through a per-wave tile in LDS).  Widths are multiples of 16; a tile's
// second column block may fall past N and then idles.  The loss terms of a
// workgroup are summed in a fixed order by its first thread.
#include <hip/hip_runtime.h>

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

enum { kMlpvFwd = 0, kMlpvAdj = 1, kMlpvNN = 2 };

constexpr int kVW = 16;  // waves per workgroup

// ND: chunks per wave and group, all in flight at once (ceil(K / 256) up to 4).
template <int MODE, int ND>
__global__ __launch_bounds__(64 * kVW) void mlpv_gemm(MlpvArgs a) {
  __shared__ float part[kVW][32][36];  // partial tiles; rows of 36: the stores of a wave spread over the banks
  __shared__ float lpart[kVW];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r = lane & 15, q = lane >> 4;
  const int M = a.M, N = a.N, K = a.K;
  const int m0 = blockIdx.x * 32, n0 = blockIdx.y * 32;
  const int nch = K / 16;
  const int ngrp = (nch + kVW * ND - 1) / (kVW * ND);  // groups of ND chunks per wave
  const float* arow[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) arow[i] = a.A + (size_t)min(m0 + 16 * i + r, M - 1) * K + 4 * q;  // rows >= M: clamped, discarded
  int col[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) col[j] = min(n0 + 16 * j + r, N - 1);  // past N: clamped, discarded
  // NN: the B chunk (16 reduction rows x 32 columns, contiguous along the
  // columns) is read as whole 128-byte rows, 8 lanes a row, and passes through
  // the wave's own tile in LDS (rows of 36 floats: the column reads of a
  // fragment fall in 64 distinct banks); xb then holds the raw rows brow and
  // brow + 8.  The other modes read B's rows directly.
  __shared__ __attribute__((aligned(16))) float bt[MODE == kMlpvNN ? kVW : 1][16][36];
  const int brow = lane >> 3, bcol = 4 * (lane & 7);
  const float* wnn = a.W + min(n0 + bcol, N - 4);  // a float4 past N: clamped, discarded
  // chunk c of the reduction; past the last chunk the operands read the last
  // one (and are zeroed before use), so that every wave issues the same loads
  // in straight line
  auto load = [&](int c, f4 (&xa)[2], f4 (&xb)[2]) {
    const int k0 = 16 * min(c, nch - 1);
#pragma unroll
    for (int i = 0; i < 2; ++i) xa[i] = *(const f4*)(arow[i] + k0);
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      if (MODE == kMlpvNN) xb[j] = *(const f4*)(wnn + (size_t)(k0 + brow + 8 * j) * N);
      else xb[j] = *(const f4*)(a.W + (size_t)col[j] * K + k0 + 4 * q);
    }
  };
  // NN: the raw rows to the B fragments (column n0 + 16 j + r, rows 4 q .. 4 q + 3)
  auto nn_frag = [&](f4 (&xb)[2]) {
#pragma unroll
    for (int h = 0; h < 2; ++h) *(f4*)&bt[wave][brow + 8 * h][bcol] = xb[h];
#pragma unroll
    for (int j = 0; j < 2; ++j)
      xb[j] = f4{bt[wave][4 * q][16 * j + r], bt[wave][4 * q + 1][16 * j + r], bt[wave][4 * q + 2][16 * j + r],
                 bt[wave][4 * q + 3][16 * j + r]};
  };
  f4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
  for (int g = 0; g < ngrp; ++g) {
    f4 xa[ND][2], xb[ND][2];
#pragma unroll
    for (int u = 0; u < ND; ++u) load(wave + kVW * (ND * g + u), xa[u], xb[u]);
    __builtin_amdgcn_sched_barrier(0);  // every load of the group issues before its first MFMA
#pragma unroll
    for (int u = 0; u < ND; ++u) {
      if (MODE == kMlpvNN) nn_frag(xb[u]);
      if (wave + kVW * (ND * g + u) >= nch) {  // uniform: a chunk past the reduction adds nothing
#pragma unroll
        for (int i = 0; i < 2; ++i) xa[u][i] = xb[u][i] = f4{0.f, 0.f, 0.f, 0.f};
      }
#pragma unroll
      for (int k = 0; k < 4; ++k)
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j) acc[i][j] = mfma4(xa[u][i][k], xb[u][j][k], acc[i][j]);
      if (MODE == kMlpvAdj && blockIdx.y == 0 && a.ywin_out) {  // y_l beside zbar_l for dW_l
        const int c = wave + kVW * (ND * g + u);
#pragma unroll
        for (int i = 0; i < 2; ++i)
          if (c < nch && m0 + 16 * i + r < M) *(f4*)(a.ywin_out + (size_t)(m0 + 16 * i + r) * K + 16 * c + 4 * q) = xa[u][i];
      }
    }
  }
  // accumulator element v of lane l: row 4 (l >> 4) + v, column l & 15 of its block
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) part[wave][16 * i + 4 * q + v][16 * j + r] = acc[i][j][v];
  __syncthreads();

  const int ml = tid >> 5, nl = tid & 31;
  const int m = m0 + ml, n = n0 + nl;
  float sum = 0.f;
#pragma unroll
  for (int w = 0; w < kVW; ++w) sum += part[w][ml][nl];
  float lterm = 0.f;
  if (m < M && n < N) {
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
        const float yb1 = (a.nn_in ? a.nn_in[o] : 0.f) + sd;
        a.zbar_out[o] = z > 0.f ? yb1 : 0.f;
      }
    }
  }
  if (MODE == kMlpvAdj) {
    const float s = wave_sum(lterm);
    if (lane == 0) lpart[wave] = s;
    __syncthreads();
    if (tid == 0) {
      float t = 0.f;
#pragma unroll
      for (int w = 0; w < kVW; ++w) t += lpart[w];
      a.loss_acc[blockIdx.y * gridDim.x + blockIdx.x] += (double)t;
    }
  }
}

// dW_l[n][c] = sum_m zbar_l[m][n] y_l[m][c] and db_l[n] = sum_m zbar_l[m][n]
// over the R = B rows of the layer.  The same 16-wave layout: a 32 x 32 tile
// of dW_l, the rows m in chunks of 16 spread over the waves (up to ND in
// flight), partial tiles summed in wave order through LDS.  Both operands are
// read along m, so a lane reads its 4 rows of one column as 4 words,
// coalesced across the 16 lanes of a quarter wave; rows past R read row R - 1
// and are zeroed.  The first column of workgroups also sums db.
template <int ND>
__global__ __launch_bounds__(64 * kVW) void mlpv_dw(DwArgs a) {
  __shared__ float part[kVW][32][33];
  __shared__ float bpart[kVW][4][32];
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

hipError_t launch_mlpv_dw(const DwArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if (a.R < 1 || a.H < 1 || a.GH < 1 || a.D != 0) return hipErrorInvalidValue;
  const dim3 grid((a.GH + 31) / 32, (a.H + 31) / 32), block(64 * kVW);
  if ((a.R + 15) / 16 <= kVW) hipExtLaunchKernelGGL(mlpv_dw<1>, grid, block, 0, s, e0, e1, 0, a);
  else hipExtLaunchKernelGGL(mlpv_dw<2>, grid, block, 0, s, e0, e1, 0, a);
  return hipGetLastError();
}

int mlpv_tiles(int M, int N) { return ((M + 31) / 32) * ((N + 31) / 32); }

template <int MODE>
hipError_t launch_mlpv_nd(const MlpvArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  const dim3 grid((a.M + 31) / 32, (a.N + 31) / 32), block(64 * kVW);
  const int per_wave = (a.K / 16 + kVW - 1) / kVW;
  if (per_wave <= 1) hipExtLaunchKernelGGL((mlpv_gemm<MODE, 1>), grid, block, 0, s, e0, e1, 0, a);
  else if (per_wave == 2) hipExtLaunchKernelGGL((mlpv_gemm<MODE, 2>), grid, block, 0, s, e0, e1, 0, a);
  else if (per_wave == 3) hipExtLaunchKernelGGL((mlpv_gemm<MODE, 3>), grid, block, 0, s, e0, e1, 0, a);
  else hipExtLaunchKernelGGL((mlpv_gemm<MODE, 4>), grid, block, 0, s, e0, e1, 0, a);
  return hipGetLastError();
}

hipError_t launch_mlpv(int mode, const MlpvArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if (a.M < 1 || a.N < 16 || a.K < 16 || a.N % 16 || a.K % 16) return hipErrorInvalidValue;
  if (mode == kForward) return launch_mlpv_nd<kMlpvFwd>(a, s, e0, e1);
  if (mode == kAdjoint) return launch_mlpv_nd<kMlpvAdj>(a, s, e0, e1);
  return launch_mlpv_nd<kMlpvNN>(a, s, e0, e1);
}

}  // namespace ambptt
