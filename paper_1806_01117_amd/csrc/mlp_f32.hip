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
// One launch per step.  A workgroup owns 32 rows x 32 columns; each of its 4
// waves computes the whole tile (2 x 2 blocks of 16 x 16) over a quarter of
// the reduction, in chunks of 16 read straight from global memory with the
// next chunk's operands loaded before the current chunk's 16 MFMAs, and the
// four partial tiles are summed in wave order through LDS by wave 0, which
// then runs the epilogue.  Lane l reads 4 consecutive k of row l & 15 at 4
// (l >> 4) and its components feed 4 MFMAs (A and the "NT" B the same way;
// the "NN" B as 4 reads of one column each, coalesced across the 16 lanes).
// Widths are multiples of 16; a tile's second column block may fall past N
// and then idles.  The loss terms of a workgroup are summed by wave 0.
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

template <int MODE>
__global__ __launch_bounds__(256) void mlpv_gemm(MlpvArgs a) {
  __shared__ f4 part[3][4][64];  // waves 1..3: their four accumulators, lane by lane
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = lane & 15, q = lane >> 4;
  const int M = a.M, N = a.N, K = a.K;
  const int m0 = blockIdx.x * 32, n0 = blockIdx.y * 32;
  const bool two = n0 + 16 < N;  // the second column block lies inside N
  const int nch = K / 16, c0 = nch * wave / 4, c1 = nch * (wave + 1) / 4;
  const float* arow[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) arow[i] = a.A + (size_t)min(m0 + 16 * i + r, M - 1) * K + 4 * q;  // rows >= M: clamped, discarded
  int col[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) col[j] = min(n0 + 16 * j + r, N - 1);  // past N: clamped, discarded
  auto ldb = [&](int k0, int j) -> f4 {
    if (MODE == kMlpvNN) {
      const float* w = a.W + (size_t)(k0 + 4 * q) * N + col[j];
      return f4{w[0], w[N], w[2 * (size_t)N], w[3 * (size_t)N]};
    }
    return *(const f4*)(a.W + (size_t)col[j] * K + k0 + 4 * q);
  };
  f4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
  f4 xa[2], xb[2], ya[2], yb[2];
  if (c0 < c1) {
#pragma unroll
    for (int i = 0; i < 2; ++i) xa[i] = *(const f4*)(arow[i] + 16 * c0);
#pragma unroll
    for (int j = 0; j < 2; ++j) xb[j] = ldb(16 * c0, j);
  }
  for (int c = c0; c < c1; ++c) {
    if (c + 1 < c1) {  // the next chunk's operands, in flight during this chunk's MFMAs
#pragma unroll
      for (int i = 0; i < 2; ++i) ya[i] = *(const f4*)(arow[i] + 16 * (c + 1));
#pragma unroll
      for (int j = 0; j < 2; ++j) yb[j] = ldb(16 * (c + 1), j);
    }
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = mfma4(xa[i][k], xb[j][k], acc[i][j]);
#pragma unroll
    for (int i = 0; i < 2; ++i) xa[i] = ya[i];
#pragma unroll
    for (int j = 0; j < 2; ++j) xb[j] = yb[j];
  }
  if (wave > 0) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) part[wave - 1][2 * i + j][lane] = acc[i][j];
  }
  __syncthreads();
  if (wave != 0) return;
#pragma unroll
  for (int w = 0; w < 3; ++w)
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] += part[w][2 * i + j][lane];

  // accumulator element v of lane l: row 4 (l >> 4) + v, column l & 15 of its block
  float lterm = 0.f;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      if (j == 1 && !two) continue;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int m = m0 + 16 * i + 4 * q + v, n = n0 + 16 * j + r;
        if (m >= M) continue;
        const size_t o = (size_t)m * N + n;
        if (MODE == kMlpvNN) {
          a.out[o] = a.add ? a.add[o] + acc[i][j][v] : acc[i][j][v];
          continue;
        }
        const float z = acc[i][j][v] + a.bias[n];
        const float y1 = fmaxf(z, 0.f);
        if (MODE == kMlpvFwd) {
          a.out[o] = y1;
          continue;
        }
        // the loss term of y_{l+1} (already scaled by its own 1 / (B w_{l+1}))
        // and its seed dL/dy_{l+1}
        float sd = 0.f;
        if (a.loss == AMBPTT_LOSS_MEAN_SQ_ALL) {
          sd = 2.f * y1 * a.inv;
          lterm += y1 * y1 * a.inv;
        } else if (a.last) {
          if (a.loss == AMBPTT_LOSS_HALF_SQ_LAST) {
            sd = y1;
            lterm += y1 * y1;
          } else {
            sd = a.inv;
            lterm += y1 * a.inv;
          }
        }
        const float yb1 = (a.nn_in ? a.nn_in[o] : 0.f) + sd;
        a.zbar_out[o] = z > 0.f ? yb1 : 0.f;
      }
    }
  if (MODE == kMlpvAdj) {
    const float s = wave_sum(lterm);
    if (lane == 0) a.loss_acc[blockIdx.y * gridDim.x + blockIdx.x] += (double)s;
  }
}

}  // namespace

int mlpv_tiles(int M, int N) { return ((M + 31) / 32) * ((N + 31) / 32); }

hipError_t launch_mlpv(int mode, const MlpvArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if (a.M < 1 || a.N < 16 || a.K < 16 || a.N % 16 || a.K % 16) return hipErrorInvalidValue;
  const dim3 grid((a.M + 31) / 32, (a.N + 31) / 32), block(256);
  if (mode == kForward) hipExtLaunchKernelGGL(mlpv_gemm<kMlpvFwd>, grid, block, 0, s, e0, e1, 0, a);
  else if (mode == kAdjoint) hipExtLaunchKernelGGL(mlpv_gemm<kMlpvAdj>, grid, block, 0, s, e0, e1, 0, a);
  else hipExtLaunchKernelGGL(mlpv_gemm<kMlpvNN>, grid, block, 0, s, e0, e1, 0, a);
  return hipGetLastError();
}

}  // namespace ambptt
