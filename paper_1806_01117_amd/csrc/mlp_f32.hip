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
// One launch per step.  A workgroup owns 32 rows x 32 columns, each of its
// 4 waves one 16 x 16 block; the reduction runs in chunks of 16 straight from
// global memory: lane l reads 4 consecutive k of row l & 15 at 4 (l >> 4) and
// its components feed 4 MFMAs (A and the "NT" B the same way; the "NN" B as
// 4 reads of one column each, coalesced across the 16 lanes).  Widths are
// multiples of 16; a tile's second column block may fall past N and then
// idles.  The loss terms of a workgroup are summed in wave order.
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
  __shared__ float red[4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = lane & 15, q = lane >> 4;
  const int M = a.M, N = a.N, K = a.K;
  const int m0 = blockIdx.x * 32 + (wave >> 1) * 16;
  const int n0 = blockIdx.y * 32 + (wave & 1) * 16;
  const bool active = n0 < N;
  f4 acc = {0.f, 0.f, 0.f, 0.f};
  if (active) {
    const float* arow = a.A + (size_t)min(m0 + r, M - 1) * K + 4 * q;  // rows >= M: clamped, discarded
    for (int k0 = 0; k0 < K; k0 += 16) {
      const f4 av = *(const f4*)(arow + k0);
      f4 bv;
      if (MODE == kMlpvNN) {
        const float* w = a.W + (size_t)(k0 + 4 * q) * N + n0 + r;
        bv = f4{w[0], w[N], w[2 * (size_t)N], w[3 * (size_t)N]};
      } else {
        bv = *(const f4*)(a.W + (size_t)(n0 + r) * K + k0 + 4 * q);
      }
      acc = mfma4(av.x, bv.x, acc);
      acc = mfma4(av.y, bv.y, acc);
      acc = mfma4(av.z, bv.z, acc);
      acc = mfma4(av.w, bv.w, acc);
    }
  }
  // accumulator element v of lane l: row 4 (l >> 4) + v, column l & 15 of the block
  float lterm = 0.f;
  if (active) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int m = m0 + 4 * q + v, n = n0 + r;
      if (m >= M) continue;
      const size_t o = (size_t)m * N + n;
      if (MODE == kMlpvNN) {
        a.out[o] = a.add ? a.add[o] + acc[v] : acc[v];
        continue;
      }
      const float z = acc[v] + a.bias[n];
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
      const float yb = (a.nn_in ? a.nn_in[o] : 0.f) + sd;
      a.zbar_out[o] = z > 0.f ? yb : 0.f;
    }
  }
  if (MODE == kMlpvAdj) {
    const float s = wave_sum(lterm);
    if (lane == 0) red[wave] = s;
    __syncthreads();
    if (tid == 0)
      a.loss_acc[blockIdx.y * gridDim.x + blockIdx.x] +=
          (double)red[0] + (double)red[1] + (double)red[2] + (double)red[3];
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
