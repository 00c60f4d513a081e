// Residual MLP treated as a sequence (depth = steps), gfx950.
//
//   forward   y_{l+1} = y_l + relu(z_l),  z_l = y_l W_l^T + b_l,  W_l[w][w] (out x in)
//   adjoint   ybar_{l+1} = ybar_{l+2} + zbar_{l+1} W_{l+1}   (ybar_L = dL/dy_L)
//             zbar_l = ybar_{l+1} * 1[z_l > 0]   (relu'(0) = 0)
//             dW_l = zbar_l^T y_l,  db_l = sum_rows zbar_l   (weight-gradient kernel)
//   final     dL/dy_0 = ybar_1 + zbar_0 W_0
//
// One launch per step, with the small-batch tile of the recurrent cells: a
// workgroup owns 16 batch rows x 16 output columns and its 8 waves split the
// reduction, summed through LDS in wave order.  The adjoint launch of layer l
// recomputes z_l (an "NT" product: both operands contiguous in the reduction
// index) and forms ybar_{l+1} with the previous launch's zbar_{l+1} (an "NN"
// product: W_{l+1}[k][c] is contiguous in c, not in the reduction index k).
// For the NN product each wave loads a CW x 16 block of W_{l+1} with
// coalesced 16-byte row reads, stages it in a wave-private LDS tile and reads
// it back transposed, so no transposed copy of the weights is kept (they are
// 67 GB at width 4096 and 2000 layers).  ybar (fp32) is carried between
// launches like the LSTM's cell-state adjoint.
#include <hip/hip_runtime.h>

#include "ambptt.h"
#include "kernels.hpp"
#include "mfma.hpp"

namespace ambptt {
namespace {

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

template <class T>
struct Mop;
template <>
struct Mop<float> {
  using V = f4;
  static constexpr int CW = 16, LE = 4;
  static __device__ __forceinline__ f4 mma(const V& a, const V& b, f4 c) {
    c = mfma_f32_16x16x4(a.x, b.x, c);
    c = mfma_f32_16x16x4(a.y, b.y, c);
    c = mfma_f32_16x16x4(a.z, b.z, c);
    return mfma_f32_16x16x4(a.w, b.w, c);
  }
  static __device__ __forceinline__ float store(float v) { return v; }
  static __device__ __forceinline__ float load(float v) { return v; }
};
template <>
struct Mop<__bf16> {
  using V = bf16x8;
  static constexpr int CW = 32, LE = 8;
  static __device__ __forceinline__ f4 mma(const V& a, const V& b, f4 c) { return mfma_bf16_16x16x32(a, b, c); }
  static __device__ __forceinline__ __bf16 store(float v) { return (__bf16)v; }
  static __device__ __forceinline__ float load(__bf16 v) { return (float)v; }
};

constexpr int kWaves = 8;
constexpr int kU = 4;

template <class T, int MODE>
__global__ __launch_bounds__(64 * kWaves) void resmlp_step(MlpArgs a) {
  using V = typename Mop<T>::V;
  constexpr int CW = Mop<T>::CW, LE = Mop<T>::LE;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = lane & 15, q = lane >> 4;
  const int B = a.B, w = a.w;
  const int mtiles = (B + 15) / 16, ntile = mtiles * (w / 16);
  const int per = (ntile + 7) / 8;  // XCD-aware order, as in the recurrent cells
  const int tile = (blockIdx.x % 8) * per + blockIdx.x / 8;
  if (tile >= ntile) return;
  const int m0 = (tile % mtiles) * 16;
  const int c0 = (tile / mtiles) * 16;
  const int row = min(m0 + r, B - 1);

  __shared__ float zs[kWaves][16][17];
  __shared__ float ys[kWaves][16][17];
  __shared__ __attribute__((aligned(16))) T wt[kWaves][CW][16 + LE];

  const int nch = w / CW;
  const int k0c = (nch * wave) / kWaves, k1c = (nch * (wave + 1)) / kWaves;

  // z_l = y_l W_l^T for this tile (forward and adjoint)
  if (MODE != kFinal) {
    f4 acc = {0.f, 0.f, 0.f, 0.f};
    const T* yr = (const T*)a.y + (size_t)row * w;
    const T* wr = (const T*)a.W + (size_t)(c0 + r) * w;
    V av[kU], bv[kU];
    for (int g = k0c; g < k1c; g += kU) {
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const int ch = min(g + u, k1c - 1);
        av[u] = *(const V*)(yr + ch * CW + LE * q);
        bv[u] = *(const V*)(wr + ch * CW + LE * q);
      }
#pragma unroll
      for (int u = 0; u < kU; ++u)
        if (g + u < k1c) acc = Mop<T>::mma(av[u], bv[u], acc);
    }
#pragma unroll
    for (int v = 0; v < 4; ++v) zs[wave][4 * q + v][r] = acc[v];
  }
  // ybar_{l+1} - ybar_{l+2} = zbar_{l+1} W_{l+1} (adjoint after the first, and final)
  const bool do_nn = (MODE == kFinal) || (MODE == kAdjoint && !a.first);
  if (do_nn) {
    f4 acc = {0.f, 0.f, 0.f, 0.f};
    const T* zr = (const T*)a.zbar_in + (size_t)row * w;
    // coalesced block load: lane -> row (lane / (16 / LE)), columns LE * (lane % (16 / LE))
    constexpr int LPR = 16 / LE;  // lanes per 16-column row segment
    const int lr = lane / LPR, lc = LE * (lane % LPR);
    const T* wsrc = (const T*)a.Wn + (size_t)lr * w + c0 + lc;
    V av[kU], gv[kU];
    for (int g = k0c; g < k1c; g += kU) {
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const int ch = min(g + u, k1c - 1);
        av[u] = *(const V*)(zr + ch * CW + LE * q);
        gv[u] = *(const V*)(wsrc + (size_t)ch * CW * w);
      }
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        if (g + u < k1c) {
          *(V*)&wt[wave][lr][lc] = gv[u];  // rows k of the block, 16 columns
          V bt;
#pragma unroll
          for (int e = 0; e < LE; ++e) bt[e] = wt[wave][LE * q + e][r];  // column r, LE consecutive k
          acc = Mop<T>::mma(av[u], bt, acc);
        }
      }
    }
#pragma unroll
    for (int v = 0; v < 4; ++v) ys[wave][4 * q + v][r] = acc[v];
  }
  __syncthreads();

  // epilogue: thread (m, c), 16 x 16 per workgroup
  float lterm = 0.f;
  if (tid < 256) {
    const int ml = tid >> 4, cl = tid & 15;
    const int m = m0 + ml, c = c0 + cl;
    if (m < B) {
      const size_t o = (size_t)m * w + c;
      float nn = 0.f;
      if (do_nn) {
#pragma unroll
        for (int v = 0; v < kWaves; ++v) nn += ys[v][ml][cl];
      }
      if (MODE == kFinal) {
        a.dy0[o] = a.ybar_in[o] + nn;
      } else {
        float z = 0.f;
#pragma unroll
        for (int v = 0; v < kWaves; ++v) z += zs[v][ml][cl];
        z += a.bias[c];
        const float yv = Mop<T>::load(((const T*)a.y)[o]);
        const float y1 = yv + fmaxf(z, 0.f);
        const T y1s = Mop<T>::store(y1);
        if (MODE == kForward) {
          ((T*)a.y_out)[o] = y1s;
        } else {
          float yb;
          if (a.first) {
            const float hl = Mop<T>::load(y1s);  // loss reads the stored y_L
            if (a.loss == AMBPTT_LOSS_HALF_SQ_LAST) {
              yb = hl;
              lterm = hl * hl;
            } else if (a.loss == AMBPTT_LOSS_MEAN_LAST) {
              yb = a.inv_bw;
              lterm = hl;
            } else {
              yb = 2.f * hl * a.inv_bw;
              lterm = hl * hl;
            }
          } else {
            yb = a.ybar_in[o] + nn;
            if (a.loss == AMBPTT_LOSS_MEAN_SQ_ALL) {  // loss term of y_{l+1}
              const float hl = Mop<T>::load(y1s);
              yb += 2.f * hl * a.inv_bw;
              lterm = hl * hl;
            }
          }
          a.ybar_out[o] = yb;
          ((T*)a.zbar_out)[o] = Mop<T>::store(z > 0.f ? yb : 0.f);
          ((T*)a.ywin_out)[o] = ((const T*)a.y)[o];
        }
      }
    }
  }
  if (MODE == kAdjoint) {
    const float s = wave_sum(lterm);
    __shared__ float wsum[kWaves];
    if (lane == 0) wsum[wave] = s;
    __syncthreads();
    if (tid == 0) {
      float t = 0.f;
#pragma unroll
      for (int v = 0; v < kWaves; ++v) t += wsum[v];
      a.loss_acc[tile] += (double)t;
    }
  }
}

}  // namespace

void resmlp_grid(int B, int w, dim3* grid, dim3* block) {
  const int ntile = ((B + 15) / 16) * (w / 16);
  *grid = dim3(8 * ((ntile + 7) / 8), 1, 1);
  *block = dim3(64 * kWaves, 1, 1);
}

hipError_t launch_resmlp(int bf16, int mode, const MlpArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  dim3 grid, block;
  resmlp_grid(a.B, a.w, &grid, &block);
#define AMB_M(T_, M_) hipExtLaunchKernelGGL((resmlp_step<T_, M_>), grid, block, 0, s, e0, e1, 0, a)
  if (bf16) {
    if (mode == kForward) AMB_M(__bf16, kForward);
    else if (mode == kAdjoint) AMB_M(__bf16, kAdjoint);
    else AMB_M(__bf16, kFinal);
  } else {
    if (mode == kForward) AMB_M(float, kForward);
    else if (mode == kAdjoint) AMB_M(float, kAdjoint);
    else AMB_M(float, kFinal);
  }
#undef AMB_M
  return hipGetLastError();
}

}  // namespace ambptt
