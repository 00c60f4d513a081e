// One-launch step kernels for small batches (fp32, gfx950).
//
// A kernel launch costs ~3 us on its own here, so each recurrent step is one
// launch.  For a batch of 64 the gate GEMM (B x G*H x (D+H)) must still be
// spread over all 256 CUs, and what bounds a workgroup is the bytes it streams
// from L2 (~30 GB/s per workgroup), so the tile is the smallest that still
// covers the whole reduction: 16 batch rows x U hidden units, all G gates
// (U = 8 for the LSTM, i.e. 32 weight rows; U = 16 for the tanh RNN).  The 8
// waves of a workgroup split the reduction; their partial products meet in
// LDS and are summed in wave order (bit-reproducible), then one thread per
// (row, unit) runs the cell math.
//
// Within the workgroup's G*U columns the weight rows are gate-major:
// column n = g*U + u is row g*H + j0 + u of W, so the epilogue thread of unit
// u finds its gates at columns u, U+u, 2U+u, 3U+u.
//
// The adjoint launch of step t also computes hbar_{t+1} = zbar_{t+1} W_h for
// its (rows, units) tile, the one product that needs the previous launch's
// output; W_h is read through its transpose WhT[j][k] = W[k][D+j] so both
// products are row-contiguous in the reduction index.
//
// Operands are fp32 (v_mfma_f32_16x16x4_f32, chunks of 16 reduction indices,
// 4 per lane) or bf16 (v_mfma_f32_16x16x32_bf16, chunks of 32, 8 per lane):
// either way a lane loads 16 bytes per operand row per chunk.  With bf16 the
// stored h, the copy of h_t for the weight gradient and zbar (the adjoint
// GEMMs' operand) are rounded to bf16 (nearest even); accumulation, the cell
// state and its adjoint stay fp32.
#include <hip/hip_runtime.h>

#include "ambptt.h"
#include "kernels.hpp"
#include "mfma.hpp"

namespace ambptt {
namespace {

__device__ __forceinline__ f4 mfma4(float a, float b, f4 c) { return mfma_f32_16x16x4(a, b, c); }

__device__ __forceinline__ float sigm(float z) { return 1.0f / (1.0f + __expf(-z)); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

template <class T>
struct Op;
template <>
struct Op<float> {
  using V = f4;
  static constexpr int CW = 16;  // reduction indices per chunk
  static __device__ __forceinline__ f4 mma(const V& a, const V& b, f4 c) {
    c = mfma4(a.x, b.x, c);
    c = mfma4(a.y, b.y, c);
    c = mfma4(a.z, b.z, c);
    return mfma4(a.w, b.w, c);
  }
  static __device__ __forceinline__ float store(float v) { return v; }
  static __device__ __forceinline__ float load(float v) { return v; }
};
template <>
struct Op<__bf16> {
  using V = bf16x8;
  static constexpr int CW = 32;
  static __device__ __forceinline__ f4 mma(const V& a, const V& b, f4 c) {
    return mfma_bf16_16x16x32(a, b, c);
  }
  static __device__ __forceinline__ __bf16 store(float v) { return (__bf16)v; }  // nearest even
  static __device__ __forceinline__ float load(__bf16 v) { return (float)v; }
};

constexpr int kWaves = 8;
constexpr int kU = 4;  // chunks per prefetch group

// acc[nb] += sum over chunks [c0, c1) of a(ch) . b(ch, nb); loads run one group
// of kU chunks ahead of the MFMAs.
template <class T, int NB, class LA, class LB>
__device__ __forceinline__ void chunks(int c0, int c1, f4 (&acc)[NB], LA la, LB lb) {
  using V = typename Op<T>::V;
  if (c0 >= c1) return;
  V a[kU], b[kU][NB];
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    const int ch = min(c0 + u, c1 - 1);
    a[u] = la(ch);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) b[u][nb] = lb(ch, nb);
  }
  for (int g = c0; g < c1; g += kU) {
    V an[kU], bn[kU][NB];
    const bool more = g + kU < c1;
    if (more) {
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const int ch = min(g + kU + u, c1 - 1);
        an[u] = la(ch);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) bn[u][nb] = lb(ch, nb);
      }
    }
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      if (g + u < c1) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) acc[nb] = Op<T>::mma(a[u], b[u][nb], acc[nb]);
      }
    }
    if (more) {
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        a[u] = an[u];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) b[u][nb] = bn[u][nb];
      }
    }
  }
}

template <class T, int G, int MODE>
__global__ __launch_bounds__(64 * kWaves) void step_small(StepArgs a) {
  using V = typename Op<T>::V;
  constexpr int CW = Op<T>::CW;
  constexpr int LE = CW / 4;  // elements per lane per chunk (16 bytes)
  constexpr int U = (G == 4) ? 8 : 16;  // units per workgroup
  constexpr int NC = G * U;             // gate columns (32 or 16)
  constexpr int NB = NC / 16;           // MFMA column blocks
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = lane & 15, q = lane >> 4;
  const int B = a.B, D = a.D, H = a.H, GH = G * H, K1 = D + H;
  // XCD-aware tile order.  Workgroups are dealt to the 8 XCDs round-robin by
  // id, so ids with equal id % 8 share an L2.  Tiles are numbered unit-group
  // major (w = ug * mtiles + mt) and each XCD takes a contiguous run of them:
  // the row tiles of one unit group then read its weight rows through one L2.
  const int mtiles = (B + 15) / 16, ntile = mtiles * (H / U);
  const int per = (ntile + 7) / 8;
  const int w = (blockIdx.x % 8) * per + blockIdx.x / 8;
  if (w >= ntile) return;  // grid padding (the whole workgroup leaves together)
  const int m0 = (w % mtiles) * 16;
  const int j0 = (w / mtiles) * U;
  const int wg_slot = w;   // loss accumulator of this tile
  const int row = min(m0 + r, B - 1);  // rows >= B: clamped loads, results dropped

  __shared__ float zs[kWaves][16][NC + 1];
  __shared__ float hs[kWaves][16][17];

  if (MODE != kFinal) {
    f4 acc[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[nb] = f4{0.f, 0.f, 0.f, 0.f};
    const int nch = K1 / CW;
    const int c0 = (nch * wave) / kWaves, c1 = (nch * (wave + 1)) / kWaves;
    const T* xr = (const T*)a.x + (size_t)row * D;
    const T* hr = (const T*)a.h + (size_t)row * H;
    const T* wr[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int n = nb * 16 + r;  // column of this lane in block nb
      wr[nb] = (const T*)a.W + (size_t)((n / U) * H + j0 + (n % U)) * K1;
    }
    chunks<T, NB>(c0, c1, acc,
                  [&](int ch) -> V {
                    const int k = ch * CW + LE * q;
                    return *(const V*)(ch * CW < D ? xr + k : hr + (k - D));
                  },
                  [&](int ch, int nb) -> V { return *(const V*)(wr[nb] + ch * CW + LE * q); });
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int v = 0; v < 4; ++v) zs[wave][4 * q + v][nb * 16 + r] = acc[nb][v];
  }
  const bool do_hbar = (MODE == kFinal) || (MODE == kAdjoint && !a.first);
  if (do_hbar) {
    f4 acc[1] = {f4{0.f, 0.f, 0.f, 0.f}};
    const int nch = GH / CW;
    const int c0 = (nch * wave) / kWaves, c1 = (nch * (wave + 1)) / kWaves;
    const T* zr = (const T*)a.zbar_in + (size_t)row * GH;
    // U units; lanes r >= U (LSTM) repeat units so no extra rows are fetched
    const T* wt = (const T*)a.WhT + (size_t)(j0 + (r % U)) * GH;
    chunks<T, 1>(c0, c1, acc, [&](int ch) -> V { return *(const V*)(zr + ch * CW + LE * q); },
                 [&](int ch, int) -> V { return *(const V*)(wt + ch * CW + LE * q); });
#pragma unroll
    for (int v = 0; v < 4; ++v) hs[wave][4 * q + v][r] = acc[0][v];
  }
  __syncthreads();

  // epilogue: thread (m, u) for m < 16, u < U
  float lterm = 0.f;
  if (tid < 16 * U) {
    const int ml = tid / U, u = tid % U;
    const int m = m0 + ml, j = j0 + u;
    if (m < B) {
      const size_t o = (size_t)m * H + j;
      float hbar = 0.f;
      if (do_hbar) {
#pragma unroll
        for (int w = 0; w < kWaves; ++w) hbar += hs[w][ml][u];
      }
      if (MODE == kFinal) {
        a.dh0[o] = hbar;
        if (G == 4) a.dc0[o] = a.cbar_in[o];
      } else {
        float z[G];
#pragma unroll
        for (int g = 0; g < G; ++g) {
          float s = 0.f;
#pragma unroll
          for (int w = 0; w < kWaves; ++w) s += zs[w][ml][g * U + u];
          z[g] = s + a.bias[g * H + j];
        }
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
        const T h1s = Op<T>::store(h1);  // the stored state
        if (MODE == kForward) {
          ((T*)a.h_out)[o] = h1s;
          if (G == 4) a.c_out[o] = c1;
        } else {
          const float hl = Op<T>::load(h1s);  // loss and seed read the stored h_{t+1}
          float sd = 0.f;
          if (a.loss == AMBPTT_LOSS_MEAN_SQ_ALL) {
            sd = 2.f * hl * a.inv_bh;
            lterm = hl * hl;
          } else if (a.last) {
            if (a.loss == AMBPTT_LOSS_HALF_SQ_LAST) {
              sd = hl;
              lterm = hl * hl;
            } else {
              sd = a.inv_bh;
              lterm = hl;
            }
          }
          const float hb = hbar + sd;
          T* zo = (T*)a.zbar_out + (size_t)m * GH + j;
          if (G == 4) {
            const float cb = a.first ? 0.f : a.cbar_in[o];
            const float ob = hb * tc;
            const float ch = cb + hb * og * (1.f - tc * tc);
            zo[0] = Op<T>::store(ch * gg * ig * (1.f - ig));
            zo[H] = Op<T>::store(ch * cold * fg * (1.f - fg));
            zo[2 * H] = Op<T>::store(ch * ig * (1.f - gg * gg));
            zo[3 * H] = Op<T>::store(ob * og * (1.f - og));
            a.cbar_out[o] = ch * fg;
          } else {
            zo[0] = Op<T>::store(hb * (1.f - h1 * h1));
          }
          ((T*)a.hwin_out)[o] = ((const T*)a.h)[o];
        }
      }
    }
  }
  if (MODE == kAdjoint) {
    // threads >= 16 U hold 0; waves beyond the epilogue contribute nothing
    const float s = wave_sum(lterm);
    __shared__ float wsum[kWaves];
    if (lane == 0) wsum[wave] = s;
    __syncthreads();
    if (tid == 0) {
      float t = 0.f;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) t += wsum[w];
      a.loss_acc[wg_slot] += (double)t;
    }
  }
}

}  // namespace

void step_small_grid(int G, int B, int H, dim3* grid, dim3* block) {
  const int U = (G == 4) ? 8 : 16;
  const int ntile = ((B + 15) / 16) * (H / U);
  *grid = dim3(8 * ((ntile + 7) / 8), 1, 1);
  *block = dim3(64 * kWaves, 1, 1);
}

hipError_t launch_step_small(int G, int bf16, int mode, const StepArgs& a, hipStream_t s, hipEvent_t e0,
                             hipEvent_t e1) {
  dim3 grid, block;
  step_small_grid(G, a.B, a.H, &grid, &block);
#define AMB_L(T_, G_, M_) hipExtLaunchKernelGGL((step_small<T_, G_, M_>), grid, block, 0, s, e0, e1, 0, a)
#define AMB_T(T_)                                   \
  if (G == 4) {                                     \
    if (mode == kForward) AMB_L(T_, 4, kForward);   \
    else if (mode == kAdjoint) AMB_L(T_, 4, kAdjoint); \
    else AMB_L(T_, 4, kFinal);                      \
  } else {                                          \
    if (mode == kForward) AMB_L(T_, 1, kForward);   \
    else if (mode == kAdjoint) AMB_L(T_, 1, kAdjoint); \
    else AMB_L(T_, 1, kFinal);                      \
  }
  if (bf16) {
    AMB_T(__bf16)
  } else {
    AMB_T(float)
  }
#undef AMB_T
#undef AMB_L
  return hipGetLastError();
}

}  // namespace ambptt
