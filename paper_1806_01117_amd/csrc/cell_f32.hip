// fp32 step kernels for the tanh RNN (G = 1) and LSTM (G = 4) cells on
// gfx950, using v_mfma_f32_16x16x4_f32.
//
// One launch is one forward step (ADVANCE), one adjoint step (first turn or
// youturn), or the final dL/dx_0 product.  The whole gate GEMM and the cell
// math sit in one kernel; nothing but the state and the adjoint carries goes
// through HBM.
//
// Work split.  A workgroup owns RM x RJ tiles of 16 batch rows x 16 hidden
// units.  Its KS waves split the reduction dimension; the partial MFMA
// accumulators are summed through LDS in a fixed order (wave 0, 1, ...), so
// results are bit-reproducible.  Wave 0 then runs the elementwise epilogue
// straight from its accumulators: for a given (row, unit) the four gate
// accumulators sit in the same lane and register, so the cell update needs
// no data exchange.
//
// Operands are read directly from global memory as float4 per lane: lane l
// holds row (l & 15) and reduction indices 4 (l >> 4) .. +3 of a 16-wide
// chunk, and feeds them to four MFMAs (one per component), which together
// cover the chunk.  Both GEMMs are "NT": every operand row is contiguous in
// the reduction index:
//   gate GEMM     z[m][g H + j] = sum_k [x | h][m][k] W[g H + j][k]
//   adjoint GEMM  hbar[m][j]    = sum_k zbar[m][k] WhT[j][k]
// The adjoint kernel of step t fuses the h-adjoint GEMM of step t+1 (it only
// needs zbar_{t+1}, written by the previous launch) with the recomputation of
// step t's gates, so each adjoint step is a single launch.
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

template <int G, int RM, int RJ, int KS, int MODE>
__global__ __launch_bounds__(64 * KS) void step_f32(StepArgs a) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int r = lane & 15, q = lane >> 4;
  const int B = a.B, D = a.D, H = a.H;
  const int GH = G * H, K1 = D + H;
  const int m0 = blockIdx.x * (16 * RM);
  const int j0 = blockIdx.y * (16 * RJ);

  f4 acc[RM][RJ][G];
  f4 acch[RM][RJ];
#pragma unroll
  for (int i = 0; i < RM; ++i)
#pragma unroll
    for (int jj = 0; jj < RJ; ++jj) {
#pragma unroll
      for (int g = 0; g < G; ++g) acc[i][jj][g] = f4{0.f, 0.f, 0.f, 0.f};
      acch[i][jj] = f4{0.f, 0.f, 0.f, 0.f};
    }

  int rows[RM];
#pragma unroll
  for (int i = 0; i < RM; ++i) rows[i] = min(m0 + 16 * i + r, B - 1);  // rows >= B: clamped, discarded

  // ---- gate GEMM over [x_t | h_t] (forward and adjoint) -------------------
  if (MODE != kFinal) {
    const int nch = K1 / 16;
    const int c0 = (nch * wave) / KS, c1 = (nch * (wave + 1)) / KS;
    for (int ch = c0; ch < c1; ++ch) {
      const int k = ch * 16 + 4 * q;
      f4 av[RM];
      if (ch * 16 < D) {
#pragma unroll
        for (int i = 0; i < RM; ++i) av[i] = *(const f4*)(a.x + (size_t)rows[i] * D + k);
      } else {
#pragma unroll
        for (int i = 0; i < RM; ++i) av[i] = *(const f4*)(a.h + (size_t)rows[i] * H + (k - D));
      }
      f4 bv[RJ][G];
#pragma unroll
      for (int jj = 0; jj < RJ; ++jj)
#pragma unroll
        for (int g = 0; g < G; ++g)
          bv[jj][g] = *(const f4*)(a.W + (size_t)(g * H + j0 + 16 * jj + r) * K1 + k);
#pragma unroll
      for (int i = 0; i < RM; ++i)
#pragma unroll
        for (int jj = 0; jj < RJ; ++jj)
#pragma unroll
          for (int g = 0; g < G; ++g) {
            acc[i][jj][g] = mfma4(av[i].x, bv[jj][g].x, acc[i][jj][g]);
            acc[i][jj][g] = mfma4(av[i].y, bv[jj][g].y, acc[i][jj][g]);
            acc[i][jj][g] = mfma4(av[i].z, bv[jj][g].z, acc[i][jj][g]);
            acc[i][jj][g] = mfma4(av[i].w, bv[jj][g].w, acc[i][jj][g]);
          }
    }
  }

  // ---- h-adjoint GEMM of the following step: hbar_{t+1} = zbar_{t+1} W_h --
  const bool do_hbar = (MODE == kFinal) || (MODE == kAdjoint && !a.first);
  if (do_hbar) {
    const int nch = GH / 16;
    const int c0 = (nch * wave) / KS, c1 = (nch * (wave + 1)) / KS;
    for (int ch = c0; ch < c1; ++ch) {
      const int k = ch * 16 + 4 * q;
      f4 av[RM], bv[RJ];
#pragma unroll
      for (int i = 0; i < RM; ++i) av[i] = *(const f4*)(a.zbar_in + (size_t)rows[i] * GH + k);
#pragma unroll
      for (int jj = 0; jj < RJ; ++jj) bv[jj] = *(const f4*)(a.WhT + (size_t)(j0 + 16 * jj + r) * GH + k);
#pragma unroll
      for (int i = 0; i < RM; ++i)
#pragma unroll
        for (int jj = 0; jj < RJ; ++jj) {
          acch[i][jj] = mfma4(av[i].x, bv[jj].x, acch[i][jj]);
          acch[i][jj] = mfma4(av[i].y, bv[jj].y, acch[i][jj]);
          acch[i][jj] = mfma4(av[i].z, bv[jj].z, acch[i][jj]);
          acch[i][jj] = mfma4(av[i].w, bv[jj].w, acch[i][jj]);
        }
    }
  }

  // ---- fixed-order reduction of the K-split partials ----------------------
  if constexpr (KS > 1) {
    constexpr int NG = (MODE == kFinal) ? 0 : G;
    constexpr int NA = RM * RJ * (NG + (MODE == kForward ? 0 : 1));
    __shared__ f4 red[(KS - 1) * NA * 64];
    if (wave > 0) {
      f4* dst = red + (size_t)(wave - 1) * NA * 64 + lane;
      int idx = 0;
#pragma unroll
      for (int i = 0; i < RM; ++i)
#pragma unroll
        for (int jj = 0; jj < RJ; ++jj) {
#pragma unroll
          for (int g = 0; g < NG; ++g) dst[(idx++) * 64] = acc[i][jj][g];
          if (MODE != kForward) dst[(idx++) * 64] = acch[i][jj];
        }
    }
    __syncthreads();
    if (wave != 0) return;
    for (int w = 1; w < KS; ++w) {
      const f4* src = red + (size_t)(w - 1) * NA * 64 + lane;
      int idx = 0;
#pragma unroll
      for (int i = 0; i < RM; ++i)
#pragma unroll
        for (int jj = 0; jj < RJ; ++jj) {
#pragma unroll
          for (int g = 0; g < NG; ++g) acc[i][jj][g] += src[(idx++) * 64];
          if (MODE != kForward) acch[i][jj] += src[(idx++) * 64];
        }
    }
  }

  // ---- epilogue (wave 0): accumulator element v of lane l is row 4 (l>>4) + v,
  //      unit l & 15 of its 16x16 tile ------------------------------------------
  float lterm = 0.f;
#pragma unroll
  for (int i = 0; i < RM; ++i)
#pragma unroll
    for (int jj = 0; jj < RJ; ++jj)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int m = m0 + 16 * i + 4 * q + v;
        const int j = j0 + 16 * jj + r;
        if (m >= B) continue;
        const size_t o = (size_t)m * H + j;
        if (MODE == kFinal) {
          a.dh0[o] = acch[i][jj][v];
          if (G == 4) a.dc0[o] = a.cbar_in[o];
          continue;
        }
        float h1, c1 = 0.f, tc = 0.f, ig = 0.f, fg = 0.f, gg = 0.f, og = 0.f, cold = 0.f;
        if (G == 4) {
          ig = sigm(acc[i][jj][0][v] + a.bias[j]);
          fg = sigm(acc[i][jj][1 % G][v] + a.bias[H + j]);
          gg = tanhf(acc[i][jj][2 % G][v] + a.bias[2 * H + j]);
          og = sigm(acc[i][jj][3 % G][v] + a.bias[3 * H + j]);
          cold = a.c[o];
          c1 = fg * cold + ig * gg;
          tc = tanhf(c1);
          h1 = og * tc;
        } else {
          h1 = tanhf(acc[i][jj][0][v] + a.bias[j]);
        }
        if (MODE == kForward) {
          a.h_out[o] = h1;
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
        const float hb = (a.first ? 0.f : acch[i][jj][v]) + sd;
        float* zo = a.zbar_out + (size_t)m * GH + j;
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
        a.hwin_out[o] = a.h[o];
      }
  if (MODE == kAdjoint) {
    const float s = wave_sum(lterm);
    if (lane == 0) a.loss_acc[blockIdx.y * gridDim.x + blockIdx.x] += (double)s;
  }
}

// dW[k][c] += sum_r Z[r][k] X[r][c]: a "TN" product, both operands row-major in
// the reduction index r.  Lane l feeds Z[r][k0 + (l & 15)] and X[r][c0 + (l & 15)]
// for r = r0 + 4 q + (l >> 4); column D+H of X is the constant 1 (bias gradient).
template <int RK, int RC>
__global__ __launch_bounds__(64) void dw_f32(DwArgs a) {
  const int lane = threadIdx.x;
  const int li = lane & 15, lk = lane >> 4;
  const int k0 = blockIdx.x * (16 * RK);
  const int c0 = blockIdx.y * (16 * RC);
  const int D = a.D, H = a.H, GH = a.GH, R = a.R, N = D + H;

  f4 acc[RK][RC];
#pragma unroll
  for (int ik = 0; ik < RK; ++ik)
#pragma unroll
    for (int ic = 0; ic < RC; ++ic) acc[ik][ic] = f4{0.f, 0.f, 0.f, 0.f};

  for (int r0 = 0; r0 < R; r0 += 16) {
    float za[RK][4], xb[RC][4];
#pragma unroll
    for (int qq = 0; qq < 4; ++qq) {
      const int rr = r0 + 4 * qq + lk;
      const bool ok = rr < R;
#pragma unroll
      for (int ik = 0; ik < RK; ++ik) za[ik][qq] = ok ? a.zbar[(size_t)rr * GH + k0 + 16 * ik + li] : 0.f;
#pragma unroll
      for (int ic = 0; ic < RC; ++ic) {
        const int c = c0 + 16 * ic + li;
        float v = 0.f;
        if (ok) {
          if (c < D) v = a.x[(size_t)rr * D + c];
          else if (c < N) v = a.hwin[(size_t)rr * H + (c - D)];
          else if (c == N) v = 1.f;
        }
        xb[ic][qq] = v;
      }
    }
#pragma unroll
    for (int qq = 0; qq < 4; ++qq)
#pragma unroll
      for (int ik = 0; ik < RK; ++ik)
#pragma unroll
        for (int ic = 0; ic < RC; ++ic) acc[ik][ic] = mfma4(za[ik][qq], xb[ic][qq], acc[ik][ic]);
  }
#pragma unroll
  for (int ik = 0; ik < RK; ++ik)
#pragma unroll
    for (int ic = 0; ic < RC; ++ic)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int k = k0 + 16 * ik + 4 * lk + v;
        const int c = c0 + 16 * ic + li;
        if (c < N) a.dW[(size_t)k * N + c] += acc[ik][ic][v];
        else if (c == N) a.db[k] += acc[ik][ic][v];
      }
}

__global__ void transpose_wh_f32(const float* __restrict__ W, float* __restrict__ WhT, int GH, int D, int H) {
  __shared__ float tile[32][33];
  const int kb = blockIdx.x * 32, jb = blockIdx.y * 32;
  const int tx = threadIdx.x, ty = threadIdx.y;
  for (int y = ty; y < 32; y += 8) {
    const int k = kb + y, j = jb + tx;
    if (k < GH && j < H) tile[y][tx] = W[(size_t)k * (D + H) + D + j];
  }
  __syncthreads();
  for (int y = ty; y < 32; y += 8) {
    const int j = jb + y, k = kb + tx;
    if (j < H && k < GH) WhT[(size_t)j * GH + k] = tile[tx][y];
  }
}

__global__ void fill32(uint32_t* p, size_t n, uint32_t v) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) p[i] = v;
}

__global__ void loss_sum(const double* acc, int n, double scale, double* out) {
  if (threadIdx.x == 0 && blockIdx.x == 0) {
    double s = 0.0;
    for (int i = 0; i < n; ++i) s += acc[i];
    *out = s * scale;
  }
}

template <int G, int MODE>
hipError_t launch_g(const StepCfg& c, const StepArgs& a, hipStream_t s) {
  dim3 grid, block;
  step_grid(c, a.B, a.H, &grid, &block);
#define AMB_CASE(RM_, RJ_, KS_)                                                     \
  if (c.rm == RM_ && c.rj == RJ_ && c.ks == KS_) {                                  \
    hipLaunchKernelGGL((step_f32<G, RM_, RJ_, KS_, MODE>), grid, block, 0, s, a); \
    return hipGetLastError();                                                       \
  }
  AMB_CASE(1, 1, 1)
  AMB_CASE(1, 1, 2)
  AMB_CASE(1, 1, 4)
  AMB_CASE(1, 1, 8)
  AMB_CASE(2, 2, 1)
  AMB_CASE(2, 2, 2)
  AMB_CASE(2, 2, 4)
#undef AMB_CASE
  return hipErrorInvalidValue;
}

}  // namespace

StepCfg pick_step_cfg(int G, int B, int D, int H) {
  const int mt = (B + 15) / 16, jt = H / 16;
  const int nch = (D + H) / 16;
  StepCfg c{1, 1, 1};
  if (mt >= 8 && jt % 2 == 0 && (long)mt * jt >= 2048) {
    c.rm = 2;
    c.rj = 2;
    const long wgs = (long)((mt + 1) / 2) * (jt / 2);
    c.ks = wgs >= 1024 ? 1 : (wgs >= 256 ? 2 : 4);
    return c;
  }
  int ks = nch / 3;
  c.ks = ks >= 8 ? 8 : ks >= 4 ? 4 : ks >= 2 ? 2 : 1;
  (void)G;
  return c;
}

void step_grid(const StepCfg& c, int B, int H, dim3* grid, dim3* block) {
  const int mt = (B + 15) / 16;
  *grid = dim3((mt + c.rm - 1) / c.rm, H / (16 * c.rj), 1);
  *block = dim3(64 * c.ks, 1, 1);
}

hipError_t launch_step(int G, int mode, const StepCfg& c, const StepArgs& a, hipStream_t s) {
  if (G == 4) {
    if (mode == kForward) return launch_g<4, kForward>(c, a, s);
    if (mode == kAdjoint) return launch_g<4, kAdjoint>(c, a, s);
    return launch_g<4, kFinal>(c, a, s);
  }
  if (mode == kForward) return launch_g<1, kForward>(c, a, s);
  if (mode == kAdjoint) return launch_g<1, kAdjoint>(c, a, s);
  return launch_g<1, kFinal>(c, a, s);
}

hipError_t launch_dw(const DwArgs& a, hipStream_t s) {
  const int N1 = a.D + a.H + 1;
  if (a.GH % 32 == 0) {
    dim3 grid(a.GH / 32, (N1 + 31) / 32);
    hipLaunchKernelGGL((dw_f32<2, 2>), grid, dim3(64), 0, s, a);
  } else {
    dim3 grid(a.GH / 16, (N1 + 15) / 16);
    hipLaunchKernelGGL((dw_f32<1, 1>), grid, dim3(64), 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_transpose_wh(const float* W, float* WhT, int GH, int D, int H, hipStream_t s) {
  dim3 grid((GH + 31) / 32, (H + 31) / 32);
  hipLaunchKernelGGL(transpose_wh_f32, grid, dim3(32, 8), 0, s, W, WhT, GH, D, H);
  return hipGetLastError();
}

hipError_t launch_fill32(void* p, size_t words, uint32_t value, hipStream_t s) {
  if (words == 0) return hipSuccess;
  size_t blocks = (words + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(fill32, dim3((unsigned)blocks), dim3(256), 0, s, (uint32_t*)p, words, value);
  return hipGetLastError();
}

hipError_t launch_loss_sum(const double* acc, int n, double scale, double* out, hipStream_t s) {
  hipLaunchKernelGGL(loss_sum, dim3(1), dim3(64), 0, s, acc, n, scale, out);
  return hipGetLastError();
}

}  // namespace ambptt
