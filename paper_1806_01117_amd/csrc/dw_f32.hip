// fp32 weight-gradient window for large gradients (gfx950).
//
// dW[k][c] (+)= sum_r Z[r][k] X[r][c], db[k] (+)= sum_r Z[r][k] over the R
// rows of one window; Z = zbar [R][GH], X = [x | h] [R][D + H], both stored
// with the reduction index r as the row.  A workgroup of 4 waves owns a
// 128 x 128 tile of dW and each wave 64 x 64 of it, as 4 x 4 accumulators of
// v_mfma_f32_16x16x4_f32.  The accumulators are interleaved: accumulator
// (e, f) holds the rows k = 4i + e and the columns c = 4j + f of the wave's
// tile (i, j = 0..15).  With that split a lane's A operands for the four
// accumulator rows e are four consecutive floats of one Z row, and likewise
// for B, so the operands stay in the global row-major layout in LDS (no
// transpose) and 4 reduction rows cost two 16-byte LDS reads per lane for 16
// MFMAs.  Stages of 32 rows are double-buffered: the next stage's global
// reads are issued before the current one is multiplied and are in flight
// meanwhile, with one barrier per stage.
#include <hip/hip_runtime.h>

#include "kernels.hpp"
#include "mfma.hpp"

namespace ambptt {
namespace {

constexpr int kT = 128;  // tile edge
constexpr int kS = 32;   // reduction rows per stage

__global__ __launch_bounds__(256) void dw_f32_big(DwArgs a) {
  __shared__ f4 Zs[2][kS][kT / 4];  // [r][k / 4]
  __shared__ f4 Xs[2][kS][kT / 4];  // [r][c / 4]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int m = lane & 15, q = lane >> 4;
  const int D = a.D, H = a.H, GH = a.GH, R = a.R, N = D + H;
  const int k0 = blockIdx.x * kT, c0 = blockIdx.y * kT;
  const float* Z = (const float*)a.zbar;
  const float* X = (const float*)a.x;
  const float* Hw = (const float*)a.hwin;

  // loader: float4 p of thread t is stage row (t + 256 p) / 32, tile columns
  // 4 ((t + 256 p) % 32) .. + 3; GH, D and H are multiples of 4, so a float4
  // lies wholly inside or outside each operand
  f4 zr[4], xr[4];
  auto load = [&](int st) {
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const int idx = tid + 256 * p, row = st * kS + (idx >> 5), col = 4 * (idx & 31);
      const int k = k0 + col, c = c0 + col;
      zr[p] = f4{0.f, 0.f, 0.f, 0.f};
      xr[p] = f4{0.f, 0.f, 0.f, 0.f};
      if (row < R) {
        if (k < GH) zr[p] = *(const f4*)(Z + (size_t)row * GH + k);
        if (c < D) xr[p] = *(const f4*)(X + (size_t)row * D + c);
        else if (c < N) xr[p] = *(const f4*)(Hw + (size_t)row * H + (c - D));
      }
    }
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const int idx = tid + 256 * p;
      Zs[buf][idx >> 5][idx & 31] = zr[p];
      Xs[buf][idx >> 5][idx & 31] = xr[p];
    }
  };

  f4 acc[4][4];
#pragma unroll
  for (int e = 0; e < 4; ++e)
#pragma unroll
    for (int f = 0; f < 4; ++f) acc[e][f] = f4{0.f, 0.f, 0.f, 0.f};
  float bsum = 0.f;
  const bool do_bias = blockIdx.y == 0 && tid < kT;

  auto multiply = [&](int buf) {
#pragma unroll
    for (int kc = 0; kc < kS / 4; ++kc) {
      const f4 av = Zs[buf][4 * kc + q][16 * wm + m];
      const f4 bv = Xs[buf][4 * kc + q][16 * wn + m];
#pragma unroll
      for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int f = 0; f < 4; ++f) acc[e][f] = mfma_f32_16x16x4(av[e], bv[f], acc[e][f]);
    }
    if (do_bias) {
      const float* zc = (const float*)&Zs[buf][0][0] + tid;
#pragma unroll
      for (int rr = 0; rr < kS; ++rr) bsum += zc[rr * kT];
    }
  };
  // every stage but the last loads the next one while it multiplies; the
  // scheduling barriers keep the global loads ahead of the MFMAs
  const int nst = (R + kS - 1) / kS;
  load(0);
  stash(0);
  __syncthreads();
  for (int st = 0; st + 1 < nst; ++st) {
    load(st + 1);
    __builtin_amdgcn_sched_barrier(0);
    multiply(st & 1);
    __builtin_amdgcn_sched_barrier(0);
    stash((st + 1) & 1);  // that buffer was last read before the previous barrier
    __syncthreads();
  }
  multiply((nst - 1) & 1);
  // lane (q, m) holds, for accumulator (e, f) and v = 0..3, row i = 4q + v and
  // column j = m of the 16 x 16 product: k = 4i + e, c = 4j + f
  const int c = c0 + 64 * wn + 4 * m;
#pragma unroll
  for (int e = 0; e < 4; ++e)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int k = k0 + 64 * wm + 4 * (4 * q + v) + e;
      if (k < GH && c < N) {
        f4* d = (f4*)(a.dW + (size_t)k * N + c);
        f4 o = f4{acc[e][0][v], acc[e][1][v], acc[e][2][v], acc[e][3][v]};
        if (a.accumulate) o += *d;
        *d = o;
      }
    }
  if (do_bias && k0 + tid < GH) a.db[k0 + tid] = a.accumulate ? a.db[k0 + tid] + bsum : bsum;
}

}  // namespace

bool dw_f32_big_fits(const DwArgs& a) {
  return a.GH >= 256 && a.D + a.H >= 256 && a.GH % 16 == 0 && a.D % 4 == 0 && a.H % 4 == 0;
}

hipError_t launch_dw_f32_big(const DwArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if (!dw_f32_big_fits(a)) return hipErrorInvalidValue;
  const dim3 grid((a.GH + kT - 1) / kT, (a.D + a.H + kT - 1) / kT);
  hipExtLaunchKernelGGL(dw_f32_big, grid, dim3(256), 0, s, e0, e1, 0, a);
  return hipGetLastError();
}

}  // namespace ambptt
