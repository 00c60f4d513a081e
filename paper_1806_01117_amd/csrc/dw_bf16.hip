// bf16 weight-gradient window and W_h transpose (gfx950).
//
// dW[k][c] += sum_r Z[r][k] X[r][c], db[k] += sum_r Z[r][k] over the R rows of
// one window, Z = zbar and X = [x | h] in bf16, accumulation in fp32 on
// v_mfma_f32_16x16x32_bf16.  The MFMA wants each lane's 8 consecutive
// reduction indices r for one k (or c), so rows are staged through LDS
// transposed: Zt[k][r], Xt[c][r] (row stride padded to 72 elements), filled
// from coalesced 16-byte global reads of Z and X rows.  Workgroup = 4 waves
// on a 64 x 64 tile of dW (2 x 2 MFMA blocks per wave), 64 rows per stage,
// the next stage's global reads in flight while the current stage computes.
#include <hip/hip_runtime.h>

#include "kernels.hpp"
#include "mfma.hpp"

namespace ambptt {
namespace {

constexpr int kT = 64, kS = 64, kLd = 72;

__global__ __launch_bounds__(256) void dw_bf16(DwArgs a) {
  __shared__ __attribute__((aligned(16))) __bf16 Zt[2][kT][kLd];
  __shared__ __attribute__((aligned(16))) __bf16 Xt[2][kT][kLd];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int li = lane & 15, lq = lane >> 4;
  const int k0 = blockIdx.x * kT, c0 = blockIdx.y * kT;
  const int D = a.D, H = a.H, GH = a.GH, R = a.R, N = D + H;
  const bool do_bias = blockIdx.y == 0;
  const __bf16* Z = (const __bf16*)a.zbar;
  const __bf16* X = (const __bf16*)a.x;
  const __bf16* Hw = (const __bf16*)a.hwin;

  // loader: thread t moves rows (t >> 3) + 32 p (p = 0, 1), elements 8 (t & 7) .. +7
  const int lrow = tid >> 3, lcol = 8 * (tid & 7);
  const int kc = k0 + lcol, cc = c0 + lcol;
  const bool kok = kc < GH;  // GH % 32 == 0: a 16-byte group is wholly in or out
  const bool cok = cc < N;
  const __bf16* zsrc = Z + min(kc, GH - 8);
  const __bf16* xsrc = cc < D ? X + cc : Hw + (min(cc, N - 8) - D);
  const int xld = cc < D ? D : H;
  bf16x8 zr[2], xr[2];
  const bf16x8 zero = {};
  auto load = [&](int st) {
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      const int row = st * kS + lrow + 32 * p;
      const bool ok = row < R;
      zr[p] = (ok && kok) ? *(const bf16x8*)(zsrc + (size_t)row * GH) : zero;
      xr[p] = (ok && cok) ? *(const bf16x8*)(xsrc + (size_t)row * xld) : zero;
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      const int rr = lrow + 32 * p;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        Zt[buf][lcol + e][rr] = zr[p][e];
        Xt[buf][lcol + e][rr] = xr[p][e];
      }
    }
  };

  f4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
  float bsum = 0.f;

  const int nst = (R + kS - 1) / kS;
  load(0);
  store(0);
  __syncthreads();
  for (int st = 0; st < nst; ++st) {
    const int buf = st & 1;
    const bool more = st + 1 < nst;
    if (more) load(st + 1);
#pragma unroll
    for (int g = 0; g < kS / 32; ++g) {
      const int r0 = 32 * g + 8 * lq;
      const bf16x8 a0 = *(const bf16x8*)&Zt[buf][wm * 32 + li][r0];
      const bf16x8 a1 = *(const bf16x8*)&Zt[buf][wm * 32 + 16 + li][r0];
      const bf16x8 b0 = *(const bf16x8*)&Xt[buf][wn * 32 + li][r0];
      const bf16x8 b1 = *(const bf16x8*)&Xt[buf][wn * 32 + 16 + li][r0];
      acc[0][0] = mfma_bf16_16x16x32(a0, b0, acc[0][0]);
      acc[0][1] = mfma_bf16_16x16x32(a0, b1, acc[0][1]);
      acc[1][0] = mfma_bf16_16x16x32(a1, b0, acc[1][0]);
      acc[1][1] = mfma_bf16_16x16x32(a1, b1, acc[1][1]);
    }
    if (do_bias && wave == 0) {
      for (int rr = 0; rr < kS; ++rr) bsum += (float)Zt[buf][lane][rr];
    }
    if (more) store(buf ^ 1);  // buf ^ 1 was last read before the previous barrier
    __syncthreads();
  }
#pragma unroll
  for (int ik = 0; ik < 2; ++ik)
#pragma unroll
    for (int ic = 0; ic < 2; ++ic)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int k = k0 + wm * 32 + 16 * ik + 4 * lq + v;
        const int c = c0 + wn * 32 + 16 * ic + li;
        if (c < N && k < GH) {
          float* d = a.dW + (size_t)k * N + c;
          *d = a.accumulate ? *d + acc[ik][ic][v] : acc[ik][ic][v];
        }
      }
  if (do_bias && wave == 0 && k0 + lane < GH) a.db[k0 + lane] = a.accumulate ? a.db[k0 + lane] + bsum : bsum;
}

__global__ void transpose_wh_u16(const uint16_t* __restrict__ W, uint16_t* __restrict__ WhT, int GH, int D,
                                 int H) {
  __shared__ uint16_t tile[32][33];
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

}  // namespace

hipError_t launch_dw_bf16(const DwArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if (a.GH % 32 != 0 || (a.D + a.H) % 32 != 0) return hipErrorInvalidValue;
  const int N = a.D + a.H;
  dim3 grid((a.GH + kT - 1) / kT, (N + kT - 1) / kT);
  hipExtLaunchKernelGGL(dw_bf16, grid, dim3(256), 0, s, e0, e1, 0, a);
  return hipGetLastError();
}

hipError_t launch_transpose_wh_bf16(const void* W, void* WhT, int GH, int D, int H, hipStream_t s) {
  dim3 grid((GH + 31) / 32, (H + 31) / 32);
  hipLaunchKernelGGL(transpose_wh_u16, grid, dim3(32, 8), 0, s, (const uint16_t*)W, (uint16_t*)WhT, GH, D, H);
  return hipGetLastError();
}

}  // namespace ambptt
