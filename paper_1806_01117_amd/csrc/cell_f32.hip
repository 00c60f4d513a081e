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

// acc[i][nb] += sum over 16-wide chunks [c0, c1) of A_i(ch) . B_nb(ch).
// la(ch, i) / lb(ch, nb) return the lane's float4 of chunk ch.  Loads run one
// group of U chunks ahead of the MFMAs (register double buffering), so a wave
// keeps up to 2U chunks of loads in flight instead of waiting on each one.
template <int RM, int NB, int U, class LA, class LB>
__device__ __forceinline__ void nt_chunks(int c0, int c1, f4 (&acc)[RM][NB], LA la, LB lb) {
  if (c0 >= c1) return;
  f4 a[U][RM], b[U][NB];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int ch = min(c0 + u, c1 - 1);
#pragma unroll
    for (int i = 0; i < RM; ++i) a[u][i] = la(ch, i);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) b[u][nb] = lb(ch, nb);
  }
  for (int g = c0; g < c1; g += U) {
    f4 an[U][RM], bn[U][NB];
    const bool more = g + U < c1;
    if (more) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int ch = min(g + U + u, c1 - 1);
#pragma unroll
        for (int i = 0; i < RM; ++i) an[u][i] = la(ch, i);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) bn[u][nb] = lb(ch, nb);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (g + u < c1) {
#pragma unroll
        for (int i = 0; i < RM; ++i)
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) {
            acc[i][nb] = mfma4(a[u][i].x, b[u][nb].x, acc[i][nb]);
            acc[i][nb] = mfma4(a[u][i].y, b[u][nb].y, acc[i][nb]);
            acc[i][nb] = mfma4(a[u][i].z, b[u][nb].z, acc[i][nb]);
            acc[i][nb] = mfma4(a[u][i].w, b[u][nb].w, acc[i][nb]);
          }
      }
    }
    if (more) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
#pragma unroll
        for (int i = 0; i < RM; ++i) a[u][i] = an[u][i];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) b[u][nb] = bn[u][nb];
      }
    }
  }
}

template <int G, int RM, int RJ, int KS, int MODE>
__global__ __launch_bounds__(64 * KS) void step_f32(StepArgs a) {
  constexpr int U = (RM * RJ >= 4) ? 2 : 4;   // chunks per prefetch group
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int r = lane & 15, q = lane >> 4;
  const int B = a.B, D = a.D, H = a.H;
  const int GH = G * H, K1 = D + H;
  const int m0 = blockIdx.x * (16 * RM);
  const int j0 = blockIdx.y * (16 * RJ);

  f4 acc[RM][RJ * G];  // gate GEMM, column block nb = jj * G + g
  f4 acch[RM][RJ];     // h-adjoint GEMM
#pragma unroll
  for (int i = 0; i < RM; ++i) {
#pragma unroll
    for (int nb = 0; nb < RJ * G; ++nb) acc[i][nb] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int jj = 0; jj < RJ; ++jj) acch[i][jj] = f4{0.f, 0.f, 0.f, 0.f};
  }

  int rows[RM];
#pragma unroll
  for (int i = 0; i < RM; ++i) rows[i] = min(m0 + 16 * i + r, B - 1);  // rows >= B: clamped, discarded

  // ---- gate GEMM over [x_t | h_t] (forward and adjoint) -------------------
  if (MODE != kFinal) {
    const int nch = K1 / 16;
    const int c0 = (nch * wave) / KS, c1 = (nch * (wave + 1)) / KS;
    const float* x = (const float*)a.x;
    const float* h = (const float*)a.h;
    const float* W = (const float*)a.W;
    auto la = [&](int ch, int i) -> f4 {
      const int k = ch * 16 + 4 * q;
      const float* p = (ch * 16 < D) ? x + (size_t)rows[i] * D + k : h + (size_t)rows[i] * H + (k - D);
      return *(const f4*)p;
    };
    auto lb = [&](int ch, int nb) -> f4 {
      const int jj = nb / G, g = nb % G;
      return *(const f4*)(W + (size_t)(g * H + j0 + 16 * jj + r) * K1 + ch * 16 + 4 * q);
    };
    nt_chunks<RM, RJ * G, U>(c0, c1, acc, la, lb);
  }

  // ---- h-adjoint GEMM of the following step: hbar_{t+1} = zbar_{t+1} W_h --
  // (fused only when the adjoint's product did not run as a launch of its own)
  const bool do_hbar = (MODE == kFinal) || (MODE == kAdjoint && !a.first && !a.hbar_in);
  if (do_hbar) {
    const int nch = GH / 16;
    const int c0 = (nch * wave) / KS, c1 = (nch * (wave + 1)) / KS;
    const float* zb = (const float*)a.zbar_in;
    const float* wt = (const float*)a.WhT;
    const size_t ldw = a.ld_wht ? a.ld_wht : GH;
    auto la = [&](int ch, int i) -> f4 { return *(const f4*)(zb + (size_t)rows[i] * GH + ch * 16 + 4 * q); };
    auto lb = [&](int ch, int jj) -> f4 {
      return *(const f4*)(wt + (size_t)(j0 + 16 * jj + r) * ldw + ch * 16 + 4 * q);
    };
    nt_chunks<RM, RJ, U>(c0, c1, acch, la, lb);
  }

  // ---- fixed-order reduction of the K-split partials ----------------------
  if constexpr (KS > 1) {
    constexpr int NG = (MODE == kFinal) ? 0 : RJ * G;
    constexpr int NH = (MODE == kForward) ? 0 : RJ;
    constexpr int NA = RM * (NG + NH);
    __shared__ f4 red[(KS - 1) * NA * 64];
    if (wave > 0) {
      f4* dst = red + (size_t)(wave - 1) * NA * 64 + lane;
      int idx = 0;
#pragma unroll
      for (int i = 0; i < RM; ++i) {
#pragma unroll
        for (int nb = 0; nb < NG; ++nb) dst[(idx++) * 64] = acc[i][nb];
#pragma unroll
        for (int jj = 0; jj < NH; ++jj) dst[(idx++) * 64] = acch[i][jj];
      }
    }
    __syncthreads();
    if (wave != 0) return;
    for (int w = 1; w < KS; ++w) {
      const f4* src = red + (size_t)(w - 1) * NA * 64 + lane;
      int idx = 0;
#pragma unroll
      for (int i = 0; i < RM; ++i) {
#pragma unroll
        for (int nb = 0; nb < NG; ++nb) acc[i][nb] += src[(idx++) * 64];
#pragma unroll
        for (int jj = 0; jj < NH; ++jj) acch[i][jj] += src[(idx++) * 64];
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
        const int nb = jj * G;
        float h1, c1 = 0.f, tc = 0.f, ig = 0.f, fg = 0.f, gg = 0.f, og = 0.f, cold = 0.f;
        if (G == 4) {
          ig = sigm(acc[i][nb][v] + a.bias[j]);
          fg = sigm(acc[i][nb + 1 % G][v] + a.bias[H + j]);
          gg = tanhf(acc[i][nb + 2 % G][v] + a.bias[2 * H + j]);
          og = sigm(acc[i][nb + 3 % G][v] + a.bias[3 * H + j]);
          cold = a.c[o];
          c1 = fg * cold + ig * gg;
          tc = tanhf(c1);
          h1 = og * tc;
        } else {
          h1 = tanhf(acc[i][nb][v] + a.bias[j]);
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
        const float hb = (a.first ? 0.f : (a.hbar_in ? a.hbar_in[o] : acch[i][jj][v])) + sd;
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
  if (MODE == kAdjoint) {
    const float s = wave_sum(lterm);
    if (lane == 0) a.loss_acc[blockIdx.y * gridDim.x + blockIdx.x] += (double)s;
  }
}

// The adjoint's h-adjoint product as a launch of its own (fp32):
// out[m][n] = sum_k A[m][k] B[n][k] (+ add[m][n]), A = zbar_{t+1} [M][GH],
// B = W_h^T [H][GH], both rows contiguous in k.  Fused into the step kernel
// it would take the gate GEMM's tile (RJ units, K = GH), which reads 4 times
// as many operand bytes per flop as the forward's (4 RJ gate columns over
// K = D + H); here each workgroup takes RM x NB = 2 x 8 blocks of 16 x 16,
// the forward's ratio of operand loads to MFMAs.  KS waves split K; their
// partials meet in LDS in wave order (bit-reproducible).
template <int RM, int NB, int KS>
__global__ __launch_bounds__(64 * KS) void prod_f32(ProdArgs a) {
  constexpr int U = 2;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane & 15, q = lane >> 4;
  const int M = a.M, N = a.N, K = a.K;
  const int m0 = blockIdx.x * (16 * RM), n0 = blockIdx.y * (16 * NB);
  f4 acc[RM][NB];
#pragma unroll
  for (int i = 0; i < RM; ++i)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[i][nb] = f4{0.f, 0.f, 0.f, 0.f};
  int rows[RM];
#pragma unroll
  for (int i = 0; i < RM; ++i) rows[i] = min(m0 + 16 * i + r, M - 1);  // rows >= M: clamped, discarded
  const float* A = (const float*)a.A;
  const float* Bm = (const float*)a.B;
  const size_t ldb = a.ldb ? a.ldb : K;
  const int nch = K / 16;
  const int c0 = (nch * wave) / KS, c1 = (nch * (wave + 1)) / KS;
  nt_chunks<RM, NB, U>(
      c0, c1, acc, [&](int ch, int i) -> f4 { return *(const f4*)(A + (size_t)rows[i] * K + ch * 16 + 4 * q); },
      [&](int ch, int nb) -> f4 { return *(const f4*)(Bm + (size_t)(n0 + 16 * nb + r) * ldb + ch * 16 + 4 * q); });
  if constexpr (KS > 1) {
    __shared__ f4 red[(KS - 1) * RM * NB * 64];
    if (wave > 0) {
      f4* dst = red + (size_t)(wave - 1) * RM * NB * 64 + lane;
#pragma unroll
      for (int i = 0; i < RM; ++i)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) dst[(i * NB + nb) * 64] = acc[i][nb];
    }
    __syncthreads();
    if (wave != 0) return;
    for (int w = 1; w < KS; ++w) {
      const f4* src = red + (size_t)(w - 1) * RM * NB * 64 + lane;
#pragma unroll
      for (int i = 0; i < RM; ++i)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) acc[i][nb] += src[(i * NB + nb) * 64];
    }
  }
  // accumulator element v of lane l: row 4 (l >> 4) + v, column l & 15 of its block
#pragma unroll
  for (int i = 0; i < RM; ++i)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int m = m0 + 16 * i + 4 * q + v;
      if (m >= M) continue;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const size_t o = (size_t)m * N + n0 + 16 * nb + r;
        a.out[o] = a.add ? a.add[o] + acc[i][nb][v] : acc[i][nb][v];
      }
    }
}

// dW[k][c] += sum_r Z[r][k] X[r][c] and db[k] += sum_r Z[r][k] over the R rows
// of one window (a "TN" product: both operands are row-major in r).
// Workgroup = 4 waves on a 64 (k) x 64 (c) tile of dW, each wave a 32 x 32
// quarter (2 x 2 MFMA blocks).  Rows stream through LDS in stages of 64:
// every thread loads 4 float4 of Z and 4 of X per stage with coalesced
// row-contiguous reads, the next stage's loads are in flight while the
// current stage's MFMAs run, and LDS rows are padded to 80 floats so the MFMA
// operand reads (16 consecutive floats from each of 4 rows) hit distinct banks.
// Lane l feeds Z[r][k0 + (l & 15)] and X[r][c0 + (l & 15)] for
// r = 4 g + (l >> 4).  The bias gradient is the column sum of Z, taken from
// LDS by the first wave of the workgroups of column tile 0.
constexpr int kDwT = 64, kDwS = 64, kDwLd = 80;

__global__ __launch_bounds__(256) void dw_lds_f32(DwArgs a) {
  __shared__ float Zs[2][kDwS][kDwLd];
  __shared__ float Xs[2][kDwS][kDwLd];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int li = lane & 15, lk = lane >> 4;
  const int k0 = blockIdx.x * kDwT, c0 = blockIdx.y * kDwT;
  const int D = a.D, H = a.H, GH = a.GH, R = a.R, N = D + H;
  const bool do_bias = blockIdx.y == 0;

  // loader: thread t moves rows (t >> 4) + 16 p, columns 4 (t & 15) .. +3
  const int lrow = tid >> 4, lcol = 4 * (tid & 15);
  const int c = c0 + lcol;
  const bool cok = c < N;
  const float* xsrc = c < D ? (const float*)a.x + c : (const float*)a.hwin + (min(c, N - 1) - D);
  const int xld = c < D ? D : H;
  const bool kok = k0 + lcol < GH;  // GH % 16 == 0: a float4 is wholly in or out
  const float* zsrc = (const float*)a.zbar + min(k0 + lcol, GH - 4);
  f4 zr[4], xr[4];
  auto load = [&](int st) {
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const int row = st * kDwS + lrow + 16 * p;
      const bool ok = row < R;
      zr[p] = (ok && kok) ? *(const f4*)(zsrc + (size_t)row * GH) : f4{0.f, 0.f, 0.f, 0.f};
      xr[p] = (ok && cok) ? *(const f4*)(xsrc + (size_t)row * xld) : f4{0.f, 0.f, 0.f, 0.f};
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      *(f4*)&Zs[buf][lrow + 16 * p][lcol] = zr[p];
      *(f4*)&Xs[buf][lrow + 16 * p][lcol] = xr[p];
    }
  };

  f4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
  float bsum = 0.f;

  const int nst = (R + kDwS - 1) / kDwS;
  load(0);
  store(0);
  __syncthreads();
  for (int st = 0; st < nst; ++st) {
    const int buf = st & 1;
    const bool more = st + 1 < nst;
    if (more) load(st + 1);
#pragma unroll 4
    for (int g = 0; g < kDwS / 4; ++g) {
      const int rr = 4 * g + lk;
      const float a0 = Zs[buf][rr][wm * 32 + li], a1 = Zs[buf][rr][wm * 32 + 16 + li];
      const float b0 = Xs[buf][rr][wn * 32 + li], b1 = Xs[buf][rr][wn * 32 + 16 + li];
      acc[0][0] = mfma4(a0, b0, acc[0][0]);
      acc[0][1] = mfma4(a0, b1, acc[0][1]);
      acc[1][0] = mfma4(a1, b0, acc[1][0]);
      acc[1][1] = mfma4(a1, b1, acc[1][1]);
    }
    if (do_bias && wave == 0) {
      for (int rr = 0; rr < kDwS; ++rr) bsum += Zs[buf][rr][lane];
    }
    if (more) store(buf ^ 1);
    __syncthreads();
  }
#pragma unroll
  for (int ik = 0; ik < 2; ++ik)
#pragma unroll
    for (int ic = 0; ic < 2; ++ic)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int k = k0 + wm * 32 + 16 * ik + 4 * lk + v;
        const int cc = c0 + wn * 32 + 16 * ic + li;
        if (cc < N && k < GH) {
          float* d = a.dW + (size_t)k * N + cc;
          *d = a.accumulate ? *d + acc[ik][ic][v] : acc[ik][ic][v];
        }
      }
  if (do_bias && wave == 0 && k0 + lane < GH) a.db[k0 + lane] = a.accumulate ? a.db[k0 + lane] + bsum : bsum;
}

__global__ void transpose_wh_f32(const float* __restrict__ W, float* __restrict__ WhT, int GH, int D, int H, int ld) {
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
    if (j < H && k < GH) WhT[(size_t)j * ld + k] = tile[tx][y];
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
hipError_t launch_g(const StepCfg& c, const StepArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  dim3 grid, block;
  step_grid(c, a.B, a.H, &grid, &block);
#define AMB_CASE(RM_, RJ_, KS_)                                                                   \
  if (c.rm == RM_ && c.rj == RJ_ && c.ks == KS_) {                                                \
    hipExtLaunchKernelGGL((step_f32<G, RM_, RJ_, KS_, MODE>), grid, block, 0, s, e0, e1, 0, a); \
    return hipGetLastError();                                                                     \
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

hipError_t launch_step(int G, int mode, const StepCfg& c, const StepArgs& a, hipStream_t s, hipEvent_t e0,
                       hipEvent_t e1) {
  if (G == 4) {
    if (mode == kForward) return launch_g<4, kForward>(c, a, s, e0, e1);
    if (mode == kAdjoint) return launch_g<4, kAdjoint>(c, a, s, e0, e1);
    return launch_g<4, kFinal>(c, a, s, e0, e1);
  }
  if (mode == kForward) return launch_g<1, kForward>(c, a, s, e0, e1);
  if (mode == kAdjoint) return launch_g<1, kAdjoint>(c, a, s, e0, e1);
  return launch_g<1, kFinal>(c, a, s, e0, e1);
}

hipError_t launch_dw(const DwArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if (a.GH % 16 != 0) return hipErrorInvalidValue;
  if (dw_f32_big_fits(a)) return launch_dw_f32_big(a, s, e0, e1);
  const int N = a.D + a.H;
  dim3 grid((a.GH + kDwT - 1) / kDwT, (N + kDwT - 1) / kDwT);
  hipExtLaunchKernelGGL(dw_lds_f32, grid, dim3(256), 0, s, e0, e1, 0, a);
  return hipGetLastError();
}
hipError_t launch_prod_f32(const ProdArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if (a.K % 16 != 0 || a.N % 16 != 0 || a.M < 1 || a.K < 16) return hipErrorInvalidValue;
  if (a.N % 128 == 0) {
    const dim3 grid((a.M + 31) / 32, a.N / 128);
    hipExtLaunchKernelGGL((prod_f32<2, 8, 4>), grid, dim3(256), 0, s, e0, e1, 0, a);
  } else {
    const dim3 grid((a.M + 15) / 16, a.N / 16);
    hipExtLaunchKernelGGL((prod_f32<1, 1, 4>), grid, dim3(256), 0, s, e0, e1, 0, a);
  }
  return hipGetLastError();
}

hipError_t launch_transpose_wh(const float* W, float* WhT, int GH, int D, int H, int ld, hipStream_t s) {
  if (ld < GH) return hipErrorInvalidValue;
  dim3 grid((GH + 31) / 32, (H + 31) / 32);
  hipLaunchKernelGGL(transpose_wh_f32, grid, dim3(32, 8), 0, s, W, WhT, GH, D, H, ld);
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
