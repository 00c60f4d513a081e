// bf16 weight-gradient window and W_h transpose (gfx950).
//
// dW[k][c] (+)= sum_r Z[r][k] X[r][c], db[k] (+)= sum_r Z[r][k] over the R rows
// of one window, Z = zbar [R][GH] and X = [x | h] [R][D + H] in bf16,
// accumulation in fp32 on v_mfma_f32_16x16x32_bf16.
//
// Both operands have the reduction index r as their row, while the MFMA wants
// each lane's 8 reduction indices of one k (or c) together.  The rows are
// staged in LDS as they are stored in memory (coalesced 16-byte reads, one
// 16-byte LDS write each) and the fragments come out of LDS with gfx950's
// transposing read ds_read_b64_tr_b16: within a group of 16 lanes, lane i
// names 4 consecutive 16-bit values (row kb + (i >> 2), columns 4 (i & 3) ..
// +3 of a 16-column block) and lane j receives value j & 3 of lanes
// 4 e + (j >> 2), e = 0..3, i.e. rows kb .. kb + 3 of column j.  Two such reads
// (rows kb and kb + 4) make one bf16x8 fragment.
//
// Workgroup: TM / 32 waves on a TM x 128 tile of dW, each wave 64 x 64 (4 x 4
// MFMA blocks); 64 reduction rows per stage, double-buffered, the next
// stage's global reads in flight while the current one is multiplied.  LDS
// rows have a pitch of 32 bytes modulo 256 and rows r with (r >> 3) odd have
// their two 128-byte halves swapped, so the 16 row segments of one
// transposing read spread over all banks.  TM = 256 (8 waves, 106 KB of LDS,
// one workgroup per CU) for long windows, whose MFMAs dominate; TM = 128
// (4 waves, 74 KB, two workgroups per CU) for windows of a few hundred rows,
// where writing the fp32 tile takes longer than forming it and the other
// workgroup's loads and MFMAs run meanwhile.
#include <hip/hip_runtime.h>

#include "kernels.hpp"
#include "mfma.hpp"

namespace ambptt {
namespace {

constexpr int kTN = 128;   // dW tile columns (input columns); rows: TM gate rows
constexpr int kS = 64;     // reduction rows per stage
constexpr int kPX = kTN + 16;  // LDS row pitch (bf16) of X: 288 bytes; of Z: TM + 16
constexpr int kPT = kTN + 4;   // pitch (floats) of the staged output rows
static_assert((256 / 2) * kPT * 4 <= 2 * 64 * (256 + 16) * 2, "the staged half tile fits in the Z stages");
static_assert((128 / 2) * kPT * 4 <= 2 * 64 * (128 + 16) * 2, "the staged half tile fits in the Z stages");

typedef short s4 __attribute__((ext_vector_type(4)));
typedef unsigned int u4v __attribute__((ext_vector_type(4)));

// column of element (r, col) of a staged row r (bf16 units): halves swapped for (r >> 3) odd
__device__ __forceinline__ int swz(int r, int col) { return col ^ (64 * ((r >> 3) & 1)); }

// fragment of the 16 x 32 block (columns c0 .. c0 + 15, rows kb .. kb + 31) of a staged operand
__device__ __forceinline__ bf16x8 tr_frag(const __bf16* base, int pitch, int kb, int c0) {
  const int lane = threadIdx.x & 63, g = lane >> 4, i = lane & 15;
  const int r0 = kb + 8 * g + (i >> 2), col = c0 + 4 * (i & 3);
  typedef __attribute__((address_space(3))) s4 lds_s4;
  const s4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4*)(base + r0 * pitch + swz(r0, col)));
  const s4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4*)(base + (r0 + 4) * pitch + swz(r0 + 4, col)));
  typedef short s8 __attribute__((ext_vector_type(8)));
  const s8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, v);
}

template <int TM>
__global__ __launch_bounds__(2 * TM, TM == 128 ? 2 : 1) void dw_bf16(DwArgs a) {
  constexpr int kPZ = TM + 16;  // LDS row pitch (bf16) of Z: 544 or 288 bytes
  constexpr int NT = 2 * TM;    // threads: TM / 32 waves
  constexpr int ZP = TM / 8;    // 16-byte pieces of a Z row of the tile
  constexpr int JZ = 64 * ZP / NT, JX = 64 * (kTN / 8) / NT;  // pieces per thread and stage
  __shared__ __attribute__((aligned(16))) __bf16 Zs[2][kS][kPZ];
  __shared__ __attribute__((aligned(16))) __bf16 Xs[2][kS][kPX];
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int D = a.D, H = a.H, GH = a.GH, R = a.R, N = D + H;
  const int k0 = blockIdx.x * TM, c0 = blockIdx.y * kTN;
  const __bf16* Z = (const __bf16*)a.zbar;
  const __bf16* X = (const __bf16*)a.x;
  const __bf16* Hw = (const __bf16*)a.hwin;

  // loader: 16-byte piece p = tid + NT j; Z: row p / ZP, columns 8 (p % ZP) ..;
  // X: row p >> 4, columns 8 (p & 15) ..  (GH, D, H are multiples of 8: a piece
  // lies wholly inside or outside each operand)
  const int zr = tid / ZP, zc = 8 * (tid % ZP), xr = tid >> 4, xc = 8 * (tid & 15);
  const bool zok = k0 + zc < GH;
  const int xcol = c0 + xc;
  const bool xok = xcol < N;
  const __bf16* zsrc = Z + (zok ? k0 + zc : 0);
  const __bf16* xsrc = xcol < D ? X + xcol : Hw + (xok ? xcol - D : 0);
  const int xld = xcol < D ? D : H;
  // two register sets: stage s is loaded into set s & 1 two stages before
  // its MFMAs, so each load has a whole stage of MFMAs to land behind
  u4v zv[2][JZ], xv[2][JX];
  auto load = [&](int st, int set) {
#pragma unroll
    for (int j = 0; j < JZ; ++j) {
      const int row = st * kS + zr + (NT / ZP) * j;
      zv[set][j] = (zok && row < R) ? *(const u4v*)(zsrc + (size_t)row * GH) : u4v{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int j = 0; j < JX; ++j) {
      const int row = st * kS + xr + (NT / 16) * j;
      xv[set][j] = (xok && row < R) ? *(const u4v*)(xsrc + (size_t)row * xld) : u4v{0u, 0u, 0u, 0u};
    }
  };
  auto stash = [&](int buf, int set) {
#pragma unroll
    for (int j = 0; j < JZ; ++j) {
      const int r = zr + (NT / ZP) * j;
      *(u4v*)&Zs[buf][r][swz(r, zc)] = zv[set][j];
    }
#pragma unroll
    for (int j = 0; j < JX; ++j) {
      const int r = xr + (NT / 16) * j;
      *(u4v*)&Xs[buf][r][swz(r, xc)] = xv[set][j];
    }
  };

  f4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
  float bsum = 0.f;
  const bool do_bias = blockIdx.y == 0 && tid < TM;

  auto compute = [&](int buf) {
#pragma unroll
    for (int kc = 0; kc < kS / 32; ++kc) {
      bf16x8 af[4], bf[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) af[i] = tr_frag(&Zs[buf][0][0], kPZ, 32 * kc, 64 * wm + 16 * i);
#pragma unroll
      for (int j = 0; j < 4; ++j) bf[j] = tr_frag(&Xs[buf][0][0], kPX, 32 * kc, 64 * wn + 16 * j);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = mfma_bf16_16x16x32(af[i], bf[j], acc[i][j]);
    }
    if (do_bias) {
#pragma unroll 8
      for (int rr = 0; rr < kS; ++rr) bsum += (float)Zs[buf][rr][swz(rr, tid)];
    }
  };
  const int nst = (R + kS - 1) / kS;
  // stage st: its rows are in LDS buffer st & 1; stage st + 1's rows are in
  // register set (st + 1) & 1; stage st + 2 is loaded into set st & 1
  auto stage = [&](int st, int p) {  // p = st & 1, a constant in each unrolled half
    if (st + 2 < nst) load(st + 2, p);
    compute(p);
    if (st + 1 < nst) stash(p ^ 1, p ^ 1);  // buffer p ^ 1 was last read before the previous barrier
    __syncthreads();
  };

  load(0, 0);
  if (nst > 1) load(1, 1);
  stash(0, 0);
  __syncthreads();
  int st = 0;
  for (; st + 1 < nst; st += 2) {
    stage(st, 0);
    stage(st + 1, 1);
  }
  if (st < nst) stage(st, 0);
  // The tile goes out through LDS (free after the main loop), TM / 2 rows at
  // a time, so that dW is read and written in whole rows with 16-byte accesses
  // (each 16-lane group of the MFMA layout would touch a 64-byte row segment).
  // Lane l holds, for block (i, j) and v = 0..3, row 4 (l >> 4) + v and column l & 15.
  constexpr int HM = TM / 64 / 2;  // wave rows (wm) per half: the half's rows are theirs
  const int q = lane >> 4, cl = lane & 15;
  float* T = (float*)&Zs[0][0][0];  // TM / 2 x kPT floats (67.6 or 33.8 KB of the 69.6 or 36.9 KB of Zs)
  const bool vec = (N % 4) == 0;
#pragma unroll
  for (int half = 0; half < 2; ++half) {
    if (wm / HM == half) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            T[(64 * (wm % HM) + 16 * i + 4 * q + v) * kPT + 64 * wn + 16 * j + cl] = acc[i][j][v];
    }
    __syncthreads();
    // 32 lanes per row, 4 columns each: NT / 32 rows per pass, 8 passes
#pragma unroll
    for (int p = 0; p < 8; ++p) {
      const int row = (NT / 32) * p + (tid >> 5), c4 = 4 * (tid & 31);
      const int k = k0 + (TM / 2) * half + row, c = c0 + c4;
      if (k >= GH || c >= N) continue;
      float* d = a.dW + (size_t)k * N + c;
      f4 t = *(const f4*)&T[row * kPT + c4];
      if (vec) {  // c + 3 < N: N is a multiple of 4 (of 8, by the launch check)
        if (a.accumulate) t += *(const f4*)d;
        __builtin_nontemporal_store(t, (f4*)d);  // streamed: dW is not read again by this launch
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (c + e < N) d[e] = a.accumulate ? d[e] + t[e] : t[e];
      }
    }
    __syncthreads();  // the next half overwrites T
  }
  if (do_bias && k0 + tid < GH) a.db[k0 + tid] = a.accumulate ? a.db[k0 + tid] + bsum : bsum;
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
  if (a.GH % 8 != 0 || a.D % 8 != 0 || a.H % 8 != 0 || a.R < 1) return hipErrorInvalidValue;
  const int N = a.D + a.H;
  if (a.R <= 512) {  // a few stages: the fp32 tile's write outweighs forming it
    dim3 grid((a.GH + 127) / 128, (N + kTN - 1) / kTN);
    hipExtLaunchKernelGGL(dw_bf16<128>, grid, dim3(256), 0, s, e0, e1, 0, a);
  } else {
    dim3 grid((a.GH + 255) / 256, (N + kTN - 1) / kTN);
    hipExtLaunchKernelGGL(dw_bf16<256>, grid, dim3(512), 0, s, e0, e1, 0, a);
  }
  return hipGetLastError();
}

hipError_t launch_transpose_wh_bf16(const void* W, void* WhT, int GH, int D, int H, hipStream_t s) {
  dim3 grid((GH + 31) / 32, (H + 31) / 32);
  hipLaunchKernelGGL(transpose_wh_u16, grid, dim3(32, 8), 0, s, (const uint16_t*)W, (uint16_t*)WhT, GH, D, H);
  return hipGetLastError();
}

}  // namespace ambptt
