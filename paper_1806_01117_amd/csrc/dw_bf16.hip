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
// Workgroup: TM / 32 waves on a TM x TN tile of dW, each wave 64 rows x TN / 2
// columns (4 x TN / 32 MFMA blocks); 64 reduction rows per stage,
// double-buffered, the next stage's global reads in flight while the current
// one is multiplied.  LDS rows have a pitch of 32 bytes modulo 256 and rows r
// with (r >> 3) odd have their 64-column groups swapped in pairs, so the 16
// row segments of one transposing read spread over all banks (X rows of 192
// columns are laid out 256 wide for that).  TM = 256 (8 waves, one
// workgroup per CU) for long windows, whose MFMAs dominate: TN = 192 there
// (123 KB of LDS), so that each CU pulls 56 KB of operands and its LDS moves
// 216 KB per 1536 MFMA cycles, where 256 x 128 tiles moved 48 KB and 176 KB
// per 1024; TM = 128, TN = 128 (4 waves, 74 KB, two workgroups per CU) for
// windows of a few hundred rows, where writing the fp32 tile takes longer
// than forming it and the other workgroup's loads and MFMAs run meanwhile.
#include <hip/hip_runtime.h>

#include "kernels.hpp"
#include "mfma.hpp"

namespace ambptt {
namespace {

constexpr int kS = 64;  // reduction rows per stage

typedef short s4 __attribute__((ext_vector_type(4)));
typedef unsigned int u4v __attribute__((ext_vector_type(4)));

// column of element (r, col) of a staged row r (bf16 units): 64-column groups swapped in pairs for (r >> 3) odd
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

template <int TM, int TN>
__global__ __launch_bounds__(2 * TM, TM == 128 ? 2 : 1) void dw_bf16(DwArgs a) {
  constexpr int kPZ = TM + 16;                   // LDS row pitch (bf16) of Z: 544 or 288 bytes
  constexpr int kPX = (TN > 128 ? 256 : TN) + 16;  // of X: 544 or 288 bytes
  constexpr int NT = 2 * TM;                     // threads: TM / 32 waves
  constexpr int NBW = TN / 32;                   // 16-column blocks of a wave
  constexpr int ZP = TM / 8, XP = TN / 8;        // 16-byte pieces of a Z / X row of the tile
  constexpr int JZ = 64 * ZP / NT, JX = 64 * XP / NT;  // pieces per thread and stage
  static_assert(JZ * NT == 64 * ZP && JX * NT == 64 * XP, "loader");
  constexpr int PR = TN > 128 ? 64 : TM / 2;     // rows of the output tile staged per pass
  constexpr int kPT = TN + 4;                    // pitch (floats) of the staged output rows
  static_assert(PR * kPT * 4 <= 2 * kS * kPZ * 2, "a staged pass fits in the Z stages");
  __shared__ __attribute__((aligned(16))) __bf16 Zs[2][kS][kPZ];
  __shared__ __attribute__((aligned(16))) __bf16 Xs[2][kS][kPX];
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int D = a.D, H = a.H, GH = a.GH, R = a.R, N = D + H;
  const int k0 = blockIdx.x * TM, c0 = blockIdx.y * TN;
  const __bf16* Z = (const __bf16*)a.zbar;
  const __bf16* X = (const __bf16*)a.x;
  const __bf16* Hw = (const __bf16*)a.hwin;

  // loader: 16-byte piece p = tid + NT j; Z: row p / ZP, columns 8 (p % ZP) ..;
  // X: row p / XP, columns 8 (p % XP) ..  (GH, D, H are multiples of 8: a piece
  // lies wholly inside or outside each operand)
  const int zr = tid / ZP, zc = 8 * (tid % ZP);
  const bool zok = k0 + zc < GH;
  const __bf16* zsrc = Z + (zok ? k0 + zc : 0);
  int xr[JX], xc[JX];
#pragma unroll
  for (int j = 0; j < JX; ++j) {
    const int p = tid + NT * j;
    xr[j] = p / XP;
    xc[j] = 8 * (p % XP);
  }
  // TN = 192: one register set, stage s loaded while stage s - 1 is
  // multiplied (the registers of a second set would spill); otherwise two
  // sets, stage s loaded two stages before its MFMAs
  constexpr int NSET = TN > 128 ? 1 : 2;
  u4v zv[NSET][JZ], xv[NSET][JX];
  auto load = [&](int st, int set) {
#pragma unroll
    for (int j = 0; j < JZ; ++j) {
      const int row = st * kS + zr + (NT / ZP) * j;
      zv[set][j] = (zok && row < R) ? *(const u4v*)(zsrc + (size_t)row * GH) : u4v{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int j = 0; j < JX; ++j) {  // the piece's source: x, h, or past the last column (zero)
      const int row = st * kS + xr[j], xcol = c0 + xc[j];
      const __bf16* src = xcol < D ? X + (size_t)row * D + xcol : Hw + (size_t)row * H + (xcol < N ? xcol - D : 0);
      xv[set][j] = (xcol < N && row < R) ? *(const u4v*)src : u4v{0u, 0u, 0u, 0u};
    }
  };
  auto stash = [&](int buf, int set) {
#pragma unroll
    for (int j = 0; j < JZ; ++j) {
      const int r = zr + (NT / ZP) * j;
      *(u4v*)&Zs[buf][r][swz(r, zc)] = zv[set][j];
    }
#pragma unroll
    for (int j = 0; j < JX; ++j) *(u4v*)&Xs[buf][xr[j]][swz(xr[j], xc[j])] = xv[set][j];
  };

  f4 acc[4][NBW];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < NBW; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
  float bsum = 0.f;
  const bool do_bias = blockIdx.y == 0 && tid < TM;

  auto compute = [&](int buf) {
#pragma unroll
    for (int kc = 0; kc < kS / 32; ++kc) {
      bf16x8 af[4], bf[NBW];
#pragma unroll
      for (int i = 0; i < 4; ++i) af[i] = tr_frag(&Zs[buf][0][0], kPZ, 32 * kc, 64 * wm + 16 * i);
#pragma unroll
      for (int j = 0; j < NBW; ++j) bf[j] = tr_frag(&Xs[buf][0][0], kPX, 32 * kc, (TN / 2) * wn + 16 * j);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < NBW; ++j) acc[i][j] = mfma_bf16_16x16x32(af[i], bf[j], acc[i][j]);
    }
    if (do_bias) {
#pragma unroll 8
      for (int rr = 0; rr < kS; ++rr) bsum += (float)Zs[buf][rr][swz(rr, tid)];
    }
  };
  const int nst = (R + kS - 1) / kS;
  // stage st: its rows are in LDS buffer st & 1; two sets: stage st + 1's
  // rows are in register set (st + 1) & 1 and stage st + 2 is loaded into set
  // st & 1; one set: stage st + 1 is loaded now and stashed after the MFMAs
  auto stage = [&](int st, int p) {  // p = st & 1, a constant in each unrolled half
    if (NSET == 2) {
      if (st + 2 < nst) load(st + 2, p);
    } else {
      if (st + 1 < nst) load(st + 1, 0);
    }
    compute(p);
    if (st + 1 < nst) stash(p ^ 1, NSET == 2 ? p ^ 1 : 0);  // buffer p ^ 1 was last read before the previous barrier
    __syncthreads();
  };

  load(0, 0);
  stash(0, 0);
  if (NSET == 2 && nst > 1) load(1, 1);
  __syncthreads();
  int st = 0;
  for (; st + 1 < nst; st += 2) {
    stage(st, 0);
    stage(st + 1, 1);
  }
  if (st < nst) stage(st, 0);
  // The tile goes out through LDS (free after the main loop), PR rows at a
  // time, so that dW is read and written in whole rows with 16-byte accesses
  // (each 16-lane group of the MFMA layout would touch a 64-byte row segment).
  // Lane l holds, for block (i, j) and v = 0..3, row 4 (l >> 4) + v and column l & 15.
  constexpr int HM = PR / 64;  // wave rows (wm) per pass: the pass's rows are theirs
  constexpr int LPR = TN / 4;  // threads per output row, 4 columns each
  const int q = lane >> 4, cl = lane & 15;
  float* T = (float*)&Zs[0][0][0];
  const bool vec = (N % 4) == 0;
#pragma unroll
  for (int pass = 0; pass < TM / PR; ++pass) {
    if (wm / HM == pass) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v)
#pragma unroll
          for (int j = 0; j < NBW; ++j)
            T[(64 * (wm % HM) + 16 * i + 4 * q + v) * kPT + (TN / 2) * wn + 16 * j + cl] = acc[i][j][v];
    }
    __syncthreads();
    for (int idx = tid; idx < PR * LPR; idx += NT) {
      const int row = idx / LPR, c4 = 4 * (idx % LPR);
      const int k = k0 + PR * pass + row, c = c0 + c4;
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
    __syncthreads();  // the next pass overwrites T
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
    dim3 grid((a.GH + 127) / 128, (N + 127) / 128);
    hipExtLaunchKernelGGL((dw_bf16<128, 128>), grid, dim3(256), 0, s, e0, e1, 0, a);
  } else {
    dim3 grid((a.GH + 255) / 256, (N + 191) / 192);
    hipExtLaunchKernelGGL((dw_bf16<256, 192>), grid, dim3(512), 0, s, e0, e1, 0, a);
  }
  return hipGetLastError();
}

hipError_t launch_transpose_wh_bf16(const void* W, void* WhT, int GH, int D, int H, hipStream_t s) {
  dim3 grid((GH + 31) / 32, (H + 31) / 32);
  hipLaunchKernelGGL(transpose_wh_u16, grid, dim3(32, 8), 0, s, (const uint16_t*)W, (uint16_t*)WhT, GH, D, H);
  return hipGetLastError();
}

}  // namespace ambptt
