// Device kernels of one recurrent step and of the weight-gradient windows,
// with their host launchers.  Host code includes this header; the kernels
// live in the .hip files.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "resident_prog.hpp"

namespace ambptt {

// Arguments of one step kernel.  G = 1 (tanh RNN) or 4 (LSTM, gate blocks
// i, f, g, o).  Layouts are row-major with batch rows.  "op" pointers hold the
// operand dtype (fp32 or bf16); the cell state, its adjoint, biases and
// gradients are fp32.
struct StepArgs {
  const void* x;         // op: x_t [B][D]
  const void* h;         // op: h_t [B][H]
  const float* c;        // c_t [B][H] (LSTM)
  void* h_out;           // op: forward: h_{t+1} [B][H]
  float* c_out;          // forward: c_{t+1} [B][H] (LSTM)
  const void* W;         // op: [G*H][D+H]
  const float* bias;     // [G*H]
  const void* WhT;       // op: [H][G*H]: WhT[j][k] = W[k][D+j]
  const void* zbar_in;   // op: adjoint: zbar_{t+1} [B][G*H] (unused when first)
  const float* cbar_in;  // adjoint: cbar_{t+1} [B][H] (LSTM; unused when first)
  void* zbar_out;        // op: adjoint: zbar_t [B][G*H]
  float* cbar_out;       // adjoint: cbar_t [B][H] (LSTM)
  void* hwin_out;        // op: adjoint: copy of h_t for the weight-gradient window
  const float* hbar_in;  // wide-batch adjoint: hbar_{t+1} = zbar_{t+1} W_h [B][H] (unused when first)
  double* loss_acc;      // adjoint: one accumulator per workgroup
  float* dh0;            // final: dL/dh_0 [B][H]
  float* dc0;            // final: dL/dc_0 [B][H] (LSTM)
  int B, D, H;
  int loss;              // AMBPTT_LOSS_*
  int first;             // adjoint of step n-1: no incoming adjoint
  int last;              // the step's output is x_n
  float inv_bh;          // 1 / (B H)
  int ld_wht = 0;        // row stride of WhT in elements (0: G*H)
  int hbar_parts = 1;    // hbar_in holds this many [B][H] partial sums, added in order
};

// Weight-gradient window: dW[k][c] += sum_r Z[r][k] X[r][c], db[k] += sum_r Z[r][k],
// where X[r] = [x row | h row] for the R = w*B rows of w consecutive steps.
struct DwArgs {
  const void* zbar;  // op: [R][G*H]
  const void* x;     // op: [R][D]
  const void* hwin;  // op: [R][H]
  float* dW;         // [G*H][D+H]
  float* db;         // [G*H]
  int R, D, H, GH;
  int accumulate;    // 1: dW += ..., 0: dW = ... (one window per weight set)
};

// Arguments of one residual-MLP step kernel (layer l).
struct MlpArgs {
  const void* y;          // op: y_l [B][w]
  void* y_out;            // op: forward: y_{l+1}
  const void* W;          // op: W_l [w][w]
  const float* bias;      // b_l [w]
  const void* Wn;         // op: adjoint: W_{l+1}; final: W_0
  const void* zbar_in;    // op: adjoint: zbar_{l+1}; final: zbar_0
  const float* ybar_in;   // adjoint: ybar_{l+2}; final: ybar_1
  void* zbar_out;         // op: zbar_l
  float* ybar_out;        // ybar_{l+1}
  void* ywin_out;         // op: copy of y_l for the weight gradient
  const float* nn_in;     // wide-batch adjoint: ybar_{l+2} + zbar_{l+1} W_{l+1} [B][w] (unused when first)
  double* loss_acc;
  float* dy0;
  int B, w, loss, first;
  float inv_bw;
};

// One product of the wide-batch adjoint: out = add (if given) + A Bm, A [M][K]
// bf16 row-major; Bm(k, n) = B[n][k] ("NT", the cell's W_h^T) or B[k][n]
// ("NN", the MLP's W_{l+1}); out and add fp32 [M][N].
struct ProdArgs {
  const void* A;
  const void* B;
  const float* add;
  float* out;
  int M, N, K;
  int ldb = 0;  // row stride of B in elements (0: K)
};

// One launch of the MLP whose layers change width (mlp_f32.hip):
//   kForward  out = relu(A W^T + bias)                  A [M][K], W [N][K]
//   kAdjoint  zbar_out = (nn_in + dL/dy') * 1[A W^T + bias > 0], y' = relu(...),
//             its loss term added to loss_acc[workgroup]
//   kFinal    out = A W (+ add)                          A [M][K], W [K][N]
// M >= 1 rows; N and K multiples of 16.  inv = 1 / (M N) of the layer's output.
struct MlpvArgs {
  const float* A;
  const float* W;
  const float* bias;
  const float* add;
  float* out;
  const float* nn_in;  // adjoint: zbar_{l+1} W_{l+1} [M][N], NULL for the last layer
  float* zbar_out;
  float* ywin_out;     // adjoint: a copy of A (y_l) for the weight gradient, NULL for none
  const float* A2;     // adjoint in one launch: zbar_{l+1} [M][K2], NULL: nn_in (or nothing) instead
  const float* W2;     // W_{l+1} [K2][N]
  double* loss_acc;
  int M, N, K, K2;
  int loss, last;
  float inv;
};

enum StepMode { kForward = 0, kAdjoint = 1, kFinal = 2 };

// Resident whole-pass kernel (fp32 tanh RNN / LSTM with small states): one
// launch runs a program compiled from the schedule (resident_prog.hpp).
struct ResidentArgs {
  const int* prog;      // [nprog][4]
  int nprog;
  const float* x;       // [n][B][D]
  const float* W;       // [G*H][D+H]
  const float* bias;    // [G*H]
  char* pool;           // slot k at pool + k * stride
  char* live0;
  char* live1;
  size_t stride;        // bytes between slots
  size_t c_off;         // byte offset of c within a state (LSTM)
  int nslots;
  char* host;           // host tier (device-visible): [host slot][workgroup][1 KiB]
  float* Z;             // zbar slices for the octets [2][mtiles][ng][16][G U]
  float* P;             // octet partial h-adjoints [2][mtiles][ng / S][H][16]
  float* dWp;           // per row tile dW partials [mtiles][G*H][D+H]
  float* dbp;           // [mtiles][G*H]
  float* dh0;           // [B][H]
  float* dc0;           // [B][H] (LSTM)
  double* loss_acc;     // [mtiles * ng]
  unsigned* ready;      // [mtiles * ng] syncs entered (zero before launch)
  unsigned* consumed;   // [mtiles * ng] syncs whose inputs are read (zero before launch)
  unsigned* oflag;      // [mtiles * ng] adjoint steps whose zbar slice is out (zero before launch)
  unsigned* status;     // [0]: abort flag, [1]: op index of the abort + 1
  long long timeout;    // s_memrealtime ticks (100 MHz) a wait may take
  int B, D, H, loss;
  int mtiles, ng;       // row tiles (16 rows); unit groups per row tile
  int S;                // octet size: min(8, ng), dividing ng, with H / S <= 64
  int xcd_map;          // 1: place each row tile's workgroups on 8 / mtiles XCDs
  float inv_bh;
};

// units per workgroup of the resident kernel (8 LSTM, 16 RNN)
int resident_units(int G);
// largest D + H and H the resident kernel holds in registers
int resident_max_k(int G);
int resident_max_h(int G);
// octet size for ng unit groups of hidden size H (0: the kernel cannot take it)
int resident_octet(int ng, int H);
// workgroups of the resident kernel variant that (G, D, H) launches that can
// be resident at once on the current device
hipError_t resident_capacity(int G, int D, int H, int* blocks);
// cooperative: hipLaunchCooperativeKernel (the runtime guarantees that the
// whole grid is resident); otherwise a plain launch of a grid that fits
hipError_t launch_resident(int G, const ResidentArgs& a, hipStream_t s, bool cooperative);
// dW = sum over row tiles of dWp (fixed order), db likewise
hipError_t launch_resident_reduce(const float* dWp, const float* dbp, int mtiles, int GH, int K1, float* dW,
                                  float* db, hipStream_t s);

struct StepCfg {
  int rm, rj, ks;  // 16x16 tiles per wave in m and j; waves splitting K
};

StepCfg pick_step_cfg(int G, int B, int D, int H);
void step_grid(const StepCfg& cfg, int B, int H, dim3* grid, dim3* block);
// Launchers take an optional pair of events that the dispatch itself records
// at kernel start and end (hipExtLaunchKernel); pass nullptr for none.
hipError_t launch_step(int G, int mode, const StepCfg& cfg, const StepArgs& a, hipStream_t s,
                       hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr);
hipError_t launch_dw(const DwArgs& a, hipStream_t s, hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr);
// fp32 out = A B^T (+ add): the adjoint's h-adjoint product zbar W_h through W_h^T (K % 16 == 0, N % 16 == 0)
hipError_t launch_prod_f32(const ProdArgs& a, hipStream_t s, hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr);
// LDS-tiled fp32 kernels for large batches (gemm_f32.hip): the gate product
// with the cell epilogue on 128 x 256 tiles (forward, and the adjoint when its
// h-adjoint product runs as a launch of its own), and that product on
// 64 x 128 tiles.  *_fits: the shape constraints; *_tiles: workgroups.
bool cell_gemm_f32_fits(int G, int B, int D, int H);
int cell_gemm_f32_tiles(int G, int B, int H);
hipError_t launch_cell_gemm_f32(int G, int mode, const StepArgs& a, hipStream_t s, hipEvent_t e0 = nullptr,
                                hipEvent_t e1 = nullptr);
bool prod_gemm_f32_fits(int M, int N, int K);
int prod_gemm_f32_tiles(int M, int N);
hipError_t launch_prod_gemm_f32(const ProdArgs& a, hipStream_t s, hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr);
// The same product on 128 x 128 tiles with the reduction split `parts` ways:
// part s goes to out + s M N (no add).  kProdSplitMax parts at most.
constexpr int kProdSplitMax = 4;
int prod_split_f32_parts(int M, int N, int K);  // 1: the split does not fit or does not pay
hipError_t launch_prod_split_f32(const ProdArgs& a, int parts, hipStream_t s, hipEvent_t e0 = nullptr,
                                 hipEvent_t e1 = nullptr);
// 128 x 128-tile fp32 weight gradient for GH, D + H >= 256 (launch_dw picks it when it fits).
bool dw_f32_big_fits(const DwArgs& a);
hipError_t launch_dw_f32_big(const DwArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1);
// Small-batch path: one launch per step, 16 rows x (8 LSTM | 16 RNN) units per workgroup.
void step_small_grid(int G, int B, int H, dim3* grid, dim3* block);
hipError_t launch_step_small(int G, int bf16, int mode, const StepArgs& a, hipStream_t s,
                             hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr);
void resmlp_grid(int B, int w, dim3* grid, dim3* block);
hipError_t launch_resmlp(int bf16, int mode, const MlpArgs& a, hipStream_t s, hipEvent_t e0 = nullptr,
                         hipEvent_t e1 = nullptr);
// Wide-batch bf16 path (B >= 48): the cell kernel takes 64 rows x 64 gate
// columns per workgroup; the adjoint's products run as launches of their own.
// The cell's a.W and the NT product's B are fragment-order copies made by
// launch_pack_nt_bf16 (of W [G H][D + H] and of W_h^T [H][G H]).
bool cell_wide_fits(int G, int B, int D, int H);  // D and H multiples of 64, operands under 4 GiB
bool mlp_wide_fits(int B, int w);                  // w a multiple of 64, operands under 4 GiB
int cell_wide_tiles(int G, int B, int H);
hipError_t launch_cell_wide(int G, int mode, const StepArgs& a, hipStream_t s, hipEvent_t e0 = nullptr,
                            hipEvent_t e1 = nullptr);
hipError_t launch_prod_nt(const ProdArgs& a, hipStream_t s, hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr);
// dst (N K bf16, fragment order) <- the [N][K] bf16 rows of src with row stride ld
hipError_t launch_pack_nt_bf16(const void* src, int N, int K, int ld, void* dst, hipStream_t s);
hipError_t launch_prod_nn(const ProdArgs& a, hipStream_t s, hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr);
int mlp_wide_tiles(int B, int w);
hipError_t launch_mlp_wide(int mode, const MlpArgs& a, hipStream_t s, hipEvent_t e0 = nullptr,
                           hipEvent_t e1 = nullptr);
hipError_t launch_dw_bf16(const DwArgs& a, hipStream_t s, hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr);
// The MLP of layers of different widths: workgroups of one launch on M x N,
// and the launch (mode kForward, kAdjoint, or kFinal for the NN product).
int mlpv_tiles(int M, int N);
hipError_t launch_mlpv(int mode, const MlpvArgs& a, hipStream_t s, hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr);
// The weight gradients of up to kMlpvDwGroup layers in one launch: member i
// is dW = zbar^T y [GH][H] and db, written (accumulate 0) or added, with
// zbar = DwArgs::zbar [R][GH], y = DwArgs::hwin [R][H].
constexpr int kMlpvDwGroup = 8;
hipError_t launch_mlpv_dw(const DwArgs* a, int count, hipStream_t s, hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr);
hipError_t launch_transpose_wh_bf16(const void* W, void* WhT, int GH, int D, int H, hipStream_t s);
// WhT[j][k] = W[k][D + j] with rows of ld >= GH floats
hipError_t launch_transpose_wh(const float* W, float* WhT, int GH, int D, int H, int ld, hipStream_t s);
hipError_t launch_fill32(void* p, size_t words, uint32_t value, hipStream_t s);
hipError_t launch_loss_sum(const double* acc, int n, double scale, double* out, hipStream_t s);

}  // namespace ambptt
