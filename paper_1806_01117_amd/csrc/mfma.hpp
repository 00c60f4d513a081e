// Device-side MFMA helpers shared by the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>

namespace ambptt {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ f4 mfma_f32_16x16x4(float a, float b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// v_mfma_f32_16x16x32_bf16 followed by an empty asm statement with a memory
// clobber, which keeps LDS and global accesses from moving across it.  With
// nothing after the MFMA, the ROCm 7.2 build of the small-batch bf16 step
// kernel gives wrong results (loss off by 180 %); with this statement, or
// with an `s_nop 3` without the clobber, every bf16 kernel is bit-exact
// across schedules and within tolerance of the float64 oracle.  In the ISA of
// the failing build the only pattern its passing builds lack is a VALU write
// of the MFMA's B register in the very next cycle, but the weight-gradient
// kernel holds such writes in every build and is correct, so the mechanism
// is not established; the GPU tests of every bf16 kernel are the check.  Of
// the two statements the clobber is also the faster: with `s_nop 3` the wide
// kernels' passes ran 2.7 % (residual MLP) and 3.1 % (2048-LSTM) slower.
__device__ __forceinline__ f4 mfma_bf16_16x16x32(const bf16x8& a, const bf16x8& b, f4 c) {
  c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  asm volatile("" ::: "memory");
  return c;
}

}  // namespace ambptt
