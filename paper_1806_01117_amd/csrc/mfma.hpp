// Device-side MFMA helpers shared by the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>

namespace ambptt {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ f4 mfma_f32_16x16x4(float a, float b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// v_mfma_f32_16x16x32_bf16 followed by four explicit wait states.  With the
// ROCm 7.2 compiler, a vector instruction that overwrote one of this MFMA's
// A/B source registers right after it was issued corrupted the product (the
// bf16 step kernels disagreed with the float64 reference by ~25% until the
// pad was added; the pad after the last MFMA alone did not help, so the
// hazard is on the sources).  The pad costs ~4 cycles per 16x16x32 MFMA.
__device__ __forceinline__ f4 mfma_bf16_16x16x32(const bf16x8& a, const bf16x8& b, f4 c) {
  c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  asm volatile("s_nop 3" ::: "memory");
  return c;
}

}  // namespace ambptt
