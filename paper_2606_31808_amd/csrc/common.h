// Device-side types shared by the gfx950 kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef _Float16 f16;
typedef f16 f16x2 __attribute__((ext_vector_type(2)));
typedef f16 f16x4 __attribute__((ext_vector_type(4)));
typedef f16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

#define LMOP_DEVICE __device__ __forceinline__

// v_mfma_f32_16x16x32_f16 (CDNA4).  Operand layout (wave64, lane = 16*g + c):
//   A: lane holds A[row c][k 8g .. 8g+7]      B: lane holds B[k 8g .. 8g+7][col c]
//   D: lane holds D[row 4g + r][col c], r = 0..3
LMOP_DEVICE f32x4 mfma16x16x32(f16x8 a, f16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

template <typename T>
LMOP_DEVICE T shfl_xor(T v, int mask) {
  return __shfl_xor(v, mask, 64);
}
