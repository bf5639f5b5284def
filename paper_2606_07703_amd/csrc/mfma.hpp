// gfx950 bf16 MFMA fragments.
//
// v_mfma_f32_16x16x32_bf16, for C[16x16] += A[16x32] * B[32x16], with lane
// l (0..63), g = l/16:
//   A: lane l holds row l%16, columns 8g..8g+7 (8 bf16, 16 bytes)
//   B: lane l holds column l%16, rows 8g..8g+7
//   C: lane l holds column l%16, rows 4g..4g+3 (4 floats)
// These layouts were checked on the device against a host matmul.
//
// v_mfma_f32_32x32x16_bf16, for C[32x32] += A[32x16] * B[16x32], with lane
// l, n = l%32, h = l/32:
//   A: lane l holds row n, columns 8h..8h+7
//   B: lane l holds column n, rows 8h..8h+7
//   C: lane l holds column n; element 4i+r (i, r in 0..3) is row 8i + 4h + r
// It retires twice the work of the 16x16x32 form per instruction, and on
// gfx950 it sustains a higher share of the bf16 peak in long chains.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sp {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ f32x4 mfma16(const bf16x8 &a, const bf16x8 &b, const f32x4 &c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x16 mfma32(const bf16x8 &a, const bf16x8 &b, const f32x16 &c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 as_bf16x8(const uint4 &u) {
  bf16x8 r;
  __builtin_memcpy(&r, &u, sizeof(r));
  return r;
}

__device__ __forceinline__ uint4 ldg16(const void *p) {
  return *reinterpret_cast<const uint4 *>(p);
}

__device__ __forceinline__ uint4 lds16(const void *p) {
  return *reinterpret_cast<const uint4 *>(p);
}

__device__ __forceinline__ void sts16(void *p, const uint4 &v) {
  *reinterpret_cast<uint4 *>(p) = v;
}

}  // namespace sp
