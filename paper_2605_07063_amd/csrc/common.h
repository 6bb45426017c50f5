// Internal helpers shared by the library's translation units (not part of
// the C ABI).  gfx950 only.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dr_api.h"

namespace dr {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;

// 16x16x32 bf16 MFMA, fp32 accumulate.  Lane l supplies A[l%16][8*(l/16)..+8]
// and B[8*(l/16)..+8][l%16]; C[4*(l/16)+j][l%16] lands in register j.
__device__ __forceinline__ f32x4 mma_bf16(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// 16x16x4 fp32 MFMA.  Lane l supplies A[l%16][l/16] and B[l/16][l%16]; the
// C layout is the same as for mma_bf16.
__device__ __forceinline__ f32x4 mma_f32(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

inline dr_status launch_status() {
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? DR_OK : DR_ERR_HIP;
}

inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

}  // namespace dr
