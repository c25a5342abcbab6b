// Internal helpers shared by the library's kernels (gfx950 / CDNA4 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/local.h"

namespace localk {

constexpr int kBlockSize = 16;  // KV tokens per paged block
constexpr int kWave = 64;       // CDNA wavefront width

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// ---------------------------------------------------------------- bf16
__device__ __forceinline__ float bf16_to_f32(uint16_t h) {
  return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

// Round-to-nearest-even float -> bf16 bits (finite inputs; NaN stays NaN).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return 0x7fc0;
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

// Two floats -> packed bf16 pair (low = a), round to nearest even.
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  return static_cast<uint32_t>(f32_to_bf16(a)) |
         (static_cast<uint32_t>(f32_to_bf16(b)) << 16);
}

// ---------------------------------------------------------------- MFMA
// v_mfma_f32_16x16x32_bf16: D[16x16] += A[16x32] * B[32x16].
// Lane l supplies A row (l%16) and B column (l%16), eight k values each for
// k-group l/16; it receives D rows 4*(l/16)+i, column l%16 (i < 4). Both
// operands use the same k-group/element order, so any permutation of k that
// is applied to A and B alike leaves the product unchanged.
__device__ __forceinline__ f32x4 mfma16x16x32(const bf16x8& a, const bf16x8& b,
                                              f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) {
  return __builtin_bit_cast(bf16x8, v);
}

// ---------------------------------------------------------------- loads
template <typename T>
__device__ __forceinline__ T ld_global(const void* p) {
  return *reinterpret_cast<const T*>(p);
}

template <typename T>
__device__ __forceinline__ T ld_stream(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const T*>(p));
}

// ---------------------------------------------------------------- math
__device__ __forceinline__ float fast_exp2(float x) {
  return __builtin_amdgcn_exp2f(x);
}

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

}  // namespace localk

// ---------------------------------------------------------------- status
// Host-side error reporting shared by the entry points (defined in capi.hip).
local_status_t local_fail(local_status_t code, const char* fmt, ...);
local_status_t local_check_launch(const char* what);
