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

// v_mfma_f32_16x16x16_bf16: D[16x16] += A[16x16] * B[16x16], four k values
// per lane (k-group l/16), same row/column/accumulator layout as above.
__device__ __forceinline__ f32x4 mfma16x16x16(const bf16x4& a, const bf16x4& b, f32x4 c) {
  typedef short s16x4 __attribute__((ext_vector_type(4)));
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4, a),
                                                   __builtin_bit_cast(s16x4, b), c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) {
  return __builtin_bit_cast(bf16x8, v);
}

__device__ __forceinline__ bf16x4 as_bf16x4(u32x2 v) {
  return __builtin_bit_cast(bf16x4, v);
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

// Buffer loads: a descriptor covers [base, base + bytes); a load outside it
// returns zeros and issues no memory request, so a zero-size descriptor is a
// free "absent" load that keeps the instruction stream branch-free.
constexpr int32_t kBufferConfig = 0x00020000;  // CDNA raw-buffer descriptor word 3

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), static_cast<short>(0),
                                           static_cast<int>(bytes), kBufferConfig);
}

__device__ __forceinline__ u32x4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, static_cast<int>(byte_off), 0, 0);
}

__device__ __forceinline__ u32x2 buf_load8(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_amdgcn_raw_buffer_load_b64(r, static_cast<int>(byte_off), 0, 0);
}

// Streaming (non-temporal) variants for data read once per call, such as the
// KV blocks of decode attention: the loads carry the nt cache policy, which
// on gfx950 lets a pure read stream reach about 7 TB/s instead of about 6.3.
constexpr int kCacheStream = 2;  // cache-policy operand: nt

__device__ __forceinline__ u32x4 buf_load16_stream(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, static_cast<int>(byte_off), 0, kCacheStream);
}

__device__ __forceinline__ u32x2 buf_load8_stream(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_amdgcn_raw_buffer_load_b64(r, static_cast<int>(byte_off), 0, kCacheStream);
}

// ---------------------------------------------------------------- lanes
// max(a, b) in one instruction: fmaxf of values the compiler cannot prove
// canonical (a lane swap's result, say) adds a NaN-quieting maximum per
// operand. The operands here are never NaN.
__device__ __forceinline__ float max2f(float a, float b) {
  float r;
  asm("v_max_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}

// Maximum of v over lanes l and l ^ 16 (l ^ 32), by the gfx950 lane swaps of
// the vector unit (no LDS round trip): swapping a register with itself
// leaves each lane its own value in one result and its partner's in the
// other, so their maximum is the pair's.
__device__ __forceinline__ float max_xor16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                  false);
  return max2f(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float max_xor32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                  false);
  return max2f(__uint_as_float(r[0]), __uint_as_float(r[1]));
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
