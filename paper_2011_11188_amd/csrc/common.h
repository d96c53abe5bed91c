// Device-side helpers shared by the mdnn kernels (gfx950 / CDNA4 only).
//
// Storage types: fp32, IEEE fp16 and bfloat16 (section 3.2 of the paper).
// 16-bit values are moved as raw uint16_t bit patterns; arithmetic is fp32.
// Every narrowing conversion rounds to nearest even, keeps fp16 subnormals,
// overflows to +-inf and keeps NaN.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/mdnn.h"

namespace mdnn {

typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bhalf8_t __attribute__((ext_vector_type(8)));
typedef float float4_t __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------------------
// element type tags
// ---------------------------------------------------------------------------
struct F32 {
  typedef float storage;
  static constexpr mdnn_dtype_t id = MDNN_F32;
};
struct F16 {
  typedef uint16_t storage;
  static constexpr mdnn_dtype_t id = MDNN_F16;
};
struct BF16 {
  typedef uint16_t storage;
  static constexpr mdnn_dtype_t id = MDNN_BF16;
};

__device__ __forceinline__ float f16_to_f32(uint16_t u) {
  return (float)__builtin_bit_cast(_Float16, u);
}
__device__ __forceinline__ uint16_t f32_to_f16(float x) {
  // v_cvt_f16_f32 under the default round-to-nearest-even mode; fp16
  // denormals are enabled by default on gfx9.
  return __builtin_bit_cast(uint16_t, (_Float16)x);
}
__device__ __forceinline__ float bf16_to_f32(uint16_t u) {
  return __builtin_bit_cast(float, (uint32_t)u << 16);
}
__device__ __forceinline__ uint16_t f32_to_bf16(float x) {
  uint32_t u = __builtin_bit_cast(uint32_t, x);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x0040u);  // quiet NaN
  u += 0x7fffu + ((u >> 16) & 1u);  // ties to even; carries into the exponent, inf on overflow
  return (uint16_t)(u >> 16);
}

template <class T> __device__ __forceinline__ float load_f(const typename T::storage* p);
template <> __device__ __forceinline__ float load_f<F32>(const float* p) { return *p; }
template <> __device__ __forceinline__ float load_f<F16>(const uint16_t* p) { return f16_to_f32(*p); }
template <> __device__ __forceinline__ float load_f<BF16>(const uint16_t* p) { return bf16_to_f32(*p); }

template <class T> __device__ __forceinline__ float to_f(typename T::storage v);
template <> __device__ __forceinline__ float to_f<F32>(float v) { return v; }
template <> __device__ __forceinline__ float to_f<F16>(uint16_t v) { return f16_to_f32(v); }
template <> __device__ __forceinline__ float to_f<BF16>(uint16_t v) { return bf16_to_f32(v); }

template <class T> __device__ __forceinline__ typename T::storage from_f(float v);
template <> __device__ __forceinline__ float from_f<F32>(float v) { return v; }
template <> __device__ __forceinline__ uint16_t from_f<F16>(float v) { return f32_to_f16(v); }
template <> __device__ __forceinline__ uint16_t from_f<BF16>(float v) { return f32_to_bf16(v); }

__device__ __forceinline__ float relu_f(float v) { return v < 0.0f ? 0.0f : v; }  // keeps NaN

__host__ __device__ constexpr int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace mdnn
