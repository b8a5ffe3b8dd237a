// Device-side helpers shared by the exit-head kernels (gfx950 / CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

namespace ee {

typedef uint16_t bf16_t;  // bfloat16 storage bits

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

// Lambdas that touch register arrays must be inlined: an out-of-line call
// would take the arrays' address and move them to scratch memory.
#define EE_ALWAYS_INLINE __attribute__((always_inline))

// Compile-time loop: f(std::integral_constant<int, I>) for I = 0..N-1, so
// that register arrays indexed by I are never addressed dynamically.
template <class F, int... I>
__device__ __forceinline__ void static_for_impl(F &&f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void static_for(F &&f) {
  static_for_impl(static_cast<F &&>(f), std::make_integer_sequence<int, N>{});
}

// f(integral_constant<bool, a>) for a runtime flag a that is uniform across
// the wave: the branch is taken once, outside f, so the loads inside f are
// never predicated one by one (a predicated load ends in a full vmcnt wait).
template <class F>
__device__ __forceinline__ void with_flag(bool a, F &&f) {
  if (a)
    f(std::true_type{});
  else
    f(std::false_type{});
}

__device__ __forceinline__ float bf16_to_f32(bf16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// Round to nearest even; NaN stays a quiet NaN.  gfx950 lowers the __bf16
// conversion to its hardware convert, which rounds to nearest even.
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  __bf16 h = static_cast<__bf16>(f);
  return __builtin_bit_cast(bf16_t, h);
}

// Storage conversions for the two element types the kernels handle.
template <typename T> __device__ __forceinline__ float to_f32(T v);
template <> __device__ __forceinline__ float to_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f32<bf16_t>(bf16_t v) { return bf16_to_f32(v); }

template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16_t from_f32<bf16_t>(float v) { return f32_to_bf16(v); }

__device__ __forceinline__ float fast_exp(float x) { return __expf(x); }

// sigma(t) = 1 / (1 + exp(-t)) with the hardware exponential and reciprocal
// (about 1 ulp each): exp(-t) overflows to +inf for t < -88, and rcp(inf) = 0
// is the correct limit.
__device__ __forceinline__ float sigmoid_f(float t) { return __builtin_amdgcn_rcpf(1.0f + __expf(-t)); }

__device__ __forceinline__ float silu_f(float t) { return t * sigmoid_f(t); }

// silu(t) = t sigma(t) and d silu / dt = sigma(t) (1 + t (1 - sigma(t))),
// sharing one sigmoid.
__device__ __forceinline__ void silu_and_grad(float t, float &silu, float &grad) {
  const float s = sigmoid_f(t);
  silu = t * s;
  grad = s * (1.0f + t * (1.0f - s));
}

__device__ __forceinline__ float warp_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__device__ __forceinline__ float warp_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

}  // namespace ee
