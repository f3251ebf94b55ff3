// Device-side helpers shared by the encoder-stage kernels (gfx950 / CDNA4).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef uint16_t bf16_t;  // bfloat16 storage (upper half of an fp32)

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

#define WAVE 64

__device__ __forceinline__ float bf2f(bf16_t v) {
  return __uint_as_float(((uint32_t)v) << 16);
}

// Round-to-nearest-even fp32 -> bf16 (NaN kept quiet).
__device__ __forceinline__ bf16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (bf16_t)((u >> 16) | 0x40);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

// Storage conversions: T is float or bf16_t.
template <typename T> __device__ __forceinline__ float ld_f(const T* p);
template <> __device__ __forceinline__ float ld_f<float>(const float* p) { return *p; }
template <> __device__ __forceinline__ float ld_f<bf16_t>(const bf16_t* p) { return bf2f(*p); }

template <typename T> __device__ __forceinline__ void st_f(T* p, float v);
template <> __device__ __forceinline__ void st_f<float>(float* p, float v) { *p = v; }
template <> __device__ __forceinline__ void st_f<bf16_t>(bf16_t* p, float v) { *p = f2bf(v); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, WAVE);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, WAVE));
  return v;
}

// GELU u * Phi(u) = u/2 * (1 + erf(u / sqrt 2)) and its derivative
// Phi(u) + u * phi(u).  erf is evaluated with the rational approximation of
// Abramowitz & Stegun, Handbook of Mathematical Functions, formula 7.1.26
// (after Hastings): erf(x) = 1 - (a1 t + ... + a5 t^5) exp(-x^2),
// t = 1 / (1 + p x), x >= 0, |error| <= 1.5e-7.  It is branch-free, and the
// exp(-x^2) = exp(-u^2 / 2) term is shared with the derivative.
struct ErfParts {
  float onep;  // 1 + erf(u / sqrt 2) = 2 Phi(u), without cancellation for u < 0
  float e;     // exp(-u^2 / 2)
};
__device__ __forceinline__ ErfParts erf_parts(float u) {
  const float x = u * 0.70710678118654752f;
  const float ax = fabsf(x);
  const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, ax, 1.0f));
  const float poly =
      t * fmaf(t, fmaf(t, fmaf(t, fmaf(t, 1.061405429f, -1.453152027f), 1.421413741f),
                       -0.284496736f),
               0.254829592f);
  const float e = __builtin_amdgcn_exp2f(-x * x * 1.4426950408889634f);
  const float erfc_ax = poly * e;  // 1 - erf(|x|)
  return {x < 0.0f ? erfc_ax : 2.0f - erfc_ax, e};
}
__device__ __forceinline__ float gelu_f(float u) {
  const ErfParts p = erf_parts(u);
  return 0.5f * u * p.onep;
}
__device__ __forceinline__ float gelu_grad_f(float u) {
  const ErfParts p = erf_parts(u);
  return fmaf(u * 0.39894228040143268f, p.e, 0.5f * p.onep);
}
