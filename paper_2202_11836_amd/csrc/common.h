// Device-side helpers shared by the encoder-stage kernels (gfx950 / CDNA4).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

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

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// fp32 -> bf16, round to nearest even (the hardware conversion).
__device__ __forceinline__ bf16_t f2bf(float f) { return __builtin_bit_cast(bf16_t, (__bf16)f); }

// Two fp32 values -> one packed pair of bf16 (lo in bits 0-15), round to
// nearest even, in a single conversion instruction.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
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

// Transposing LDS read ds_read_b64_tr_b16 (gfx950) as inline assembly.
// With the compiler builtin for it, the compiler first waits for every
// direct-to-LDS load the wavefront has in flight (vmcnt 0: it cannot tell
// which LDS bytes they write), which drains a prefetch ring whose next
// loads were issued just before; the kernels wait for those loads
// explicitly instead.  The compiler does not track this read either: every
// result must pass lds_wait() and then lds_hold() before any use, and must
// stay live until then (its register could otherwise be reused while the
// read is in flight).
// OFF: a constant byte offset, carried in the instruction's offset field.
template <int OFF = 0>
__device__ __forceinline__ u32x2_t ds_read_tr16_b64(uint32_t lds_addr) {
  static_assert(OFF >= 0 && OFF < 65536, "LDS instruction offset range");
  u32x2_t r;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(lds_addr), "i"(OFF));
  return r;
}

// f(std::integral_constant<int, I>()) for I = B .. E - 1: a loop whose index
// is a constant expression in the body.
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>());
    static_for<B + 1, E>(f);
  }
}
// Wait for this wavefront's outstanding LDS operations (lgkmcnt = 0).
__device__ __forceinline__ void lds_wait() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
// Orders the uses of v after the preceding lds_wait() (emits nothing).
__device__ __forceinline__ void lds_hold(u32x2_t& v) { asm volatile("" : "+v"(v)); }

// GELU u * Phi(u) = u/2 * (1 + erf(u / sqrt 2)) and its derivative
// Phi(u) + u * phi(u).  erfc(|u| / sqrt 2) is evaluated with the rational
// approximation of Abramowitz & Stegun, Handbook of Mathematical Functions,
// formula 7.1.26 (after Hastings): erfc(x) = (a1 t + ... + a5 t^5) exp(-x^2),
// t = 1 / (1 + p x), x >= 0, |error| <= 1.5e-7, with its coefficients halved
// so that the polynomial yields erfc / 2 = min(Phi(u), 1 - Phi(u)) directly.
// It is branch-free, and exp(-x^2) = exp(-u^2 / 2) is shared with the
// derivative.
struct GeluParts {
  float cdf;  // Phi(u), without cancellation for u < 0
  float e;    // exp(-u^2 / 2)
};
__device__ __forceinline__ GeluParts gelu_parts(float u) {
  const float t = __builtin_amdgcn_rcpf(fmaf(fabsf(u), 0.3275911f * 0.70710678118654752f, 1.0f));
  const float hp =
      t * fmaf(t, fmaf(t, fmaf(t, fmaf(t, 0.5307027145f, -0.7265760135f), 0.7107068705f),
                       -0.142248368f),
               0.127414796f);
  const float e = __builtin_amdgcn_exp2f(u * (u * -0.72134752044448170f));  // exp(-u^2/2)
  const float h = hp * e;  // erfc(|u| / sqrt 2) / 2
  return {u < 0.0f ? h : 1.0f - h, e};
}
__device__ __forceinline__ float gelu_f(float u) { return u * gelu_parts(u).cdf; }
__device__ __forceinline__ float gelu_grad_f(float u) {
  const GeluParts p = gelu_parts(u);
  return fmaf(u * 0.39894228040143268f, p.e, p.cdf);
}

// One block (256 threads) of a column reduction: out[c .. c + 15] (16
// columns from bx * 16) = the sum over partial rows b < nblk of
// part[(b * nvec + v) * n + c]; 4 threads x 4 columns per partial row, 64
// stripes of rows, the stripe sums combined in LDS (sm) by a fixed-order
// tree.  out may be null (nothing stored).
__device__ __forceinline__ void colred_block(const float* __restrict__ part, int nblk, int nvec,
                                             int n, int v, int bx, float* out, f32x4_t (*sm)[4]) {
  const int q = threadIdx.x & 3, stripe = threadIdx.x >> 2;
  const int c = bx * 16 + 4 * q;
  f32x4_t s = {0.0f, 0.0f, 0.0f, 0.0f};
  if (c < n) {
#pragma unroll 8
    for (int b = stripe; b < nblk; b += 64) s += *(const f32x4_t*)(part + ((int64_t)b * nvec + v) * n + c);
  }
  sm[stripe][q] = s;
  __syncthreads();
  for (int w = 32; w > 0; w >>= 1) {
    if (stripe < w) sm[stripe][q] += sm[stripe + w][q];
    __syncthreads();
  }
  if (stripe == 0 && c < n && out) *(f32x4_t*)(out + c) = sm[0][q];
}
