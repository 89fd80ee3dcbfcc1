// Device-side helpers shared by the HIP kernels: bfloat16 storage type,
// conversions and element traits.  gfx950 only.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef uint16_t bf16_t;  // raw bfloat16 storage

__device__ __forceinline__ float bf2f(uint32_t b) { return __uint_as_float(b << 16); }

// float -> bfloat16, round to nearest even (NaN kept quiet).
__device__ __forceinline__ uint32_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0u;
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

// Element traits: load as float, store from float (rounded for bf16).
template <typename T> struct Elt;
template <> struct Elt<float> {
  static __device__ __forceinline__ float ld(const float* p) { return *p; }
  static __device__ __forceinline__ void st(float* p, float v) { *p = v; }
};
template <> struct Elt<bf16_t> {
  static __device__ __forceinline__ float ld(const bf16_t* p) { return bf2f(*p); }
  static __device__ __forceinline__ void st(bf16_t* p, float v) { *p = (bf16_t)f2bf(v); }
};

__host__ __device__ __forceinline__ int cdiv(long a, long b) { return (int)((a + b - 1) / b); }

// Element k (wave-uniform, 0 <= k < N) of a kernel-argument array, read at
// constant indices so that the array stays in the argument segment rather
// than being copied to private memory for a dynamic index.
template <typename T, int N>
__device__ __forceinline__ T pickg(const T (&a)[N], int k) {
  T r = a[0];
#pragma unroll
  for (int i = 1; i < N; ++i) r = k == i ? a[i] : r;
  return r;
}
