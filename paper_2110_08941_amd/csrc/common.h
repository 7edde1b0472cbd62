// Internal helpers shared by the HIP kernels and the host code of libhs.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hs {

typedef uint16_t bf16_t;  // bf16 storage: the upper 16 bits of an IEEE fp32

// fp32 -> bf16, round to nearest even on the dropped 16 bits; NaN stays a
// quiet NaN.
__host__ __device__ inline bf16_t f2bf(float f) {
  uint32_t u;
  __builtin_memcpy(&u, &f, 4);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return (bf16_t)((u >> 16) | 0x40);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

__host__ __device__ inline float bf2f(bf16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  __builtin_memcpy(&f, &u, 4);
  return f;
}

// Element access for the two storage types of activations.
template <typename T> __device__ inline float ld(const T* p, int64_t i);
template <> __device__ inline float ld<float>(const float* p, int64_t i) { return p[i]; }
template <> __device__ inline float ld<bf16_t>(const bf16_t* p, int64_t i) { return bf2f(p[i]); }
template <typename T> __device__ inline void st(T* p, int64_t i, float v);
template <> __device__ inline void st<float>(float* p, int64_t i, float v) { p[i] = v; }
template <> __device__ inline void st<bf16_t>(bf16_t* p, int64_t i, float v) { p[i] = f2bf(v); }

// Unsigned division by a run-time constant d >= 1 with a precomputed
// multiplier (round-up method): q = (umulhi(n, mul) + n) >> shift for
// n < 2^31.
struct FastDiv {
  uint32_t d, mul, shift;
};

inline FastDiv make_fastdiv(uint32_t d) {
  FastDiv f;
  f.d = d;
  uint32_t s = 0;
  while ((1ull << s) < d) ++s;
  f.shift = s;
  // mul = floor(2^32 * (2^s - d) / d) + 1
  f.mul = (uint32_t)(((1ull << 32) * ((1ull << s) - d)) / d + 1);
  return f;
}

__device__ inline uint32_t fdiv(uint32_t n, const FastDiv& f) {
  uint32_t hi = __umulhi(n, f.mul);
  return (hi + n) >> f.shift;
}

// Geometry of one convolution (or of a linear layer: H = W = R = S = 1).
// Activations are NHWC, weights OHWI.
struct ConvGeom {
  int n, H, W, C;       // input
  int Ho, Wo, K;        // output (K = output channels)
  int R, S, stride, pad;
  FastDiv HWo, Wo_, HWi, Wi_, Cdiv, Kdiv, Sdiv;
};

inline int ceil_div(int64_t a, int64_t b) { return (int)((a + b - 1) / b); }

}  // namespace hs
