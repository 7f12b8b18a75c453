// Element-wise arithmetic shared by the decode-step kernels and the
// projection kernel's fused inputs, so that a fused input rounds exactly as
// the separate kernel it replaces.
#ifndef LAMINAR_ACTIVATION_H
#define LAMINAR_ACTIVATION_H

#include <hip/hip_runtime.h>

#include <cstdint>

namespace laminar {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// SwiGLU of one element in fp32: silu(g) * u with silu(g) = g / (1 + e^-g),
// e^-g as 2^(-g log2 e) on the hardware exponential and the division as a
// hardware reciprocal: a few ulp of fp32 (far below the bf16 rounding that
// follows) in 5 instructions, which matters where every tile of a
// projection recomputes its input. Large |g| behaves: e^-g overflows to
// infinity and the reciprocal to 0 for g << 0, and e^-g is 0 for g >> 0.
__device__ __forceinline__ float silu_mul(float g, float u) {
  const float e = __builtin_amdgcn_exp2f(g * -1.44269504088896341f);
  return g * __builtin_amdgcn_rcpf(1.0f + e) * u;
}

// Eight outputs of SwiGLU, rounded once to bf16 (nearest even).
__device__ __forceinline__ bf16x8_t silu_mul8(bf16x8_t g, bf16x8_t u) {
  bf16x8_t o;
#pragma unroll
  for (int e = 0; e < 8; ++e) o[e] = (__bf16)silu_mul(float(g[e]), float(u[e]));
  return o;
}

// Eight fp32 values rounded to bf16 (nearest even).
__device__ __forceinline__ bf16x8_t round8(f32x4_t lo, f32x4_t hi) {
  bf16x8_t o;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    o[e] = (__bf16)lo[e];
    o[4 + e] = (__bf16)hi[e];
  }
  return o;
}

// RMS norm pieces, shared by laminar_rmsnorm and the projection's fused
// norm so that both sum in the same order and round identically.
//
// Sum of squares of one 16-byte chunk added to a running fma chain.
__device__ __forceinline__ float sumsq8(bf16x8_t v, float ss) {
#pragma unroll
  for (int e = 0; e < 8; ++e) ss = fmaf(float(v[e]), float(v[e]), ss);
  return ss;
}

// Butterfly sum over a 64-lane wavefront: every lane ends with the same
// value (each stage adds the same two operands on both lanes).
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// 1 / sqrt(mean of squares + eps) from the sums of four 64-thread groups.
__device__ __forceinline__ float rms_inverse(float p0, float p1, float p2,
                                             float p3, float inv_n,
                                             float eps) {
  const float total = (p0 + p1) + (p2 + p3);
  return 1.0f / sqrtf(total * inv_n + eps);
}

// Eight normalised outputs: (x r) w, rounded once to bf16.
__device__ __forceinline__ bf16x8_t rms_scale8(bf16x8_t x, bf16x8_t w,
                                               float r) {
  bf16x8_t o;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float s = float(x[e]) * r;
    o[e] = (__bf16)(s * float(w[e]));
  }
  return o;
}

}  // namespace laminar

#endif  // LAMINAR_ACTIVATION_H
