// Element-wise operations of a decode step on MI355X (gfx950): the RMS
// pre-norm and the SwiGLU activation, one fused kernel each. Both are a few
// kilobytes per token, so what matters at decode batch sizes is one launch
// instead of the five or six that the unfused operations take.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "activation.h"
#include "laminar_decode_step.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

// One workgroup per row: thread t sums the squares of chunks t, t + 256,
// ... in one fma chain, each wavefront adds its 64 chains by a butterfly,
// and the four wavefront sums are added as (w0 + w1) + (w2 + w3); then a
// second pass (served by L2) scales and rounds. The projection kernel's
// fused norm follows the same order.
__global__ void __launch_bounds__(256)
rmsnorm_kernel(const bf16x8* __restrict__ x, const bf16x8* __restrict__ w,
               bf16x8* __restrict__ y, int chunks, float inv_n, float eps) {
  __shared__ float part[4];
  const bf16x8* xr = x + size_t(blockIdx.x) * chunks;
  bf16x8* yr = y + size_t(blockIdx.x) * chunks;
  // rows of up to 4 x 256 chunks (8192 values) stay in registers from the
  // sum of squares to the scaling, and their weights are loaded with them:
  // one trip to memory before the workgroup's reduction instead of two
  constexpr int kHeld = 4;
  bf16x8 xv[kHeld], wv[kHeld];
#pragma unroll
  for (int h = 0; h < kHeld; ++h) {
    const int c = threadIdx.x + 256 * h;
    if (c < chunks) {
      xv[h] = xr[c];
      if (w) wv[h] = w[c];
    }
  }
  float ss = 0.f;
#pragma unroll
  for (int h = 0; h < kHeld; ++h)
    if (threadIdx.x + 256 * h < chunks) ss = laminar::sumsq8(xv[h], ss);
  for (int c = threadIdx.x + 256 * kHeld; c < chunks; c += 256)
    ss = laminar::sumsq8(xr[c], ss);
  ss = laminar::wave_sum(ss);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float r =
      laminar::rms_inverse(part[0], part[1], part[2], part[3], inv_n, eps);
  auto scale = [&](const bf16x8& v, const bf16x8* wc) {
    if (wc) return laminar::rms_scale8(v, *wc, r);
    bf16x8 o;
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = (__bf16)(float(v[e]) * r);
    return o;
  };
#pragma unroll
  for (int h = 0; h < kHeld; ++h) {
    const int c = threadIdx.x + 256 * h;
    if (c < chunks) yr[c] = scale(xv[h], w ? &wv[h] : nullptr);
  }
  for (int c = threadIdx.x + 256 * kHeld; c < chunks; c += 256)
    yr[c] = scale(xr[c], w ? &w[c] : nullptr);
}

// Eight outputs per thread: y[m, i..i+7] from gate gu[m, i..] and up
// gu[m, I + i..].
__global__ void __launch_bounds__(256)
silu_mul_kernel(const bf16x8* __restrict__ gu, bf16x8* __restrict__ y,
                int rows, int chunks) {
  const size_t t = size_t(blockIdx.x) * 256 + threadIdx.x;
  if (t >= size_t(rows) * chunks) return;
  const size_t m = t / chunks, c = t - m * chunks;
  const bf16x8 g = gu[m * 2 * chunks + c];
  const bf16x8 u = gu[m * 2 * chunks + chunks + c];
  y[t] = laminar::silu_mul8(g, u);
}

bool misaligned16(const void* p) {
  return reinterpret_cast<uintptr_t>(p) & 15;
}

}  // namespace

extern "C" {

laminar_status laminar_rmsnorm(const void* x, const void* weight, void* y,
                               int32_t m, int32_t n, float eps,
                               hipStream_t stream) {
  if (!x || !y || misaligned16(x) || misaligned16(y) || misaligned16(weight))
    return LAMINAR_ERR_INVALID_ARG;
  if (m < 1 || n < 8 || n % 8 || !(eps >= 0.f) || !std::isfinite(eps))
    return LAMINAR_ERR_INVALID_ARG;
  hipLaunchKernelGGL(rmsnorm_kernel, dim3(unsigned(m)), dim3(256), 0, stream,
                     static_cast<const bf16x8*>(x),
                     static_cast<const bf16x8*>(weight),
                     static_cast<bf16x8*>(y), n / 8, 1.0f / float(n), eps);
  return hipGetLastError() == hipSuccess ? LAMINAR_OK : LAMINAR_ERR_HIP;
}

laminar_status laminar_silu_mul(const void* gu, void* y, int32_t m,
                                int32_t inter, hipStream_t stream) {
  if (!gu || !y || misaligned16(gu) || misaligned16(y))
    return LAMINAR_ERR_INVALID_ARG;
  if (m < 1 || inter < 8 || inter % 8) return LAMINAR_ERR_INVALID_ARG;
  const size_t total = size_t(m) * (inter / 8);
  hipLaunchKernelGGL(silu_mul_kernel, dim3(unsigned((total + 255) / 256)),
                     dim3(256), 0, stream, static_cast<const bf16x8*>(gu),
                     static_cast<bf16x8*>(y), m, inter / 8);
  return hipGetLastError() == hipSuccess ? LAMINAR_OK : LAMINAR_ERR_HIP;
}

}  // extern "C"
