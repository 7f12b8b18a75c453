// Skinny projection product y = x w^T for decode batches (M <= 64) on
// MI355X (gfx950).
//
// At decode batch sizes the product streams the whole weight matrix w
// [N, K] for a few rows of x, so it is bound by HBM bandwidth. Each
// wavefront owns 16 rows of w (16 output features) over a range of K and
// runs v_mfma_f32_16x16x32_bf16 with the weights as the A operand and the
// batch (padded to 16 per tile) as B, so each weight byte is read once and
// used for all M rows. Within a step of 128 k values, matrix-core step j
// takes k = 32j .. 32j+31, lane group q holding k = 32j + 8q .. +7 of its
// row: each load instruction reads 64 contiguous bytes of each of 16 rows.
// Loads run NB steps ahead of the step being computed (plain loads:
// measured 10-25% faster here than non-temporal ones). When
// N alone gives too few wavefronts to keep HBM busy, K is split and a
// second kernel adds the partial sums in a fixed order.

#include <hip/hip_runtime.h>

#include <cstdint>

#include "laminar_linear.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kStepK = 128;          // k values per pipeline step
constexpr int kMaxM = 64;
constexpr int kTargetWaves = 2048;   // 2 per SIMD: ~16 MB of weights in flight

struct LinearArgs {
  const uint16_t* x;     // [M, K]
  const uint16_t* w;     // [N, K]
  float* y;              // [M, N]
  float* part;           // [splits, M, N] when split
  int32_t m, n, k;
  int32_t n_tiles, splits, steps_per_split;
};

template <int MT>
struct StepRegs {
  u32x4 w[4];
  u32x4 x[MT][4];
};

template <int MT>
__device__ __forceinline__ void load_step(const LinearArgs& a, int row_n,
                                          int kb, int q, int r16,
                                          StepRegs<MT>& s) {
  // load j of lane group q: k = kb + 32 j + 8 q .. +7, so each load
  // instruction reads 64 contiguous bytes of each of the 16 rows
  const u32x4* wp = reinterpret_cast<const u32x4*>(
      a.w + size_t(row_n) * a.k + kb + 8 * q);
#pragma unroll
  for (int j = 0; j < 4; ++j) s.w[j] = wp[4 * j];
#pragma unroll
  for (int t = 0; t < MT; ++t) {
    const int m = 16 * t + r16;
    const bool ok = m < a.m;
    const u32x4* xp = reinterpret_cast<const u32x4*>(
        a.x + size_t(ok ? m : 0) * a.k + kb + 8 * q);
#pragma unroll
    for (int j = 0; j < 4; ++j) s.x[t][j] = ok ? xp[4 * j] : u32x4{0, 0, 0, 0};
  }
}

template <int MT>
__device__ __forceinline__ void mma_step(const StepRegs<MT>& s,
                                         f32x4 (&acc)[MT]) {
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const bf16x8 av = __builtin_bit_cast(bf16x8, s.w[j]);
#pragma unroll
    for (int t = 0; t < MT; ++t)
      acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
          av, __builtin_bit_cast(bf16x8, s.x[t][j]), acc[t], 0, 0, 0);
  }
}

template <int MT>
__global__ void __launch_bounds__(256) linear_kernel(const LinearArgs a) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int gw = blockIdx.x * 4 + wave;                // global wavefront
  if (gw >= a.n_tiles * a.splits) return;
  const int tile = gw % a.n_tiles, split = gw / a.n_tiles;
  const int r16 = lane & 15, q = lane >> 4;
  const int n0 = tile * 16;
  const int total_steps = a.k / kStepK;
  const int s0 = split * a.steps_per_split;
  const int s1 = min(total_steps, s0 + a.steps_per_split);

  f32x4 acc[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};

  // NB steps in flight: a ring of register buffers, refilled NB steps
  // ahead of the step being computed
  constexpr int NB = MT == 1 ? 4 : 2;
  StepRegs<MT> buf[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i)
    if (s0 + i < s1) load_step<MT>(a, n0 + r16, (s0 + i) * kStepK, q, r16, buf[i]);
  for (int st = s0; st < s1; st += NB) {
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      if (st + i < s1) {
        mma_step<MT>(buf[i], acc);
        if (st + i + NB < s1)
          load_step<MT>(a, n0 + r16, (st + i + NB) * kStepK, q, r16, buf[i]);
      }
    }
  }

  // lane (group q, column r16) holds D[n0 + 4q + r][m = 16t + r16]
  float* dst = a.splits > 1 ? a.part + size_t(split) * a.m * a.n : a.y;
#pragma unroll
  for (int t = 0; t < MT; ++t) {
    const int m = 16 * t + r16;
    if (m < a.m)
      *reinterpret_cast<f32x4*>(dst + size_t(m) * a.n + n0 + 4 * q) = acc[t];
  }
}

// y[m, n] = sum over splits s (in order) of part[s, m, n]; four n per thread.
__global__ void __launch_bounds__(256) linear_reduce(const LinearArgs a) {
  const size_t i = size_t(blockIdx.x) * 256 + threadIdx.x;    // float4 index
  const size_t total = size_t(a.m) * a.n / 4;
  if (i >= total) return;
  const f32x4* p = reinterpret_cast<const f32x4*>(a.part);
  f32x4 s = p[i];
  for (int k = 1; k < a.splits; ++k) s += p[size_t(k) * total + i];
  reinterpret_cast<f32x4*>(a.y)[i] = s;
}

bool shape_ok(int32_t m, int32_t n, int32_t k) {
  return m >= 1 && m <= kMaxM && n >= 16 && n % 16 == 0 && k >= kStepK &&
         k % kStepK == 0;
}

void split_plan(int32_t n, int32_t k, int32_t* splits, int32_t* per) {
  const int32_t tiles = n / 16, steps = k / kStepK;
  int32_t want = (kTargetWaves + tiles - 1) / tiles;
  if (want < 1) want = 1;
  if (want > steps) want = steps;
  *per = (steps + want - 1) / want;
  *splits = (steps + *per - 1) / *per;
}

}  // namespace

extern "C" {

int32_t laminar_linear_splits(int32_t m, int32_t n, int32_t k) {
  if (!shape_ok(m, n, k)) return 0;
  int32_t s, per;
  split_plan(n, k, &s, &per);
  return s;
}

size_t laminar_linear_workspace_bytes(int32_t m, int32_t n, int32_t k) {
  const int32_t s = laminar_linear_splits(m, n, k);
  return s > 1 ? (size_t(s) * m * n * sizeof(float) + 255) & ~size_t(255) : 0;
}

laminar_status laminar_linear(const void* x, const void* w, float* y,
                              int32_t m, int32_t n, int32_t k, void* workspace,
                              size_t workspace_bytes, hipStream_t stream) {
  if (!x || !w || !y) return LAMINAR_ERR_INVALID_ARG;
  if ((reinterpret_cast<uintptr_t>(x) | reinterpret_cast<uintptr_t>(w) |
       reinterpret_cast<uintptr_t>(y)) & 15)
    return LAMINAR_ERR_INVALID_ARG;
  if (!shape_ok(m, n, k)) return LAMINAR_ERR_UNSUPPORTED;
  LinearArgs a;
  a.x = static_cast<const uint16_t*>(x);
  a.w = static_cast<const uint16_t*>(w);
  a.y = y;
  a.m = m;
  a.n = n;
  a.k = k;
  a.n_tiles = n / 16;
  split_plan(n, k, &a.splits, &a.steps_per_split);
  a.part = nullptr;
  if (a.splits > 1) {
    const size_t need = laminar_linear_workspace_bytes(m, n, k);
    if (!workspace || workspace_bytes < need ||
        (reinterpret_cast<uintptr_t>(workspace) & 255))
      return LAMINAR_ERR_INVALID_ARG;
    a.part = static_cast<float*>(workspace);
  }
  const int waves = a.n_tiles * a.splits;
  const dim3 grid((waves + 3) / 4);
  const int mt = (m + 15) / 16;
  switch (mt) {
    case 1: hipLaunchKernelGGL(linear_kernel<1>, grid, dim3(256), 0, stream, a); break;
    case 2: hipLaunchKernelGGL(linear_kernel<2>, grid, dim3(256), 0, stream, a); break;
    case 3: hipLaunchKernelGGL(linear_kernel<3>, grid, dim3(256), 0, stream, a); break;
    default: hipLaunchKernelGGL(linear_kernel<4>, grid, dim3(256), 0, stream, a); break;
  }
  if (hipGetLastError() != hipSuccess) return LAMINAR_ERR_HIP;
  if (a.splits > 1) {
    const size_t total = size_t(m) * n / 4;
    hipLaunchKernelGGL(linear_reduce, dim3(unsigned((total + 255) / 256)),
                       dim3(256), 0, stream, a);
    if (hipGetLastError() != hipSuccess) return LAMINAR_ERR_HIP;
  }
  return LAMINAR_OK;
}

}  // extern "C"
