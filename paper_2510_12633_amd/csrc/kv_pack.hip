// Conversion of row-major KV pages into the attention kernels' tile order.
//
// A caller whose cache holds each (page, kv-head) tile as 16 token rows of
// head_dim elements (the usual paged layout) packs it once into the order
// the decode kernels read with 16-byte matrix-core operand loads:
//   K: token t, dim d at ((d / X) * 16 + t) * X + d % X   (X = 16 / bytes)
//   V: token t, dim d at ((t / 4) * head_dim + d) * 4 + t % 4
// It is a copy bound by HBM bandwidth: each workgroup stages 4 KiB of row-
// major tiles in LDS with 16-byte loads and writes the packed 16-byte
// chunks, gathering each chunk's elements from LDS.

#include <hip/hip_runtime.h>

#include <cstdint>

#include "laminar_decode_attn.h"
#include "laminar_kv_append.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kStageBytes = 4096;            // 256 threads x 16 bytes

// One pass moves TPW = 4096 / tile bytes whole tiles; workgroups stride
// over the passes.
template <int D, int EB, bool V>
__global__ void __launch_bounds__(256)
kv_pack_kernel(const u32x4* __restrict__ src, u32x4* __restrict__ dst,
               int64_t num_tiles) {
  constexpr int TB = 16 * D * EB;            // bytes per tile
  constexpr int CH = TB / 16;                // 16-byte chunks per tile
  constexpr int TPW = kStageBytes / TB;      // tiles per pass
  constexpr int X = 16 / EB;                 // elements per chunk
  __shared__ __align__(16) unsigned char stage[kStageBytes];
  const int tid = threadIdx.x;
  const int tl = tid / CH, c = tid % CH;     // tile of the pass, chunk
  const int64_t passes = (num_tiles + TPW - 1) / TPW;
  for (int64_t p = blockIdx.x; p < passes; p += gridDim.x) {
    const int64_t tile = p * TPW + tl;
    const bool ok = tile < num_tiles;
    if (ok)
      reinterpret_cast<u32x4*>(stage)[tid] = src[tile * CH + c];
    __syncthreads();
    if (ok) {
      const unsigned char* row = stage + tl * TB;   // [16][D] row-major
      u32x4 out;
      if constexpr (!V) {
        // chunk c holds dims (c / 16) * X .. + X - 1 of token c % 16: one
        // 16-byte run of the row-major tile
        out = *reinterpret_cast<const u32x4*>(
            row + ((c % 16) * D + (c / 16) * X) * EB);
      } else {
        // element e of chunk c sits at packed offset o = c * X + e: token
        // (o / (4 D)) * 4 + o % 4, dim (o / 4) % D
        unsigned char bytes[16];
#pragma unroll
        for (int e = 0; e < X; ++e) {
          const int o = c * X + e;
          const int t = (o / (4 * D)) * 4 + o % 4;
          const int d = (o / 4) % D;
#pragma unroll
          for (int k = 0; k < EB; ++k) bytes[e * EB + k] = row[(t * D + d) * EB + k];
        }
        out = *reinterpret_cast<const u32x4*>(bytes);
      }
      dst[tile * CH + c] = out;
    }
    __syncthreads();                          // the stage is reused
  }
}

template <int D, int EB>
void launch(const void* src, void* dst, int64_t num_tiles, bool v,
            hipStream_t stream) {
  constexpr int TPW = kStageBytes / (16 * D * EB);
  const int64_t passes = (num_tiles + TPW - 1) / TPW;
  const dim3 grid(unsigned(passes < 8192 ? passes : 8192));
  const u32x4* s = static_cast<const u32x4*>(src);
  u32x4* d = static_cast<u32x4*>(dst);
  if (v)
    hipLaunchKernelGGL((kv_pack_kernel<D, EB, true>), grid, dim3(256), 0,
                       stream, s, d, num_tiles);
  else
    hipLaunchKernelGGL((kv_pack_kernel<D, EB, false>), grid, dim3(256), 0,
                       stream, s, d, num_tiles);
}

}  // namespace

extern "C" {

laminar_status laminar_kv_pack(const void* src, void* dst, int64_t num_tiles,
                               int32_t head_dim, int32_t kv_dtype,
                               int32_t which, hipStream_t stream) {
  if (num_tiles < 0 || (which != 0 && which != 1) ||
      (kv_dtype != LAMINAR_KV_BF16 && kv_dtype != LAMINAR_KV_FP8_E4M3FN))
    return LAMINAR_ERR_INVALID_ARG;
  if (head_dim != 64 && head_dim != 128) return LAMINAR_ERR_UNSUPPORTED;
  if (num_tiles == 0) return LAMINAR_OK;
  const uintptr_t s = reinterpret_cast<uintptr_t>(src);
  const uintptr_t d = reinterpret_cast<uintptr_t>(dst);
  const int eb = kv_dtype == LAMINAR_KV_BF16 ? 2 : 1;
  const uint64_t bytes = uint64_t(num_tiles) * 16u * uint64_t(head_dim) * eb;
  if (!src || !dst || (s & 15) || (d & 15) || (s < d + bytes && d < s + bytes))
    return LAMINAR_ERR_INVALID_ARG;
  const bool v = which == 1;
  if (head_dim == 128)
    eb == 2 ? launch<128, 2>(src, dst, num_tiles, v, stream)
            : launch<128, 1>(src, dst, num_tiles, v, stream);
  else
    eb == 2 ? launch<64, 2>(src, dst, num_tiles, v, stream)
            : launch<64, 1>(src, dst, num_tiles, v, stream);
  return hipGetLastError() == hipSuccess ? LAMINAR_OK : LAMINAR_ERR_HIP;
}

}  // extern "C"
