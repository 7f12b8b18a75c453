// HBM calibration kernels (measurement support, not part of attention):
// a sequential read, a copy, and a gather of random fixed-size tiles
// through an index list, the access pattern of paged KV reads. Each
// workgroup streams 64 KiB chunks with non-temporal 16-byte accesses, eight
// in flight per lane.

#include <hip/hip_runtime.h>

#include <cstdint>

#include "laminar_decode_attn.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

constexpr int kCalibChunk16 = 4096;          // 64 KiB per workgroup
constexpr int kReadSinkFloats = 1 << 16;     // workgroups per read pass

__global__ void __launch_bounds__(256)
hbm_read_kernel(const u32x4* __restrict__ src, size_t n16, float* sink) {
  uint32_t acc = 0;
  for (size_t blk = blockIdx.x; blk * kCalibChunk16 < n16; blk += gridDim.x) {
    const size_t beg = blk * kCalibChunk16;
    const size_t end = beg + kCalibChunk16 < n16 ? beg + kCalibChunk16 : n16;
    size_t i = beg + threadIdx.x;
    for (; i + 7 * 256 < end; i += 8 * 256) {
      u32x4 v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = __builtin_nontemporal_load(&src[i + u * 256]);
#pragma unroll
      for (int u = 0; u < 8; ++u) acc ^= v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
    }
    for (; i < end; i += 256) acc ^= src[i][0];
  }
  // Every lane's value feeds the workgroup sum, so no load is dead code.
  float s = wave_sum(__uint_as_float(acc & 0x007FFFFFu));
  __shared__ float red[4];
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) sink[blockIdx.x] = (red[0] + red[1]) + (red[2] + red[3]);
}

__global__ void __launch_bounds__(256)
hbm_copy_kernel(u32x4* __restrict__ dst, const u32x4* __restrict__ src,
                size_t n16) {
  for (size_t blk = blockIdx.x; blk * kCalibChunk16 < n16; blk += gridDim.x) {
    const size_t beg = blk * kCalibChunk16;
    const size_t end = beg + kCalibChunk16 < n16 ? beg + kCalibChunk16 : n16;
    size_t i = beg + threadIdx.x;
    for (; i + 7 * 256 < end; i += 8 * 256) {
      u32x4 v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = __builtin_nontemporal_load(&src[i + u * 256]);
#pragma unroll
      for (int u = 0; u < 8; ++u) __builtin_nontemporal_store(v[u], &dst[i + u * 256]);
    }
    for (; i < end; i += 256) dst[i] = src[i];
  }
}

// Random-tile gather calibration: the 16-byte chunks of the listed tiles
// (tile t of the list is tile idx[t] of src, tile16 chunks each, a power of
// two), streamed with non-temporal loads, eight in flight per lane, as the
// attention kernel streams its pages. Indices are clamped into the buffer,
// so a bad list cannot read out of bounds. Each workgroup writes the sum of
// the 32-bit words it read (mod 2^32) into sink[blockIdx.x].
__global__ void __launch_bounds__(256)
hbm_gather_kernel(const u32x4* __restrict__ src, uint32_t num_tiles,
                  const int32_t* __restrict__ idx, int log2_tile16,
                  size_t n16, uint32_t* sink) {
  const size_t mask = (size_t(1) << log2_tile16) - 1;
  uint32_t acc = 0;
  for (size_t blk = blockIdx.x; blk * kCalibChunk16 < n16; blk += gridDim.x) {
    const size_t beg = blk * kCalibChunk16;
    const size_t end = beg + kCalibChunk16 < n16 ? beg + kCalibChunk16 : n16;
    size_t i = beg + threadIdx.x;
    for (; i + 7 * 256 < end; i += 8 * 256) {
      u32x4 v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const size_t c = i + u * 256;
        const uint32_t t = min(uint32_t(idx[c >> log2_tile16]), num_tiles - 1);
        v[u] = __builtin_nontemporal_load(
            &src[(size_t(t) << log2_tile16) + (c & mask)]);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) acc += (v[u][0] + v[u][1]) + (v[u][2] + v[u][3]);
    }
    for (; i < end; i += 256) {
      const uint32_t t = min(uint32_t(idx[i >> log2_tile16]), num_tiles - 1);
      const u32x4 v = src[(size_t(t) << log2_tile16) + (i & mask)];
      acc += (v[0] + v[1]) + (v[2] + v[3]);
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) acc += __shfl_xor(acc, o);
  __shared__ uint32_t red[4];
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) sink[blockIdx.x] = (red[0] + red[1]) + (red[2] + red[3]);
}

unsigned calib_grid(size_t n16) {
  const size_t chunks = (n16 + kCalibChunk16 - 1) / kCalibChunk16;
  return unsigned(chunks < size_t(kReadSinkFloats) ? (chunks ? chunks : 1)
                                                   : size_t(kReadSinkFloats));
}

}  // namespace

extern "C" {

int32_t laminar_hbm_read_sink_floats(void) { return kReadSinkFloats; }

laminar_status laminar_hbm_read(const void* src, size_t bytes, float* sink,
                                hipStream_t stream) {
  if (!src || !sink || (bytes & 15) ||
      (reinterpret_cast<uintptr_t>(src) & 15))
    return LAMINAR_ERR_INVALID_ARG;
  hipLaunchKernelGGL(hbm_read_kernel, dim3(calib_grid(bytes / 16)), dim3(256),
                     0, stream, static_cast<const u32x4*>(src), bytes / 16,
                     sink);
  return hipGetLastError() == hipSuccess ? LAMINAR_OK : LAMINAR_ERR_HIP;
}

int32_t laminar_hbm_gather_sink_words(int64_t n_idx, size_t tile_bytes) {
  if (n_idx <= 0 || tile_bytes < 16) return 0;
  return int32_t(calib_grid(size_t(n_idx) * (tile_bytes / 16)));
}

laminar_status laminar_hbm_gather(const void* src, size_t src_bytes,
                                  size_t tile_bytes, const int32_t* idx,
                                  int64_t n_idx, uint32_t* sink,
                                  hipStream_t stream) {
  if (!src || (reinterpret_cast<uintptr_t>(src) & 15) || tile_bytes < 16 ||
      (tile_bytes & (tile_bytes - 1)) || n_idx < 0 ||
      src_bytes < tile_bytes || src_bytes / tile_bytes > 0xFFFFFFFFull)
    return LAMINAR_ERR_INVALID_ARG;
  if (n_idx == 0) return LAMINAR_OK;
  if (!idx || !sink || (reinterpret_cast<uintptr_t>(idx) & 3) ||
      (reinterpret_cast<uintptr_t>(sink) & 3))
    return LAMINAR_ERR_INVALID_ARG;
  int log2_tile16 = 0;
  while ((size_t(16) << log2_tile16) < tile_bytes) ++log2_tile16;
  const size_t n16 = size_t(n_idx) << log2_tile16;
  hipLaunchKernelGGL(hbm_gather_kernel, dim3(calib_grid(n16)), dim3(256), 0,
                     stream, static_cast<const u32x4*>(src),
                     uint32_t(src_bytes / tile_bytes), idx, log2_tile16, n16,
                     sink);
  return hipGetLastError() == hipSuccess ? LAMINAR_OK : LAMINAR_ERR_HIP;
}

laminar_status laminar_hbm_copy(void* dst, const void* src, size_t bytes,
                                hipStream_t stream) {
  if (!src || !dst || (bytes & 15) ||
      (reinterpret_cast<uintptr_t>(src) & 15) ||
      (reinterpret_cast<uintptr_t>(dst) & 15))
    return LAMINAR_ERR_INVALID_ARG;
  if (bytes == 0) return LAMINAR_OK;
  hipLaunchKernelGGL(hbm_copy_kernel, dim3(calib_grid(bytes / 16)), dim3(256),
                     0, stream, static_cast<u32x4*>(dst),
                     static_cast<const u32x4*>(src), bytes / 16);
  return hipGetLastError() == hipSuccess ? LAMINAR_OK : LAMINAR_ERR_HIP;
}

}  // extern "C"
