// Page migration between two pools on one GPU (MI355X, gfx950): the copy
// that carries out a repack plan. One workgroup per (source, destination)
// page pair streams the page with 16-byte non-temporal loads and stores
// (pages are touched once), four in flight per lane; pages whose size is
// not a multiple of 16 bytes (fp8 scale rows) are copied in 4-byte words.
// The copy reads and writes each page once, so it is bound by HBM
// bandwidth.

#include <hip/hip_runtime.h>

#include <cstdint>

#include "laminar_repack.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__global__ void __launch_bounds__(256)
migrate_kernel16(const u32x4* __restrict__ src, int64_t src_pages,
                 u32x4* __restrict__ dst, int64_t dst_pages, int64_t page16,
                 const int2* __restrict__ pairs) {
  const int2 pr = pairs[blockIdx.x];
  if (pr.x < 0 || pr.x >= src_pages || pr.y < 0 || pr.y >= dst_pages) return;
  const u32x4* s = src + int64_t(pr.x) * page16;
  u32x4* d = dst + int64_t(pr.y) * page16;
  int64_t i = threadIdx.x;
  for (; i + 3 * 256 < page16; i += 4 * 256) {
    u32x4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = __builtin_nontemporal_load(&s[i + u * 256]);
#pragma unroll
    for (int u = 0; u < 4; ++u) __builtin_nontemporal_store(v[u], &d[i + u * 256]);
  }
  for (; i < page16; i += 256) d[i] = s[i];
}

__global__ void __launch_bounds__(256)
migrate_kernel4(const uint32_t* __restrict__ src, int64_t src_pages,
                uint32_t* __restrict__ dst, int64_t dst_pages, int64_t page4,
                const int2* __restrict__ pairs) {
  const int2 pr = pairs[blockIdx.x];
  if (pr.x < 0 || pr.x >= src_pages || pr.y < 0 || pr.y >= dst_pages) return;
  for (int64_t i = threadIdx.x; i < page4; i += 256)
    dst[int64_t(pr.y) * page4 + i] = src[int64_t(pr.x) * page4 + i];
}

}  // namespace

extern "C" laminar_status laminar_migrate_pages(const void* src_pool,
                                                int64_t src_pages,
                                                void* dst_pool, int64_t dst_pages,
                                                size_t page_bytes,
                                                const int32_t* pairs,
                                                int32_t num_pairs,
                                                hipStream_t stream) {
  if (num_pairs < 0 || src_pages < 0 || dst_pages < 0 || page_bytes == 0 ||
      (page_bytes & 3))
    return LAMINAR_ERR_INVALID_ARG;
  if (num_pairs == 0) return LAMINAR_OK;
  if (!src_pool || !dst_pool || !pairs) return LAMINAR_ERR_INVALID_ARG;
  const uintptr_t align = reinterpret_cast<uintptr_t>(src_pool) |
                          reinterpret_cast<uintptr_t>(dst_pool);
  if (reinterpret_cast<uintptr_t>(pairs) & 7) return LAMINAR_ERR_INVALID_ARG;
  if (page_bytes % 16 == 0) {
    if (align & 15) return LAMINAR_ERR_INVALID_ARG;
    hipLaunchKernelGGL(migrate_kernel16, dim3(num_pairs), dim3(256), 0, stream,
                       static_cast<const u32x4*>(src_pool), src_pages,
                       static_cast<u32x4*>(dst_pool), dst_pages,
                       int64_t(page_bytes / 16),
                       reinterpret_cast<const int2*>(pairs));
  } else {
    if (align & 3) return LAMINAR_ERR_INVALID_ARG;
    hipLaunchKernelGGL(migrate_kernel4, dim3(num_pairs), dim3(256), 0, stream,
                       static_cast<const uint32_t*>(src_pool), src_pages,
                       static_cast<uint32_t*>(dst_pool), dst_pages,
                       int64_t(page_bytes / 4),
                       reinterpret_cast<const int2*>(pairs));
  }
  return hipGetLastError() == hipSuccess ? LAMINAR_OK : LAMINAR_ERR_HIP;
}
