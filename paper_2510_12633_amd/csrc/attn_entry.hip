// C-ABI entry points of the decode-attention library: argument checks,
// the upload of a plan's tables into its workspace, and the calls that
// enqueue the kernels of decode_attn.hip.

#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstring>
#include <mutex>

#include "attn_internal.h"
#include "laminar_decode_attn.h"
#include "plan_internal.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

laminar_status check_bound(const laminar_plan* p) {
  if (!p) return LAMINAR_ERR_INVALID_ARG;
  if (p->ws_bytes > 0 && (!p->ws || p->ws_size < p->ws_bytes))
    return LAMINAR_ERR_WORKSPACE;
  return LAMINAR_OK;
}

bool aligned(const void* ptr, uintptr_t bytes) {
  return ptr && (reinterpret_cast<uintptr_t>(ptr) & (bytes - 1)) == 0;
}

// Pointers of a call: present, and aligned as the kernels access them (q
// rows, K/V tiles and out rows move in 16-byte vectors; the block table,
// lengths and lse in 4-byte words).
bool inputs_ok(const laminar_plan* p, const void* q, const void* k_pages,
               const void* v_pages, const int32_t* block_table,
               const int32_t* seq_lens, const float* out, const float* lse) {
  if (p->desc.batch == 0) return true;
  return aligned(q, 16) && aligned(k_pages, 16) && aligned(v_pages, 16) &&
         aligned(block_table, 4) && aligned(seq_lens, 4) &&
         aligned(out, 16) && aligned(lse, 4);
}

bool outputs_ok(const laminar_plan* p, const float* out, const float* lse) {
  return p->desc.batch == 0 || (aligned(out, 16) && aligned(lse, 4));
}

// Pinned staging for plan uploads. The tables are copied into one of a few
// pinned, device-mapped host slots, and a small kernel on the caller's
// stream copies them into the workspace. Compared with a DMA copy this keeps
// the upload on the same hardware queue as the attention kernels (no
// cross-engine hand-offs around it), blocks the host only when the oldest of
// eight uploads has not yet run (the host is then eight steps ahead), and
// lets the caller free the plan as soon as bind returns. One ring per
// device, created on first use and kept for the life of the process; a slot
// is reused only after the event recorded behind its last upload completed.
// Copies n16 16-byte words from device-mapped pinned host memory.
__global__ void __launch_bounds__(256)
upload_kernel(u32x4* __restrict__ dst, const u32x4* __restrict__ src,
              size_t n16) {
  const size_t stride = size_t(gridDim.x) * blockDim.x;
  for (size_t i = size_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n16;
       i += stride)
    dst[i] = src[i];
}

struct StagingRing {
  static constexpr int kSlots = 8;
  static constexpr size_t kSlotBytes = size_t(1) << 20;
  char* host = nullptr;
  char* dev_view = nullptr;    // device address of `host`
  hipEvent_t done[kSlots] = {};
  bool pending[kSlots] = {};
  int next = 0;
};

constexpr int kMaxDevices = 64;
std::mutex g_ring_mutex;
StagingRing g_rings[kMaxDevices];

laminar_status upload_tables(void* dst, const void* src, size_t bytes,
                             hipStream_t stream) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return LAMINAR_ERR_HIP;
  if (bytes > StagingRing::kSlotBytes || dev < 0 || dev >= kMaxDevices) {
    // Too large for a slot: copy straight from the plan and wait for it, so
    // the plan can still be freed when bind returns.
    hipError_t e = hipMemcpyAsync(dst, src, bytes, hipMemcpyHostToDevice, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    return e == hipSuccess ? LAMINAR_OK : LAMINAR_ERR_HIP;
  }
  std::lock_guard<std::mutex> lock(g_ring_mutex);
  StagingRing& ring = g_rings[dev];
  if (!ring.host) {
    void* h = nullptr;
    void* hd = nullptr;
    if (hipHostMalloc(&h, StagingRing::kSlots * StagingRing::kSlotBytes,
                      hipHostMallocMapped | hipHostMallocPortable) !=
            hipSuccess ||
        hipHostGetDevicePointer(&hd, h, 0) != hipSuccess)
      return LAMINAR_ERR_HIP;
    ring.dev_view = static_cast<char*>(hd);
    for (int i = 0; i < StagingRing::kSlots; ++i)
      if (hipEventCreateWithFlags(&ring.done[i], hipEventDisableTiming) !=
          hipSuccess)
        return LAMINAR_ERR_HIP;
    ring.host = static_cast<char*>(h);
  }
  const int slot = ring.next;
  ring.next = (slot + 1) % StagingRing::kSlots;
  if (ring.pending[slot] && hipEventSynchronize(ring.done[slot]) != hipSuccess)
    return LAMINAR_ERR_HIP;
  char* stage = ring.host + size_t(slot) * StagingRing::kSlotBytes;
  std::memcpy(stage, src, bytes);
  const size_t n16 = (bytes + 15) / 16;    // tables are 256-byte multiples
  const unsigned blocks = unsigned(n16 < 64 * 256 ? (n16 + 255) / 256 : 64);
  hipLaunchKernelGGL(upload_kernel, dim3(blocks), dim3(256), 0, stream,
                     static_cast<u32x4*>(dst),
                     reinterpret_cast<const u32x4*>(
                         ring.dev_view + size_t(slot) * StagingRing::kSlotBytes),
                     n16);
  if (hipGetLastError() != hipSuccess ||
      hipEventRecord(ring.done[slot], stream) != hipSuccess)
    return LAMINAR_ERR_HIP;
  ring.pending[slot] = true;
  return LAMINAR_OK;
}

laminar_detail::AttnCall make_call(const laminar_plan* p, const void* q,
                                   const void* k_pages, const void* v_pages,
                                   const int32_t* block_table,
                                   const int32_t* seq_lens, float* out,
                                   float* lse) {
  return laminar_detail::AttnCall{q, k_pages, v_pages, block_table, seq_lens,
                                  out, lse, p->ws};
}

// The library's own workspace for laminar_decode_attn_static: one
// LAMINAR_STATIC_WORKSPACE_BYTES array per GPU, held until the process
// ends. `scratch` names a host-side stand-in in host code; kernels get the
// device address that hipGetSymbolAddress returns for the current device.
__device__ __align__(256) unsigned char scratch[LAMINAR_STATIC_WORKSPACE_BYTES];

std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on the current device, looked up once per
// device; nullptr on failure.
void* scratch_on_current_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
    return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr)
      return nullptr;
    g_scratch_ptr[dev] = ptr;
  }
  return g_scratch_ptr[dev];
}

}  // namespace

extern "C" {

laminar_status laminar_plan_bind_workspace(laminar_plan* plan, void* workspace,
                                           size_t bytes, hipStream_t stream) {
  if (!plan) return LAMINAR_ERR_INVALID_ARG;
  if (plan->ws_bytes == 0) {
    plan->ws = workspace;
    plan->ws_size = bytes;
    return LAMINAR_OK;
  }
  if (!workspace || bytes < plan->ws_bytes ||
      (reinterpret_cast<uintptr_t>(workspace) & 255) != 0)
    return LAMINAR_ERR_WORKSPACE;
  plan->ws = workspace;
  plan->ws_size = bytes;
  const size_t table_bytes = plan->tables.size() * sizeof(int32_t);
  if (table_bytes == 0) return LAMINAR_OK;
  return upload_tables(workspace, plan->tables.data(), table_bytes, stream);
}

laminar_status laminar_decode_attn_partial(const laminar_plan* plan,
                                           const void* q, const void* k_pages,
                                           const void* v_pages,
                                           const int32_t* block_table,
                                           const int32_t* seq_lens, float* out,
                                           float* lse, hipStream_t stream) {
  if (!plan) return LAMINAR_ERR_INVALID_ARG;
  if (!inputs_ok(plan, q, k_pages, v_pages, block_table, seq_lens, out, lse))
    return LAMINAR_ERR_INVALID_ARG;
  laminar_status st = check_bound(plan);
  if (st != LAMINAR_OK) return st;
  return laminar_detail::enqueue_partial(
      *plan, make_call(plan, q, k_pages, v_pages, block_table, seq_lens, out,
                       lse), stream);
}

laminar_status laminar_decode_attn_merge(const laminar_plan* plan, float* out,
                                         float* lse, hipStream_t stream) {
  if (!plan) return LAMINAR_ERR_INVALID_ARG;
  if (!outputs_ok(plan, out, lse)) return LAMINAR_ERR_INVALID_ARG;
  laminar_status st = check_bound(plan);
  if (st != LAMINAR_OK) return st;
  return laminar_detail::enqueue_merge(
      *plan, make_call(plan, nullptr, nullptr, nullptr, nullptr, nullptr, out,
                       lse), stream);
}

laminar_status laminar_decode_attn(const laminar_plan* plan, const void* q,
                                   const void* k_pages, const void* v_pages,
                                   const int32_t* block_table,
                                   const int32_t* seq_lens, float* out,
                                   float* lse, hipStream_t stream) {
  if (!plan) return LAMINAR_ERR_INVALID_ARG;
  if (!inputs_ok(plan, q, k_pages, v_pages, block_table, seq_lens, out, lse))
    return LAMINAR_ERR_INVALID_ARG;
  laminar_status st = check_bound(plan);
  if (st != LAMINAR_OK) return st;
  const laminar_detail::AttnCall c =
      make_call(plan, q, k_pages, v_pages, block_table, seq_lens, out, lse);
  st = laminar_detail::enqueue_partial(*plan, c, stream);
  if (st != LAMINAR_OK) return st;
  return laminar_detail::enqueue_merge(*plan, c, stream);
}

laminar_status laminar_decode_attn_static(const laminar_plan* plan,
                                          const void* q, const void* k_pages,
                                          const void* v_pages,
                                          const int32_t* block_table,
                                          const int32_t* seq_lens, float* out,
                                          float* lse, hipStream_t stream) {
  if (!plan) return LAMINAR_ERR_INVALID_ARG;
  if (!inputs_ok(plan, q, k_pages, v_pages, block_table, seq_lens, out, lse))
    return LAMINAR_ERR_INVALID_ARG;
  if (plan->ws_bytes > LAMINAR_STATIC_WORKSPACE_BYTES)
    return LAMINAR_ERR_WORKSPACE;
  if (plan->num_items == 0) return LAMINAR_OK;
  void* ws = scratch_on_current_device();
  if (!ws) return LAMINAR_ERR_HIP;
  // The plan's tables (work list, merge and cascade records, and the zero
  // tail counter) go into the front of the workspace in stream order.
  const size_t table_bytes = plan->tables.size() * sizeof(int32_t);
  if (table_bytes > 0 &&
      hipMemcpyAsync(ws, plan->tables.data(), table_bytes,
                     hipMemcpyHostToDevice, stream) != hipSuccess)
    return LAMINAR_ERR_HIP;
  laminar_detail::AttnCall c =
      make_call(plan, q, k_pages, v_pages, block_table, seq_lens, out, lse);
  c.ws = ws;
  laminar_status st = laminar_detail::enqueue_partial(*plan, c, stream);
  if (st != LAMINAR_OK) return st;
  return laminar_detail::enqueue_merge(*plan, c, stream);
}

}  // extern "C"
