// Internal definition of the host-side plan shared by the planner and the
// HIP entry points. Not part of the public C ABI.
#pragma once

#include <cstddef>
#include <cstdint>
#include <vector>

#include "laminar_decode_attn.h"

struct laminar_plan {
  laminar_attn_desc desc;
  int32_t group = 0;           // query heads per kv-head
  int32_t pages_per_item = 0;  // chosen split size
  int32_t waves = 0;           // wavefronts per work item
  int32_t num_items = 0;
  int32_t num_merges = 0;
  int32_t num_slots = 0;       // partial (out, lse) records
  // Items [num_main, num_items) are the dynamic tail: workgroups with those
  // indices take the next of them from a counter at off_tail instead.
  int32_t num_main = 0;
  int32_t num_cascade_units = 0;  // (shared-prefix chunk, kv-head) units
  int32_t num_cascade_members = 0;  // member records over all those units
  // Host image of workspace bytes [0, off_lse): the work items (4 int32
  // each, in launch order) at off_items, the merge records at off_merges,
  // the cascade unit headers (4 int32: longest member, member count, first
  // member record, kv-head) at off_cunits and the cascade member records
  // (2 int32: trajectory, first partial slot) at off_cmembers, and the
  // dynamic-tail counter (0) at off_tail.
  std::vector<int32_t> tables;
  // Workspace layout (byte offsets, 256-byte aligned sections).
  size_t off_items = 0, off_merges = 0, off_cunits = 0, off_cmembers = 0;
  size_t off_tail = 0;         // int32 tail counter, 0 between launches
  size_t off_lse = 0, off_o = 0;
  size_t ws_bytes = 0;
  // Bound workspace (device memory owned by the caller).
  void* ws = nullptr;
  size_t ws_size = 0;
};

namespace laminar_detail {
// Wavefronts resident per CU that the automatic split assumes for one item
// of one wavefront (two per SIMD with ~200 VGPRs per lane).
constexpr int kResidentWavesPerCU = 8;
// Work items per resident slot the automatic split aims for, as a ratio
// kItemsPerSlotNum / kItemsPerSlotDen. Each item costs about one chain of
// dependent memory latencies to start, so fewer, larger items are faster
// until the longest-first order can no longer even out the tail; 1.5 was
// the measured sweet spot on the 7B and post-repack workloads.
constexpr int kItemsPerSlotNum = 3;
constexpr int kItemsPerSlotDen = 2;
// Items per resident slot for batches that mix short units (dynamic tail)
// with long ones cut in halves: 2 measured at or near the best next to 1.5,
// 2.5 and 3 on the 7B and 32B workloads and the 32B TP-4 share.
constexpr int kMixedItemsPerSlot = 2;
constexpr int kDefaultWaves = 4;
}  // namespace laminar_detail
