// Internal interface between the attention kernels (decode_attn.hip) and
// the C-ABI entry points that validate calls and launch them
// (attn_entry.hip). Not part of the public C ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "laminar_decode_attn.h"
#include "plan_internal.h"

namespace laminar_detail {

// Device pointers of one attention call. ws is the workspace whose layout
// the plan describes (work list, merge records, cascade tables, tail
// counter, partial results), already holding the plan's tables.
struct AttnCall {
  const void* q;
  const void* k_pages;
  const void* v_pages;
  const int32_t* block_table;
  const int32_t* seq_lens;
  float* out;
  float* lse;
  void* ws;
};

// Enqueue the partial pass (every work item) or the log-sum-exp merge of
// the plan's split units on `stream`. The caller has validated the call.
laminar_status enqueue_partial(const laminar_plan& p, const AttnCall& c,
                               hipStream_t stream);
laminar_status enqueue_merge(const laminar_plan& p, const AttnCall& c,
                             hipStream_t stream);

}  // namespace laminar_detail
