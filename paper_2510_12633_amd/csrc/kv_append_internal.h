// Argument checks of laminar_kv_append, shared with the projection entry
// point whose K-split reduction makes the same append
// (laminar_linear_bf16_kv_append), so that both refuse the same calls.
#ifndef LAMINAR_KV_APPEND_INTERNAL_H
#define LAMINAR_KV_APPEND_INTERNAL_H

#include "laminar_kv_append.h"

namespace laminar_detail {

// LAMINAR_OK when laminar_kv_append would accept the call; *empty is set
// when it would write nothing (batch or num_kv_heads x batch zero).
laminar_status kv_append_check(const laminar_attn_desc* d, const void* k_new,
                               const void* v_new, const int32_t* block_table,
                               const int32_t* seq_lens, const void* k_pages,
                               const void* v_pages, const float* k_scale,
                               const float* v_scale, bool* empty);

}  // namespace laminar_detail

#endif
