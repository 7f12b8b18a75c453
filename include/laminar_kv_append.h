/*
 * laminar_kv_append.h -- C ABI of the KV-cache append that precedes decode
 * attention in every decode step.
 *
 * What it computes. Each decode step of a rollout extends every running
 * trajectory's KV cache by the current token before attention reads it
 * (the KV cache whose capacity bounds the decode batch, the paper's §5.2;
 * decoding is memory-bound, §2.4). For trajectory b with n = seq_lens[b]
 * tokens *including* the new one, the token index is t = n - 1, its page
 * pp = block_table[b, t / 16] and its slot u = t % 16. For every kv-head h,
 * k_new[b, h, :] and v_new[b, h, :] are stored at slot u of the (pp, h) K
 * and V tiles, in the page formats described in laminar_decode_attn.h.
 * Nothing is written for n = 0, for t / 16 >= max_blocks_per_seq, or for a
 * table entry outside [0, num_pages).
 *
 * fp8 (OCP E4M3FN) pools. Each (page, kv-head) tile has one fp32 scale for
 * K and one for V, with the meaning the attention kernels read: scale =
 * amax / 448 over the page's valid tokens (1 when that amax is 0), code =
 * RNE(clamp(x / scale, -448, 448)). The append keeps that meaning, all in
 * float32 with each operation rounded once:
 *   a = max_d |x_d|, c = a / 448;
 *   if u == 0, or the scale is 1 and every valid older code is +-0, the
 *     scale becomes c (1 if a == 0);
 *   else if c > scale, the scale becomes c and every valid older code is
 *     re-encoded as RNE(clamp((dec(code) * old_scale) / c, +-448));
 *   the new token is stored as RNE(clamp(x_d / scale, +-448)).
 * The resulting scale equals fl(max |x| / 448) over the page's appended
 * values, as if the page were quantised at once; older codes carry one
 * extra rounding per re-encoding.
 *
 * Arguments (device pointers unless stated):
 *   desc         host; uses batch, num_kv_heads, head_dim (64 or 128),
 *                page_size (16), num_pages, max_blocks_per_seq, kv_dtype,
 *                input_row_stride. Its k_scale / v_scale fields are
 *                ignored: the writable scale arrays are passed below.
 *   k_new, v_new [batch, num_kv_heads, head_dim] bf16, 16-byte aligned;
 *                trajectory b's row starts input_row_stride elements after
 *                trajectory b-1's (0: num_kv_heads x head_dim, contiguous),
 *                so both may point into a fused QKV projection's output.
 *   block_table  [batch, max_blocks_per_seq] int32.
 *   seq_lens     [batch] int32, lengths after this append.
 *   k_pages, v_pages  the pools, updated in place.
 *   k_scale, v_scale  [num_pages, num_kv_heads] fp32, updated in place;
 *                required for fp8, ignored for bf16.
 * Ownership: nothing is retained after the call; no memory is allocated.
 * Concurrency: two trajectories may not append into the same (page, slot),
 * nor into the same fp8 (page, kv-head) tile; a page shared with other
 * trajectories must be copied before it is written. The append must be
 * ordered before the attention call that reads the token (same stream).
 * Errors: INVALID_ARG (NULL pointers when batch > 0, bad sizes, missing fp8
 * scales, k_new / v_new / the pools not 16-byte aligned, block_table /
 * seq_lens / the scales not 4-byte aligned, an input_row_stride below
 * num_kv_heads x head_dim or not a multiple of 8), UNSUPPORTED (page_size != 16, head_dim
 * not 64 or 128), HIP (launch failure).
 */
#ifndef LAMINAR_KV_APPEND_H
#define LAMINAR_KV_APPEND_H

#include "laminar_decode_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

laminar_status laminar_kv_append(const laminar_attn_desc* desc,
                                 const void* k_new, const void* v_new,
                                 const int32_t* block_table,
                                 const int32_t* seq_lens, void* k_pages,
                                 void* v_pages, float* k_scale, float* v_scale,
                                 hipStream_t stream);

/*
 * Pack row-major KV pages into the tile order of laminar_decode_attn.h, for
 * callers whose cache (or whose producer of K and V) keeps each (page,
 * kv-head) tile as 16 token rows of head_dim contiguous elements, i.e. a
 * pool [num_pages, num_kv_heads, 16, head_dim] (the paged KV cache whose
 * capacity the paper's §5.2 budgets). src holds num_tiles such tiles
 * (num_pages x num_kv_heads), dst receives them in the K order (which = 0)
 * or the V order (which = 1) for elements of kv_dtype (bf16: 2 bytes, fp8
 * e4m3fn: 1 byte; codes are moved, never converted, so fp8 scales are
 * unchanged). Both are device pointers, 16-byte aligned, and must not
 * overlap. Enqueued on `stream`; nothing is allocated or retained.
 * Errors: INVALID_ARG (NULL or misaligned pointers when num_tiles > 0,
 * overlapping buffers, num_tiles < 0, which or kv_dtype out of range),
 * UNSUPPORTED (head_dim not 64 or 128), HIP (launch failure).
 */
laminar_status laminar_kv_pack(const void* src, void* dst, int64_t num_tiles,
                               int32_t head_dim, int32_t kv_dtype,
                               int32_t which, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* LAMINAR_KV_APPEND_H */
