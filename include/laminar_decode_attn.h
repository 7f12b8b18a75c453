/*
 * laminar_decode_attn.h -- C ABI of the MI355X (gfx950) paged grouped-query
 * decode-attention library.
 *
 * What it computes. Rollout decoding in asynchronous RL post-training is
 * memory-bound and dominates the iteration (the paper's §1 and §2.4); every
 * decode step of every layer reads each trajectory's paged KV cache (§5.2).
 * For trajectory b with n = seq_lens[b] cached tokens and query head h,
 * using kv-head kvh = h / g (g = num_q_heads / num_kv_heads):
 *
 *     s_t      = softmax_scale * dot(q[b,h,:], K_t)      for t < n
 *     lse[b,h] = ln(sum_t exp(s_t))                       (natural log)
 *     out[b,h] = sum_t exp(s_t - lse[b,h]) * V_t
 *
 * where K_t, V_t are read from physical page block_table[b, t/16], slot t%16.
 * n = 0 gives out = 0 and lse = -inf. The work is split across CUs into
 * (trajectory, kv-head, page range) items whose partial (out, lse) pairs are
 * combined with the log-sum-exp merge
 *     L = ln(sum_s exp(lse_s)),  out = sum_s exp(lse_s - L) * out_s.
 *
 * Conventions for every entry point:
 *   - Functions return laminar_status and never abort or throw.
 *   - Device pointers come from the caller (e.g. torch allocations) and are
 *     not retained past the call, except the workspace bound to a plan.
 *   - Calls only enqueue work on `stream`; results are valid once the stream
 *     has been synchronised. A NULL stream is HIP's null stream.
 *   - Argument errors are reported before any launch; a failed launch
 *     returns LAMINAR_ERR_HIP. Asynchronous faults surface through HIP at
 *     the next synchronisation.
 *
 * Memory layouts (all row-major, contiguous, element = 2 bytes for bf16 and
 * 1 byte for fp8):
 *   q            [batch, num_q_heads, head_dim]         bf16 (rows
 *                input_row_stride elements apart when that is set)
 *   k_pages      [num_pages, num_kv_heads, 16*head_dim] bf16 or fp8 e4m3fn
 *   v_pages      [num_pages, num_kv_heads, 16*head_dim] bf16 or fp8 e4m3fn
 *   block_table  [batch, max_blocks_per_seq]            int32
 *   seq_lens     [batch]                                int32 (device)
 *   out          [batch, num_q_heads, head_dim]         fp32
 *   lse          [batch, num_q_heads]                   fp32
 *   k_scale, v_scale [num_pages, num_kv_heads]          fp32 (fp8 only)
 * One (page, kv-head) tile holds 16 tokens x head_dim elements. With
 * X = 16 bytes / element size, token t and dim d sit at element
 *   K: ((d / X) * 16 + t) * X + d % X          ([head_dim/X][16][X])
 *   V: ((t / 4) * head_dim + d) * 4 + t % 4    ([4][head_dim][4])
 * so that every lane of a wave reads its matrix-core operands with 16-byte
 * loads and each load instruction covers whole 256-byte runs.
 * fp8 values are OCP E4M3FN codes; the value of a code is decode(code) *
 * scale[page, kv-head] (separate scales for K and V).
 */
#ifndef LAMINAR_DECODE_ATTN_H
#define LAMINAR_DECODE_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* HIP's stream handle (identical to the typedef in hip_runtime_api.h). */
typedef struct ihipStream_t* hipStream_t;

typedef enum {
  LAMINAR_OK = 0,
  LAMINAR_ERR_INVALID_ARG = 1,  /* NULL pointer, bad size or mismatch      */
  LAMINAR_ERR_UNSUPPORTED = 2,  /* valid but not built (head_dim, group)   */
  LAMINAR_ERR_WORKSPACE = 3,    /* workspace missing, too small, misaligned */
  LAMINAR_ERR_HIP = 4           /* a HIP call or kernel launch failed      */
} laminar_status;

typedef enum {
  LAMINAR_KV_BF16 = 0,
  LAMINAR_KV_FP8_E4M3FN = 1
} laminar_kv_dtype;

/* Problem description, copied into the plan. */
typedef struct {
  int32_t batch;               /* >= 0 trajectories                          */
  int32_t num_q_heads;         /* Hq >= 1                                    */
  int32_t num_kv_heads;        /* Hkv >= 1, Hq % Hkv == 0, Hq/Hkv <= 16      */
  int32_t head_dim;            /* 64 or 128                                  */
  int32_t page_size;           /* must be 16                                 */
  int32_t num_pages;           /* >= 1 pages in the pool                     */
  int32_t max_blocks_per_seq;  /* block_table row stride, >= ceil(n/16)      */
  int32_t kv_dtype;            /* laminar_kv_dtype                           */
  float softmax_scale;         /* > 0, e.g. 1/sqrt(head_dim)                 */
  const float* k_scale;        /* device [num_pages, Hkv]; fp8 only, else NULL */
  const float* v_scale;        /* device [num_pages, Hkv]; fp8 only, else NULL */
  int32_t pages_per_item;      /* 0: automatic; > 0: at most this many pages
                                  per work item (1 .. no split)              */
  int32_t waves_per_item;      /* 0: automatic (4); else 1, 2 or 4 wavefronts
                                  cooperate on one work item                 */
  int32_t input_row_stride;    /* elements from one trajectory's row of the
                                  per-token inputs to the next: q for decode
                                  attention, k_new and v_new for KV append.
                                  0: contiguous (heads x head_dim); else at
                                  least that and a multiple of 8, e.g. the
                                  row of a fused QKV projection's output     */
} laminar_attn_desc;

typedef struct laminar_plan laminar_plan;   /* opaque, host-owned */

/*
 * Plan the split of one decode step's KV work across `num_cus` compute units
 * (256 on MI355X). seq_lens_host[batch] are the trajectory lengths the next
 * decode_attn calls will see (host memory, read during the call only). Each
 * (trajectory, kv-head) unit of ceil(n/16) pages is cut into near-equal,
 * page-aligned ranges of at most pages_per_item pages; items are ordered
 * longest first. Pure host work: no HIP call, no device memory touched.
 * The plan is reusable by every layer of the step. On success *out owns a
 * new plan (free with laminar_plan_destroy); on error *out is NULL.
 * Errors: INVALID_ARG (NULL pointers, negative or inconsistent sizes, a
 * length needing more than max_blocks_per_seq pages, fp8 without scales
 * or with scale pointers that are not 4-byte aligned,
 * an input_row_stride below num_q_heads x head_dim or not a multiple of 8),
 * UNSUPPORTED (head_dim not 64/128, group size above 16, page_size != 16).
 */
laminar_status laminar_plan_create(const laminar_attn_desc* desc,
                                   const int32_t* seq_lens_host,
                                   int32_t num_cus, laminar_plan** out);

/*
 * Cascade plan for batches whose trajectories share prompt prefixes (the
 * paper's GRPO groups: 16 responses per prompt, §8 "Settings"). Group
 * g's members are the trajectories b with group_of_host[b] == g (-1: no
 * group); the caller guarantees that blocks 0 .. group_pages_host[g] - 1 of
 * every member (as far as the member is long) map to the same physical
 * pages. The shared pages of up to waves_per_item x (16 / g_q) members
 * (g_q = num_q_heads / num_kv_heads) are then read once per kv-head: one
 * work item gives each wavefront the query rows of 16 / g_q members and
 * masks each row at its member's length, and each member's result is the
 * log-sum-exp merge of that partial with its own pages' partials. Exact:
 * the result is the same attention as laminar_plan_create's, up to fp32
 * rounding. Groups of one member, or with no shared page, decode as usual.
 * All arrays are host memory read during the call. num_groups == 0 is
 * laminar_plan_create.
 * Errors: those of laminar_plan_create, and INVALID_ARG for num_groups < 0,
 * NULL group arrays with num_groups > 0, group_of outside [-1, num_groups)
 * or a negative group_pages entry.
 */
laminar_status laminar_plan_create_cascade(const laminar_attn_desc* desc,
                                           const int32_t* seq_lens_host,
                                           const int32_t* group_of_host,
                                           int32_t num_groups,
                                           const int32_t* group_pages_host,
                                           int32_t num_cus, laminar_plan** out);

/* Bytes of device workspace the plan needs (work list, merge list, partial
 * outputs). 0 for a NULL plan. */
size_t laminar_plan_workspace_bytes(const laminar_plan* plan);

/*
 * Bind a caller-owned device workspace of `bytes` >= workspace_bytes, 256-byte
 * aligned, and enqueue the upload of the plan's work and merge lists into it
 * on `stream`. The lists are first copied into a pinned, device-mapped host
 * staging slot of the library (one small ring per device, allocated on first
 * use and kept until the process exits) and a small kernel on `stream`
 * copies them into the workspace, so the upload does not cross to a DMA
 * engine and the plan may be destroyed as soon as this call returns. The
 * ring has eight slots: the call waits only when the upload eight binds ago
 * has not run yet.
 * Lists larger than one staging slot (1 MiB, about 65k work items) are
 * copied directly and the call waits for `stream` to finish the copy.
 * The workspace must stay allocated, and must not be used by anything else,
 * while calls with this plan may run; binding another plan to the same
 * workspace on the same stream is ordered after those calls.
 * Errors: INVALID_ARG, WORKSPACE, HIP.
 */
laminar_status laminar_plan_bind_workspace(laminar_plan* plan, void* workspace,
                                           size_t bytes, hipStream_t stream);

/*
 * Paged GQA decode attention for the whole batch: the split-KV partial pass
 * followed by the log-sum-exp merge of trajectories that were split. q, the
 * page pools, block_table, seq_lens, out and lse are device pointers in the
 * layouts above; seq_lens must hold the lengths the plan was created from
 * (longer device lengths are clipped to the plan's page ranges). Block-table
 * entries outside [0, num_pages) contribute nothing. Calls with one plan
 * share its workspace (partial results and the counter that hands out the
 * dynamic tail items) and must therefore be ordered on one stream.
 * Errors, checked in this order before any launch: INVALID_ARG (NULL
 * plan; with batch > 0, a NULL pointer, or q, k_pages, v_pages or out not
 * 16-byte aligned, or block_table, seq_lens or lse not 4-byte aligned),
 * WORKSPACE (no workspace bound), HIP.
 */
laminar_status laminar_decode_attn(const laminar_plan* plan, const void* q,
                                   const void* k_pages, const void* v_pages,
                                   const int32_t* block_table,
                                   const int32_t* seq_lens, float* out,
                                   float* lse, hipStream_t stream);

/*
 * The first half of laminar_decode_attn on its own: every work item's
 * attention over its page range. Items of unsplit trajectories write out and
 * lse directly; the others write partial results into the workspace, to be
 * combined by laminar_decode_attn_merge. Same arguments and errors.
 */
laminar_status laminar_decode_attn_partial(const laminar_plan* plan,
                                           const void* q, const void* k_pages,
                                           const void* v_pages,
                                           const int32_t* block_table,
                                           const int32_t* seq_lens, float* out,
                                           float* lse, hipStream_t stream);

/*
 * The second half: merge the partial (out, lse) of each split trajectory into
 * out and lse. Must follow laminar_decode_attn_partial with the same plan on
 * the same stream. Errors: INVALID_ARG (NULL plan; with batch > 0, out
 * NULL or not 16-byte aligned, lse NULL or not 4-byte aligned), WORKSPACE,
 * HIP.
 */
laminar_status laminar_decode_attn_merge(const laminar_plan* plan, float* out,
                                         float* lse, hipStream_t stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the
 * same computation as laminar_decode_attn, with the library's own static
 * workspace of LAMINAR_STATIC_WORKSPACE_BYTES per GPU (a device array that
 * the GPU holds from the library's load until the process ends) in place
 * of a workspace bound to the plan. The plan need not be bound. Each call
 * copies the plan's tables from its host memory into that workspace with
 * hipMemcpyAsync on `stream` and launches the same kernels; it calls no
 * allocation routine. Keep the plan alive until the stream has passed the
 * call. Every call on one GPU shares that GPU's workspace, which keeps the
 * last call's contents: calls that overlap on one GPU (other streams, other
 * threads) race and give wrong results; order them on one stream.
 * Errors, before any launch: INVALID_ARG (as laminar_decode_attn),
 * WORKSPACE (the plan needs more than LAMINAR_STATIC_WORKSPACE_BYTES, see
 * laminar_plan_workspace_bytes), HIP (the workspace's device address could
 * not be found, or a copy or launch failed).
 */
#define LAMINAR_STATIC_WORKSPACE_BYTES (64u << 20)
laminar_status laminar_decode_attn_static(const laminar_plan* plan,
                                          const void* q, const void* k_pages,
                                          const void* v_pages,
                                          const int32_t* block_table,
                                          const int32_t* seq_lens, float* out,
                                          float* lse, hipStream_t stream);

/* Plan introspection (host only). Items are listed in launch order
 * (longest first, one workgroup each). Each item is 4 int32:
 * (b * num_kv_heads + kvh, first page, end page, partial slot or -1 when the
 * item writes out/lse directly), or for a cascade item (-(cascade unit) - 1,
 * first page, end page, piece index). Each merge is 4 int32: (unit, first
 * slot, number of slots, 0). Each cascade unit is 4 int32: (trajectory whose
 * block-table row is read, member count, first member record, kv-head); each
 * member record is 2 int32: (trajectory, first partial slot of its unit).
 * *_copy writes min(count, capacity) records and returns the number written,
 * or -1 for a NULL argument. */
int32_t laminar_plan_num_items(const laminar_plan* plan);
int32_t laminar_plan_num_merges(const laminar_plan* plan);
int32_t laminar_plan_pages_per_item(const laminar_plan* plan);
int32_t laminar_plan_waves_per_item(const laminar_plan* plan);
int32_t laminar_plan_items_copy(const laminar_plan* plan, int32_t* dst,
                                int32_t capacity);
int32_t laminar_plan_merges_copy(const laminar_plan* plan, int32_t* dst,
                                 int32_t capacity);
/* Items at the end of the list that are handed out dynamically (the
 * smallest ones; workgroups past the bound items take the next of them when
 * they start, so XCDs that run ahead take more). */
int32_t laminar_plan_num_dynamic_items(const laminar_plan* plan);
int32_t laminar_plan_num_cascade_units(const laminar_plan* plan);
int32_t laminar_plan_num_cascade_members(const laminar_plan* plan);
int32_t laminar_plan_cascade_units_copy(const laminar_plan* plan, int32_t* dst,
                                        int32_t capacity);
int32_t laminar_plan_cascade_members_copy(const laminar_plan* plan,
                                          int32_t* dst, int32_t capacity);

/* Free a plan (NULL is a no-op). Does not free the bound workspace. */
void laminar_plan_destroy(laminar_plan* plan);

/* Static description of a status code. */
const char* laminar_status_string(laminar_status status);

/*
 * HBM calibration kernels (measurement support, not part of the attention).
 * laminar_hbm_read streams `bytes` (a multiple of 16, 16-byte aligned) from
 * `src` and writes one fp32 partial sum per workgroup into `sink`, which must
 * hold laminar_hbm_read_sink_floats() floats. laminar_hbm_copy copies `bytes`
 * (a multiple of 16, both pointers 16-byte aligned) from src to dst.
 * Errors: INVALID_ARG, HIP.
 */
int32_t laminar_hbm_read_sink_floats(void);
/*
 * laminar_hbm_gather reads n_idx tiles of tile_bytes (a power of two, at
 * least 16) from src, tile t of the list being bytes
 * [idx[t] * tile_bytes, (idx[t] + 1) * tile_bytes) of the src_bytes-long
 * buffer (indices outside it are clamped to its last tile), the way the
 * attention kernel gathers 4 KiB KV tiles through a block table. src is
 * 16-byte aligned; idx (int32, n_idx entries) and sink are device memory.
 * sink receives laminar_hbm_gather_sink_words(n_idx, tile_bytes) uint32
 * partial sums, one per workgroup; their sum mod 2^32 is the sum of every
 * 32-bit word read, a checksum the caller can recompute. n_idx == 0 does
 * nothing. Errors: INVALID_ARG, HIP.
 */
int32_t laminar_hbm_gather_sink_words(int64_t n_idx, size_t tile_bytes);
laminar_status laminar_hbm_gather(const void* src, size_t src_bytes,
                                  size_t tile_bytes, const int32_t* idx,
                                  int64_t n_idx, uint32_t* sink,
                                  hipStream_t stream);
laminar_status laminar_hbm_read(const void* src, size_t bytes, float* sink,
                                hipStream_t stream);
laminar_status laminar_hbm_copy(void* dst, const void* src, size_t bytes,
                                hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* LAMINAR_DECODE_ATTN_H */
