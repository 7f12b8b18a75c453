/*
 * laminar_repack.h -- C ABI of trajectory repacking on one GPU: the
 * best-fit consolidation plan (host) and the page migration (device) that
 * moves the released rollouts' trajectories into their destinations.
 *
 * What it computes. Long-tail generation leaves many rollouts running a
 * few long trajectories each. Repacking (the paper's §5.2) picks rollouts
 * whose KV usage is falling (below the limit and below the previous check)
 * and that run fewer trajectories than the roofline batch bound, visits
 * them from the least used up, and moves each into the candidate that can
 * still take it (usage within kv_max, trajectories within batch_max,
 * counting everything already planned into it) and ends up fullest
 * (Algorithm 1). A rollout that has received trajectories is not moved
 * itself (the feasibility test counts only the source's own usage, so
 * moving it would strand what it received). Ties: equal usage keeps the
 * input order; among equally full destinations the first visited wins.
 * On one GPU each rollout owns a page pool; moving a trajectory copies
 * its pages into free pages of the destination pool and rewrites its
 * block-table row; page contents, and so attention, are unchanged.
 *
 * Conventions as in laminar_decode_attn.h: statuses, no exceptions, host
 * arrays read during the call only, device work enqueued on `stream`.
 */
#ifndef LAMINAR_REPACK_H
#define LAMINAR_REPACK_H

#include "laminar_decode_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

/* One rollout replica at a repack check (host struct). */
typedef struct {
  int64_t kv_used;    /* KV pages in use now                       */
  int64_t kv_prev;    /* KV pages in use at the previous check     */
  int32_t num_reqs;   /* running trajectories                      */
  int32_t reserved;   /* 0                                         */
} laminar_rollout_state;

/*
 * Consolidation plan (Algorithm 1, §5.2). Writes the (source, destination)
 * rollout indices of every planned move, in decision order, to src_out /
 * dst_out (host, capacity >= num_rollouts) and their number to *num_pairs.
 * O(candidates^2) time, host only.
 * Errors: INVALID_ARG (NULL pointers with num_rollouts > 0, num_rollouts <
 * 0, kv_max < 0, batch_max < 0, negative usage or counts).
 */
laminar_status laminar_repack_plan(const laminar_rollout_state* rollouts,
                                   int32_t num_rollouts, int64_t kv_max,
                                   int32_t batch_max, int32_t* src_out,
                                   int32_t* dst_out, int32_t* num_pairs);

/*
 * Page assignment for moving n_traj trajectories into a destination pool
 * (host bookkeeping). src_table [n_traj, src_width] holds their block-table
 * rows (-1 unused) and lens [n_traj] their lengths; block j < ceil(len/16)
 * of each is moved. Destination pages are taken in order from dst_free
 * [n_free]; a source page used by several of the trajectories (a shared
 * prefix) is copied once and shared again. Writes the destination rows to
 * dst_table [n_traj, dst_width] (-1 past each trajectory's blocks), the
 * (source page, destination page) pairs to pairs [capacity][2], their
 * number to *num_pairs and the number of free pages used to *free_used.
 * Errors: INVALID_ARG (NULL pointers, negative sizes, a length needing
 * more than src_width or dst_width blocks, a negative table entry inside a
 * length, too few free pages, capacity too small).
 */
laminar_status laminar_migration_pairs(const int32_t* src_table,
                                       const int32_t* lens, int32_t n_traj,
                                       int32_t src_width,
                                       const int32_t* dst_free, int32_t n_free,
                                       int32_t* dst_table, int32_t dst_width,
                                       int32_t* pairs, int32_t capacity,
                                       int32_t* num_pairs, int32_t* free_used);

/*
 * Copy pages between two pools (device): for every row (s, d) of pairs
 * [num_pairs][2] (device int32), bytes [s*page_bytes, (s+1)*page_bytes) of
 * src_pool go to [d*page_bytes, ...) of dst_pool. Call once per pool of a
 * rollout (K pages, V pages, and for fp8 the K and V scales, whose page is
 * num_kv_heads * 4 bytes). page_bytes must be a positive multiple of 4;
 * pools 16-byte aligned when page_bytes is a multiple of 16, 4-byte
 * aligned otherwise; pairs 8-byte aligned. Rows with s outside
 * [0, src_pages) or d outside [0, dst_pages) are skipped. Destination
 * pages must be distinct and the two pools must not overlap.
 * Errors: INVALID_ARG (NULL pointers with num_pairs > 0, bad sizes or
 * alignment), HIP (launch failure).
 */
laminar_status laminar_migrate_pages(const void* src_pool, int64_t src_pages,
                                     void* dst_pool, int64_t dst_pages,
                                     size_t page_bytes, const int32_t* pairs,
                                     int32_t num_pairs, hipStream_t stream);

/* Dense decoder shape for the roofline batch bound (host struct). */
typedef struct {
  int32_t layers, hidden, q_heads, kv_heads, head_dim, intermediate, vocab;
  int32_t weight_bytes;   /* bytes per weight element (2 for bf16)        */
  int32_t act_bytes;      /* bytes per activation element (2 for bf16)    */
  int32_t kv_bytes;       /* bytes per KV element (2 bf16, 1 fp8)         */
} laminar_model_shape;

/*
 * Roofline batch bound B of Algorithm 1 (§5.2): the smallest decode batch
 * at which one step's projections (per layer QKV, O, gate+up and down, and
 * the LM head; a [M, K] x [K, N] product does 2 M N K flops and moves
 * weight_bytes N K + act_bytes M (K + N) bytes) are compute-bound at peak
 * compute peak_flops (FLOP/s) and bandwidth peak_bw (B/s):
 *   B = min { M >= 1 : sum 2 M N K / F >= sum (wb N K + ab M (K + N)) / BW }.
 * Attention is memory-bound at every batch (its intensity is
 * q_heads / (kv_heads kv_bytes) flops per byte) and adds a cost per
 * trajectory, not a transition. Exact integer arithmetic. *bound = 0 when
 * no batch is compute-bound (activation traffic outweighs the gain).
 * Errors: INVALID_ARG (NULL pointers, non-positive sizes or peaks).
 */
laminar_status laminar_roofline_batch_bound(const laminar_model_shape* shape,
                                            uint64_t peak_flops,
                                            uint64_t peak_bw, int32_t* bound);

/*
 * Roofline time of one decode step of `batch` trajectories holding
 * `context` cached tokens each: every projection at max(flops / F,
 * bytes / BW), plus per layer attention at max(4 M c Hq D / F,
 * kv_bytes 2 Hkv D M (c + 1) / BW). Written to *seconds.
 * Errors: INVALID_ARG (NULL pointers, non-positive sizes or peaks,
 * negative batch or context).
 */
laminar_status laminar_roofline_step_seconds(const laminar_model_shape* shape,
                                             int64_t batch, int64_t context,
                                             uint64_t peak_flops,
                                             uint64_t peak_bw, double* seconds);

#ifdef __cplusplus
}
#endif

#endif /* LAMINAR_REPACK_H */
