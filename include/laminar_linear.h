/*
 * laminar_linear.h -- C ABI of the skinny projection product of a decode
 * step: y = x w^T for a small batch of tokens.
 *
 * What it computes. Each decode step runs every layer's projections (QKV,
 * O, gate and up, down) and the LM head over one token per trajectory. At
 * decode batch sizes they stream the whole weight matrix for a handful of
 * rows, so they are bound by HBM bandwidth and set the latency floor that
 * makes a small decode batch cost about as much as a larger one (the
 * paper's §2.4) and that the roofline batch bound B of Algorithm 1 refers
 * to (§5.2):
 *
 *     y[m, n] = sum_k x[m, k] * w[n, k]      m < M, n < N, k < K
 *
 * x [M, K] bf16 (one row per trajectory), w [N, K] bf16 (one row per output
 * feature: the usual layout of a linear layer's weight), y [M, N] fp32,
 * all row-major and contiguous. Products of bf16 values are exact and are
 * accumulated in fp32 on the matrix cores; with several K splits (over
 * workgroups, over the four wavefronts of one workgroup for M <= 4, or the
 * pieces of the balanced split) the partial sums are added in a fixed
 * order, so results are deterministic.
 *
 * Packed weights. laminar_linear reads w in a packed layout made once per
 * weight by laminar_linear_pack: 16-row tiles, and within a tile 16-byte
 * chunks (8 consecutive k of one row) ordered (k / 8, row):
 *
 *     packed[((n / 16) * (K / 8) + k / 8) * 16 + n % 16][k % 8] = w[n][k]
 *
 * (same size as w). The 16 rows x 32 k that one matrix-core step consumes
 * are then 1 KB of contiguous bytes, which one wavefront load reads whole.
 *
 * Limits: 1 <= M <= 128, N a multiple of 16, K a multiple of 128 and at most
 * 2^24, and x padded to 16, 32, 64 or 128 rows at most 1 GiB (the kernels'
 * buffer offsets are 32-bit); larger batches are compute-bound and belong
 * to a general GEMM.
 * Workspace: laminar_linear_workspace_bytes(M, N, K) bytes of device
 * memory (0 when K is not split over workgroups), 256-byte aligned, owned
 * by the caller, zeroed once before its first use (hipMemset): it starts
 * with 256 counters (one per group of output columns, with which, up to 32
 * rows, the last workgroup of a group to finish adds the group's partial
 * sums itself) and holds the partial sums of the K split after them. Every
 * call leaves the counters at zero again, so no clearing is needed between
 * calls (nor in a captured graph), and the counters sit at the same place
 * for every shape: one workspace of the largest size serves calls of any
 * M, N and K. Calls that share a workspace must be ordered on one
 * stream. A call that fails part-way (a kernel fault) may leave counters
 * set: zero the workspace again before reusing it.
 * Pointers: x, w, w_packed and y 16-byte aligned; the caller owns every
 * buffer.
 * Errors: INVALID_ARG (NULL pointers, misalignment, w_packed equal to w, a
 * workspace smaller than required), UNSUPPORTED (M, N or K outside the
 * limits), HIP (launch failure).
 */
#ifndef LAMINAR_LINEAR_H
#define LAMINAR_LINEAR_H

#include "laminar_decode_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Writes the packed layout of w [N, K] bf16 to w_packed (same size, not
 * overlapping w). Enqueued on `stream`; a pure permutation of 16-byte
 * chunks. */
laminar_status laminar_linear_pack(const void* w, void* w_packed, int32_t n,
                                   int32_t k, hipStream_t stream);

/* Number of K ranges the call spreads over workgroups (1: none, also when
 * K is split only among the wavefronts of each workgroup); with the
 * balanced split (from 17 rows, when N / 128 groups would leave the CUs
 * unevenly loaded), the most pieces any left-over group is cut into. The
 * same for every kind of x. 0 outside the limits. */
int32_t laminar_linear_splits(int32_t m, int32_t n, int32_t k);

/* Device workspace bytes for the K splits over workgroups, or for the
 * pieces of the balanced split (0 when there are none). */
size_t laminar_linear_workspace_bytes(int32_t m, int32_t n, int32_t k);

/* y = x w^T with w given in the packed layout. */
laminar_status laminar_linear(const void* x, const void* w_packed, float* y,
                              int32_t m, int32_t n, int32_t k,
                              void* workspace, size_t workspace_bytes,
                              hipStream_t stream);

/* The same product with a bf16 output: y[m, n] = bf16(sum_k x[m, k] w[n, k]
 * + residual[m, n]), the fp32 sum (and the bf16 residual, if not NULL)
 * rounded once to nearest even. y and residual are [M, N] bf16, 16-byte
 * aligned, and may be the same buffer (an in-place residual add); the
 * decode step uses it for the projections whose outputs feed the next
 * bf16 operation, with the residual for O and down. */
laminar_status laminar_linear_bf16(const void* x, const void* w_packed,
                                   void* y, const void* residual, int32_t m,
                                   int32_t n, int32_t k, void* workspace,
                                   size_t workspace_bytes, hipStream_t stream);

/* What the x argument of laminar_linear_bf16_ex holds. */
typedef enum {
  LAMINAR_X_BF16 = 0,      /* x [M, K] bf16, as in laminar_linear_bf16 */
  LAMINAR_X_F32 = 1,       /* x [M, K] fp32; each value is rounded to bf16
                              (nearest even) before the product, as a cast
                              of x to bf16 would */
  LAMINAR_X_SILU_MUL = 2   /* x [M, 2K] bf16, gate then up: the product's
                              operand is bf16(silu(gate) * up), exactly what
                              laminar_silu_mul writes */
} laminar_linear_x;

/* laminar_linear_bf16 with the operand made from x on load (x_kind, one of
 * laminar_linear_x). A decode step uses it to read the fp32 attention
 * output directly in the O projection and the gate+up output directly in
 * the down projection, without the separate cast and SwiGLU launches; the
 * results equal those of the separate launches bit for bit. x is 16-byte
 * aligned. Errors as laminar_linear_bf16, plus INVALID_ARG for an unknown
 * x_kind (the RMS-norm input has its own call below). */
laminar_status laminar_linear_bf16_ex(const void* x, int32_t x_kind,
                                      const void* w_packed, void* y,
                                      const void* residual, int32_t m,
                                      int32_t n, int32_t k, void* workspace,
                                      size_t workspace_bytes,
                                      hipStream_t stream);

/* laminar_linear_bf16_ex followed by the RMS norm of each row of its
 * output: y as laminar_linear_bf16_ex writes it, and y_norm [M, N] bf16
 * equal bit for bit to laminar_rmsnorm(y, norm_weight, eps) (norm_weight
 * [N] bf16 or NULL). In a decode step the O and down projections write
 * the residual stream and the next RMS norm reads it: from 33 rows, where
 * K is split and a second kernel adds the ranges, that kernel also makes
 * the norm (one launch fewer); otherwise the norm is a laminar_rmsnorm
 * launch of its own. y_norm and norm_weight are 16-byte aligned; y_norm
 * must not overlap y. Errors as laminar_linear_bf16_ex, plus INVALID_ARG
 * for a NULL or misaligned y_norm, a misaligned norm_weight, or eps
 * negative or not finite. */
laminar_status laminar_linear_bf16_norm(const void* x, int32_t x_kind,
                                        const void* w_packed, void* y,
                                        const void* residual,
                                        const void* norm_weight, float eps,
                                        void* y_norm, int32_t m, int32_t n,
                                        int32_t k, void* workspace,
                                        size_t workspace_bytes,
                                        hipStream_t stream);

/* laminar_linear_bf16_ex (no residual) followed by SwiGLU of its output's
 * halves: y [M, N] bf16 as laminar_linear_bf16_ex writes it, and y_act
 * [M, N / 2] bf16 equal bit for bit to laminar_silu_mul(y) (gate columns
 * 0 .. N/2 - 1, up columns N/2 .. N - 1). For the gate and up projection:
 * when the call takes the balanced split with groups left over, its
 * reduction kernel also makes SwiGLU (one launch fewer); otherwise
 * SwiGLU is a laminar_silu_mul launch of its own. y_act is 16-byte aligned
 * and must not overlap y. Errors as laminar_linear_bf16_ex, plus
 * INVALID_ARG for a NULL or misaligned y_act. */
laminar_status laminar_linear_bf16_swiglu(const void* x, int32_t x_kind,
                                          const void* w_packed, void* y,
                                          void* y_act, int32_t m, int32_t n,
                                          int32_t k, void* workspace,
                                          size_t workspace_bytes,
                                          hipStream_t stream);

/* laminar_linear_bf16_ex (no residual) followed by the decode step's KV
 * append: y [M, N] bf16 as laminar_linear_bf16_ex writes it, then exactly
 * laminar_kv_append(kv_desc, y + k_col, y + v_col, block_table, seq_lens,
 * k_pages, v_pages, k_scale, v_scale) with kv_desc's input_row_stride
 * taken as N (its own value is ignored): row m is trajectory m's new token,
 * columns [k_col, k_col + num_kv_heads head_dim) its K and [v_col, ...) its
 * V. For the fused QKV projection in front of attention (the paged KV cache
 * of the paper's §5.2): from 33 rows, where K is split and a second kernel
 * adds the ranges, that kernel also stores K and V into bf16 pools (one
 * launch fewer); fp8 pools, and calls without that kernel, run the append
 * as its own launch. The pools and tables are laid out and checked as
 * laminar_kv_append's; kv_desc (host) must have batch = M. Pools, tables
 * and y must not overlap. Errors as laminar_linear_bf16_ex and
 * laminar_kv_append, plus INVALID_ARG for a NULL kv_desc, batch != M, or
 * k_col / v_col negative, not a multiple of 8, past N or overlapping. */
laminar_status laminar_linear_bf16_kv_append(
    const void* x, int32_t x_kind, const void* w_packed, void* y, int32_t m,
    int32_t n, int32_t k, void* workspace, size_t workspace_bytes,
    const laminar_attn_desc* kv_desc, int32_t k_col, int32_t v_col,
    const int32_t* block_table, const int32_t* seq_lens, void* k_pages,
    void* v_pages, float* k_scale, float* v_scale, hipStream_t stream);

/* laminar_linear_bf16 on RMS-normalised rows, the norm done on load:
 * the operand is bf16((x[m, k] r_m) norm_weight[k]) with
 * r_m = 1 / sqrt(mean_k x[m, k]^2 + eps), the pre-norm of a decoder layer
 * in front of its QKV and gate+up projections. Every workgroup finds the
 * r_m it needs with the summation order of laminar_rmsnorm, so the result
 * equals laminar_rmsnorm followed by laminar_linear_bf16 bit for bit, in
 * one launch. x [M, K] bf16 and norm_weight [K] bf16, 16-byte aligned.
 * Errors: INVALID_ARG (as laminar_linear_bf16, and a NULL or misaligned
 * norm_weight, eps negative or not finite), UNSUPPORTED (also M > 8: the
 * norm of larger batches is one laminar_rmsnorm launch). */
laminar_status laminar_linear_bf16_rmsnorm(const void* x,
                                           const void* norm_weight, float eps,
                                           const void* w_packed, void* y,
                                           const void* residual, int32_t m,
                                           int32_t n, int32_t k,
                                           void* workspace,
                                           size_t workspace_bytes,
                                           hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* LAMINAR_LINEAR_H */
