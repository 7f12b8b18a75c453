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
 * to (§6.2):
 *
 *     y[m, n] = sum_k x[m, k] * w[n, k]      m < M, n < N, k < K
 *
 * x [M, K] bf16 (one row per trajectory), w [N, K] bf16 (one row per output
 * feature: the usual layout of a linear layer's weight), y [M, N] fp32,
 * all row-major and contiguous. Products of bf16 values are exact and are
 * accumulated in fp32 on the matrix cores; with several K splits the
 * partial sums are added in a fixed order, so results are deterministic.
 *
 * Limits: 1 <= M <= 64, N a multiple of 16, K a multiple of 128; larger
 * batches are compute-bound and belong to a general GEMM.
 * Workspace: laminar_linear_workspace_bytes(M, N, K) bytes of device
 * memory (0 when no K split is used), 256-byte aligned, owned by the
 * caller; calls that share a workspace must be ordered on one stream.
 * Pointers: x, w 16-byte aligned; y 16-byte aligned.
 * Errors: INVALID_ARG (NULL pointers, misalignment, a workspace smaller
 * than required), UNSUPPORTED (M, N or K outside the limits), HIP (launch
 * failure).
 */
#ifndef LAMINAR_LINEAR_H
#define LAMINAR_LINEAR_H

#include "laminar_decode_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Number of K splits the call will use (1: none). 0 outside the limits. */
int32_t laminar_linear_splits(int32_t m, int32_t n, int32_t k);

/* Device workspace bytes for the K splits (0 when there are none). */
size_t laminar_linear_workspace_bytes(int32_t m, int32_t n, int32_t k);

laminar_status laminar_linear(const void* x, const void* w, float* y,
                              int32_t m, int32_t n, int32_t k,
                              void* workspace, size_t workspace_bytes,
                              hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* LAMINAR_LINEAR_H */
