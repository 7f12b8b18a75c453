/*
 * laminar_decode_step.h -- C ABI of the element-wise operations a decode
 * step runs between its projections and its attention: the RMS pre-norm
 * and the gated (SwiGLU) activation of each layer.
 *
 * What it computes. The decode-latency curve (the paper's §2.4) and the
 * roofline batch bound B of Algorithm 1 (§5.2) are about whole decode
 * steps of the rollout models (Qwen2.5, §8 "Models"), whose layers put
 * these two operations around the projections of laminar_linear.h and the
 * attention of laminar_decode_attn.h. They move a few kilobytes per token
 * and are launch-bound at decode batch sizes; one fused kernel each keeps a
 * step from spending more time in element-wise launches than in reading
 * its weights.
 *
 *   laminar_rmsnorm:   y[m, :] = bf16(x[m, :] / sqrt(mean_k x[m, k]^2 + eps)
 *                                     * weight[:])
 *   laminar_silu_mul:  y[m, i] = bf16(silu(gu[m, i]) * gu[m, I + i]),
 *                      silu(g) = g / (1 + exp(-g)),  i < I
 *
 * All arithmetic in fp32 from bf16 inputs, one rounding to bf16 (nearest
 * even) at the end; exp(-g) and the division of silu use the hardware
 * exponential and reciprocal (a few fp32 ulp before that rounding). Layouts row-major and contiguous: x, y [M, N] bf16,
 * weight [N] bf16 (NULL for all ones), gu [M, 2I] bf16 (gate then up), y
 * [M, I] bf16. Pointers 16-byte aligned; N and I multiples of 8. y may not
 * overlap the inputs. Errors: INVALID_ARG (NULL, misaligned, M < 1, N or I
 * not a positive multiple of 8, eps not finite or negative), HIP (launch).
 */
#ifndef LAMINAR_DECODE_STEP_H
#define LAMINAR_DECODE_STEP_H

#include "laminar_decode_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

laminar_status laminar_rmsnorm(const void* x, const void* weight, void* y,
                               int32_t m, int32_t n, float eps,
                               hipStream_t stream);

laminar_status laminar_silu_mul(const void* gu, void* y, int32_t m,
                                int32_t inter, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* LAMINAR_DECODE_STEP_H */
