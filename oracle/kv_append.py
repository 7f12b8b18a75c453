"""CPU oracle for appending the current token's K and V to the paged cache.

TEST INFRASTRUCTURE. Only the tests, the package smoke check and the bench's
CPU-baseline leg may import or call this module. The GPU library never does,
and this module imports nothing from the GPU path.

What it computes. Every decode step of a rollout extends each running
trajectory's KV cache by one token before attention reads it (the KV cache
whose capacity bounds the decode batch, §5.2; decoding itself is
memory-bound, §2.4). The paper says nothing about how the cache is written,
so this module states the plain operation on the library's page formats:

  For trajectory b whose length n_b >= 1 already counts the new token, the
  token index is t = n_b - 1, its physical page pp = block_table[b, t // 16]
  and its slot u = t % 16. For every kv-head h the new key k_new[b, h] and
  value v_new[b, h] (bf16 codes, [D] each) are stored at slot u of the
  (pp, h) tiles. A trajectory with n_b = 0, a block index past the table
  width, or a table entry outside the pool appends nothing.

bf16 pools store the codes unchanged. fp8 (OCP E4M3FN) pools keep one fp32
scale per (page, kv-head) for K and one for V with the meaning the fp8
workloads use: scale = amax / 448 over the page's valid tokens (1 when that
amax is 0) and stored code = RNE(clamp(x / scale, -448, 448)). Appending one
token keeps that meaning incrementally (all arithmetic in float32, each
operation rounded once, which is what decides the codes):

  a_new = max_d |x_d|,  c = a_new / 448
  * u = 0, or s_old == 1 and every valid old code (slots < u) is +-0:
        the page holds no magnitude yet: s = c if a_new > 0 else 1.
  * otherwise s = s_old if c <= s_old, else s = c and every valid old code
        is re-encoded: code' = RNE(clamp((dec(code) * s_old) / s, +-448)).
  The new token is stored as RNE(clamp(x_d / s, +-448)) and the scale as s.

Because fl(./448) is monotone, s always equals fl(max over the page's
appended values of |x| / 448), the same scale the whole page would get if
quantised at once; only the codes of older tokens carry the extra rounding
of each re-encoding. Slots >= u + 1 are left as they are.

Two trajectories that append into the same (page, slot), or into the same
fp8 (page, kv-head) tile, are outside the operation: a shared page must be
copied before it is written.
"""
from __future__ import annotations

from typing import Tuple

import numpy as np

from .decode_attention import (E4M3FN_TABLE, PAGE, k_tile_offsets,
                               v_tile_offsets)

FP8_MAX = np.float32(448.0)

# Finite non-negative E4M3FN magnitudes, codes 0x00..0x7E, increasing.
_MAGS = E4M3FN_TABLE[:0x7F].astype(np.float64)


def e4m3fn_round(y: np.ndarray) -> np.ndarray:
    """float32 values with |y| <= 448 -> E4M3FN codes (uint8), round to
    nearest, ties to the even code; the sign bit follows the sign of y
    (so -0.0 and negatives that round to zero give 0x80)."""
    y = np.asarray(y, dtype=np.float32)
    a = np.abs(y).astype(np.float64).reshape(-1)
    assert np.all(a <= 448.0), "clamp before rounding"
    dist = np.abs(_MAGS[None, :] - a[:, None])              # [n, 127]
    best = dist.min(axis=1, keepdims=True)
    tie = dist == best
    codes = np.argmax(tie, axis=1)                          # lowest candidate
    two = tie.sum(axis=1) == 2                              # exact midpoint
    codes = np.where(two & (codes % 2 == 1), codes + 1, codes)
    codes = codes.astype(np.uint8).reshape(y.shape)
    return codes | (np.signbit(y).astype(np.uint8) << 7)


def quantize(x: np.ndarray, scale: np.float32) -> np.ndarray:
    """RNE(clamp(x / scale, +-448)) in float32, x float32."""
    y = np.asarray(x, dtype=np.float32) / np.float32(scale)
    return e4m3fn_round(np.clip(y, -FP8_MAX, FP8_MAX))


def _bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits).astype(np.uint32) << np.uint32(16)).view(np.float32)


def append_scale(old_codes: np.ndarray, s_old: np.float32,
                 x: np.ndarray) -> Tuple[np.float32, bool]:
    """(new scale, whether the old codes must be re-encoded) for one fp8
    (page, kv-head) tile, given its valid old codes [u, D] and the new
    token's float32 values [D]."""
    a_new = np.float32(np.abs(x).max()) if x.size else np.float32(0)
    c = np.float32(a_new / FP8_MAX)
    s_old = np.float32(s_old)
    empty = old_codes.shape[0] == 0 or (
        s_old == np.float32(1) and not np.any(old_codes & 0x7F))
    if empty:
        return (c if a_new > 0 else np.float32(1)), False
    if c > s_old:
        return c, True
    return s_old, False


def kv_append(k_pages, v_pages, k_scale, v_scale, block_table, seq_lens,
              k_new, v_new, *, head_dim: int, num_kv_heads: int,
              kv_dtype: str):
    """Return updated copies (k_pages, v_pages, k_scale, v_scale).

    k_pages/v_pages: [P, Hkv, 16*D] uint16 (bf16) or uint8 (fp8) codes in
    the library's tile order; k_scale/v_scale: float32 [P, Hkv] (fp8) or
    None; block_table int [B, W]; seq_lens int [B]; k_new/v_new: bf16 codes
    uint16 [B, Hkv, D].
    """
    fp8 = kv_dtype == "fp8_e4m3fn"
    kp, vp = np.array(k_pages), np.array(v_pages)
    ks = None if k_scale is None else np.array(k_scale, dtype=np.float32)
    vs = None if v_scale is None else np.array(v_scale, dtype=np.float32)
    bt = np.asarray(block_table)
    n_pages, width = kp.shape[0], bt.shape[1]
    ko = k_tile_offsets(head_dim, 1 if fp8 else 2)          # [16, D]
    vo = v_tile_offsets(head_dim)
    for b in range(len(seq_lens)):
        n = int(seq_lens[b])
        if n < 1 or (n - 1) // PAGE >= width:
            continue
        t = n - 1
        pp = int(bt[b, t // PAGE])
        if pp < 0 or pp >= n_pages:
            continue
        u = t % PAGE
        for h in range(num_kv_heads):
            for pages, scales, offs, new in ((kp, ks, ko, k_new),
                                             (vp, vs, vo, v_new)):
                if not fp8:
                    pages[pp, h, offs[u]] = new[b, h]
                    continue
                x = _bf16_to_f32(new[b, h])
                old = pages[pp, h, offs[:u]]                # [u, D]
                s_old = scales[pp, h]
                s, recode = append_scale(old, s_old, x)
                if recode:
                    deq = E4M3FN_TABLE[old.astype(np.int64)].astype(np.float32)
                    pages[pp, h, offs[:u]] = quantize(deq * s_old, s)
                scales[pp, h] = s
                pages[pp, h, offs[u]] = quantize(x, s)
    return kp, vp, ks, vs
