"""fp64 CPU oracle for paged grouped-query decode attention.

TEST INFRASTRUCTURE. Only the tests, the package smoke check and the bench's
CPU-baseline leg may import or call this module. The GPU library never does,
and this module imports nothing from the GPU path.

What it computes. The paper states that rollout decoding is memory-bound
(§2.4) and reads each trajectory's KV cache (§5.2) through its generation
engine (§8, "Testbed"), but never writes out the attention step. The method
is exact attention computed faster, so this oracle is the plain definition:
for trajectory b of length n, query head h (kv-head h // g with g = Hq/Hkv),
and tokens t < n read through the block table,

    s_t   = scale * <q[b, h], k_t>
    lse   = M + ln(sum_t exp(s_t - M)),   M = max_t s_t
    out   = sum_t exp(s_t - lse) * v_t

in float64. n = 0 gives out = 0 and lse = -inf.

Token t lives in physical page block_table[b, t // 16] at slot t % 16. Inside
one (page, kv-head) tile of 16 x D elements the library stores
  K element (t, d) at ((d // X) * 16 + t) * X + d % X,  X = 16 bytes / elem,
  V element (t, d) at ((t // 4) * D + d) * 4 + t % 4.
bf16 codes are the top half of an IEEE binary32; fp8 codes are OCP E4M3FN
(bias 7, subnormals down to 2^-9, max 448, 0x7F/0xFF NaN, no infinity),
multiplied by the per-(page, kv-head) fp32 scale.
"""
from __future__ import annotations

from concurrent.futures import ThreadPoolExecutor
from typing import Optional, Tuple

import numpy as np

PAGE = 16


# ---------------------------------------------------------------- decoders

def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """bf16 codes (uint16) -> float64: the code is the high half of a
    binary32 whose low half is zero."""
    b32 = bits.astype(np.uint32) << np.uint32(16)
    return b32.view(np.float32).astype(np.float64)


def _e4m3fn_value(code: int) -> float:
    sign = -1.0 if code & 0x80 else 1.0
    exp = (code >> 3) & 0xF
    man = code & 0x7
    if exp == 0xF and man == 0x7:
        return float("nan")
    if exp == 0:
        return sign * man * 2.0 ** -9          # subnormal: m/8 * 2^(1-7)
    return sign * (1.0 + man / 8.0) * 2.0 ** (exp - 7)


E4M3FN_TABLE = np.array([_e4m3fn_value(c) for c in range(256)],
                        dtype=np.float64)


def e4m3fn_bytes_to_f64(codes: np.ndarray) -> np.ndarray:
    return E4M3FN_TABLE[codes.astype(np.int64)]


# ---------------------------------------------------------- page addressing

def k_tile_offsets(head_dim: int, elem_bytes: int) -> np.ndarray:
    """[16, D] element offsets of K(t, d) inside one tile."""
    x = 16 // elem_bytes
    t = np.arange(PAGE)[:, None]
    d = np.arange(head_dim)[None, :]
    return ((d // x) * PAGE + t) * x + d % x


def v_tile_offsets(head_dim: int) -> np.ndarray:
    """[16, D] element offsets of V(t, d) inside one tile."""
    t = np.arange(PAGE)[:, None]
    d = np.arange(head_dim)[None, :]
    return ((t // 4) * head_dim + d) * 4 + t % 4


def gather_kv(k_pages, v_pages, block_table_row, n, kvh, head_dim, kv_dtype,
              k_scale=None, v_scale=None) -> Tuple[np.ndarray, np.ndarray]:
    """K and V of tokens 0..n-1 of one trajectory and kv-head, float64 [n, D]."""
    fp8 = kv_dtype == "fp8_e4m3fn"
    t = np.arange(n)
    page = block_table_row[t // PAGE].astype(np.int64)
    slot = t % PAGE
    ko = k_tile_offsets(head_dim, 1 if fp8 else 2)[slot]     # [n, D]
    vo = v_tile_offsets(head_dim)[slot]
    k_raw = k_pages[page[:, None], kvh, ko]
    v_raw = v_pages[page[:, None], kvh, vo]
    if fp8:
        k = e4m3fn_bytes_to_f64(k_raw) * k_scale[page, kvh].astype(np.float64)[:, None]
        v = e4m3fn_bytes_to_f64(v_raw) * v_scale[page, kvh].astype(np.float64)[:, None]
    else:
        k = bf16_bits_to_f64(k_raw)
        v = bf16_bits_to_f64(v_raw)
    return k, v


# -------------------------------------------------------------- definition

def attend(q_rows: np.ndarray, k: np.ndarray, v: np.ndarray,
           scale: float) -> Tuple[np.ndarray, np.ndarray]:
    """Softmax attention of query rows [g, D] over keys/values [n, D]."""
    g, d = q_rows.shape
    n = k.shape[0]
    if n == 0:
        return np.zeros((g, v.shape[1])), np.full(g, -np.inf)
    s = scale * (q_rows @ k.T)                      # [g, n]
    m = s.max(axis=1)
    lse = m + np.log(np.exp(s - m[:, None]).sum(axis=1))
    out = np.exp(s - lse[:, None]) @ v
    return out, lse


def decode_attention(q, k_pages, v_pages, block_table, seq_lens, *,
                     head_dim: int, num_kv_heads: int, kv_dtype: str,
                     softmax_scale: float, k_scale=None, v_scale=None,
                     workers: int = 1, **_unused):
    """out [B, Hq, D] and lse [B, Hq], float64.

    q: bf16 codes uint16 [B, Hq, D]; k_pages/v_pages: uint16 (bf16) or uint8
    (fp8) codes [P, Hkv, 16*D] in the library's tile order; block_table int
    [B, W]; seq_lens int [B]; k_scale/v_scale float [P, Hkv] for fp8.
    ``workers`` threads share the trajectories.
    """
    q = np.asarray(q)
    b_count, hq, d = q.shape
    assert d == head_dim and hq % num_kv_heads == 0
    g = hq // num_kv_heads
    qf = bf16_bits_to_f64(q)
    out = np.zeros((b_count, hq, d), dtype=np.float64)
    lse = np.zeros((b_count, hq), dtype=np.float64)

    def one(b):
        n = int(seq_lens[b])
        for kvh in range(num_kv_heads):
            k, v = gather_kv(k_pages, v_pages, block_table[b], n, kvh,
                             head_dim, kv_dtype, k_scale, v_scale)
            h0 = kvh * g
            o, l = attend(qf[b, h0:h0 + g], k, v, softmax_scale)
            out[b, h0:h0 + g] = o
            lse[b, h0:h0 + g] = l

    # one BLAS thread per worker: a full BLAS pool in every worker
    # oversubscribes the host and runs ~40x slower; the serial path uses one
    # too, so the result does not depend on the number of workers
    with _blas_threads(1):
        if workers <= 1:
            for b in range(b_count):
                one(b)
        else:
            with ThreadPoolExecutor(max_workers=workers) as ex:
                list(ex.map(one, range(b_count)))
    return out, lse


def _blas_threads(n: int):
    try:
        from threadpoolctl import threadpool_limits
    except ImportError:          # no control over BLAS threads: run as is
        from contextlib import nullcontext
        return nullcontext()
    return threadpool_limits(n)


def decode_attention_from_host(arrays: dict, workers: int = 1):
    """Convenience: call ``decode_attention`` on a dict of host arrays with
    the keys q, k_pages, v_pages, block_table, seq_lens, head_dim,
    num_kv_heads, kv_dtype, softmax_scale, k_scale, v_scale."""
    return decode_attention(workers=workers, **arrays)
