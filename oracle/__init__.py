"""fp64 CPU oracle for paged grouped-query decode attention.

TEST INFRASTRUCTURE: imported only by the tests, the package smoke check and
the bench's CPU-baseline leg. Never imported by the GPU library.
"""
from .decode_attention import (E4M3FN_TABLE, attend, bf16_bits_to_f64,
                               decode_attention, decode_attention_from_host,
                               e4m3fn_bytes_to_f64, gather_kv)
from .decoder import rmsnorm, silu_mul
from .kv_append import append_scale, e4m3fn_round, kv_append, quantize
