"""ctypes binding of the C ABI in include/laminar_decode_attn.h,
include/laminar_kv_append.h, include/laminar_repack.h and
include/laminar_linear.h.

Argument marshalling only: every step of the computation runs in the HIP
library. Importing this module does not touch the GPU; loading fails loudly
when the library has not been built.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import (POINTER, c_float, c_int32, c_size_t, c_void_p)

import numpy as np

from .build import LIB_PATH

LAMINAR_OK = 0
LAMINAR_ERR_INVALID_ARG = 1
LAMINAR_ERR_UNSUPPORTED = 2
LAMINAR_ERR_WORKSPACE = 3
LAMINAR_ERR_HIP = 4

LAMINAR_KV_BF16 = 0
LAMINAR_KV_FP8_E4M3FN = 1

LAMINAR_X_BF16 = 0
LAMINAR_X_F32 = 1
LAMINAR_X_SILU_MUL = 2


class LaminarAttnDesc(ctypes.Structure):
    _fields_ = [
        ("batch", c_int32),
        ("num_q_heads", c_int32),
        ("num_kv_heads", c_int32),
        ("head_dim", c_int32),
        ("page_size", c_int32),
        ("num_pages", c_int32),
        ("max_blocks_per_seq", c_int32),
        ("kv_dtype", c_int32),
        ("softmax_scale", c_float),
        ("k_scale", c_void_p),
        ("v_scale", c_void_p),
        ("pages_per_item", c_int32),
        ("waves_per_item", c_int32),
        ("input_row_stride", c_int32),
    ]


class LaminarRolloutState(ctypes.Structure):
    _fields_ = [("kv_used", ctypes.c_int64), ("kv_prev", ctypes.c_int64),
                ("num_reqs", c_int32), ("reserved", c_int32)]


class LaminarModelShape(ctypes.Structure):
    _fields_ = [(n, c_int32) for n in (
        "layers", "hidden", "q_heads", "kv_heads", "head_dim", "intermediate",
        "vocab", "weight_bytes", "act_bytes", "kv_bytes")]


class LaminarError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = int(status)
        super().__init__(f"{where}: {laminar_status_string(status)} "
                         f"(status {status})")


_LIB = None

# name -> (restype, argtypes)
_SIGNATURES = {
    "laminar_plan_create": (c_int32, [POINTER(LaminarAttnDesc), POINTER(c_int32),
                                      c_int32, POINTER(c_void_p)]),
    "laminar_plan_create_cascade": (c_int32, [POINTER(LaminarAttnDesc),
                                              POINTER(c_int32), POINTER(c_int32),
                                              c_int32, POINTER(c_int32), c_int32,
                                              POINTER(c_void_p)]),
    "laminar_plan_workspace_bytes": (c_size_t, [c_void_p]),
    "laminar_plan_bind_workspace": (c_int32, [c_void_p, c_void_p, c_size_t,
                                              c_void_p]),
    "laminar_decode_attn": (c_int32, [c_void_p] + [c_void_p] * 7 + [c_void_p]),
    "laminar_decode_attn_partial": (c_int32, [c_void_p] + [c_void_p] * 7
                                    + [c_void_p]),
    "laminar_decode_attn_merge": (c_int32, [c_void_p, c_void_p, c_void_p,
                                            c_void_p]),
    "laminar_decode_attn_static": (c_int32, [c_void_p] + [c_void_p] * 7
                                   + [c_void_p]),
    "laminar_plan_num_items": (c_int32, [c_void_p]),
    "laminar_plan_num_merges": (c_int32, [c_void_p]),
    "laminar_plan_pages_per_item": (c_int32, [c_void_p]),
    "laminar_plan_waves_per_item": (c_int32, [c_void_p]),
    "laminar_plan_items_copy": (c_int32, [c_void_p, POINTER(c_int32), c_int32]),
    "laminar_plan_merges_copy": (c_int32, [c_void_p, POINTER(c_int32), c_int32]),
    "laminar_plan_num_dynamic_items": (c_int32, [c_void_p]),
    "laminar_plan_num_cascade_units": (c_int32, [c_void_p]),
    "laminar_plan_num_cascade_members": (c_int32, [c_void_p]),
    "laminar_plan_cascade_units_copy": (c_int32, [c_void_p, POINTER(c_int32),
                                                  c_int32]),
    "laminar_plan_cascade_members_copy": (c_int32, [c_void_p, POINTER(c_int32),
                                                    c_int32]),
    "laminar_plan_destroy": (None, [c_void_p]),
    "laminar_status_string": (ctypes.c_char_p, [c_int32]),
    "laminar_hbm_read_sink_floats": (c_int32, []),
    "laminar_hbm_read": (c_int32, [c_void_p, c_size_t, c_void_p, c_void_p]),
    "laminar_hbm_copy": (c_int32, [c_void_p, c_void_p, c_size_t, c_void_p]),
    "laminar_hbm_gather_sink_words": (c_int32, [ctypes.c_int64, c_size_t]),
    "laminar_hbm_gather": (c_int32, [c_void_p, c_size_t, c_size_t, c_void_p,
                                     ctypes.c_int64, c_void_p, c_void_p]),
    "laminar_kv_append": (c_int32, [POINTER(LaminarAttnDesc)] + [c_void_p] * 8
                          + [c_void_p]),
    "laminar_kv_pack": (c_int32, [c_void_p, c_void_p, ctypes.c_int64, c_int32,
                                  c_int32, c_int32, c_void_p]),
    "laminar_repack_plan": (c_int32, [POINTER(LaminarRolloutState), c_int32,
                                      ctypes.c_int64, c_int32, POINTER(c_int32),
                                      POINTER(c_int32), POINTER(c_int32)]),
    "laminar_migration_pairs": (c_int32, [POINTER(c_int32), POINTER(c_int32),
                                          c_int32, c_int32, POINTER(c_int32),
                                          c_int32, POINTER(c_int32), c_int32,
                                          POINTER(c_int32), c_int32,
                                          POINTER(c_int32), POINTER(c_int32)]),
    "laminar_roofline_batch_bound": (c_int32, [POINTER(LaminarModelShape),
                                               ctypes.c_uint64, ctypes.c_uint64,
                                               POINTER(c_int32)]),
    "laminar_roofline_step_seconds": (c_int32, [POINTER(LaminarModelShape),
                                                ctypes.c_int64, ctypes.c_int64,
                                                ctypes.c_uint64, ctypes.c_uint64,
                                                POINTER(ctypes.c_double)]),
    "laminar_linear_pack": (c_int32, [c_void_p, c_void_p, c_int32, c_int32,
                                      c_void_p]),
    "laminar_linear_bf16": (c_int32, [c_void_p, c_void_p, c_void_p, c_void_p,
                                      c_int32, c_int32, c_int32, c_void_p,
                                      c_size_t, c_void_p]),
    "laminar_linear_bf16_kv_append": (c_int32, [c_void_p, c_int32, c_void_p,
                                                c_void_p, c_int32, c_int32,
                                                c_int32, c_void_p, c_size_t,
                                                POINTER(LaminarAttnDesc),
                                                c_int32, c_int32]
                                      + [c_void_p] * 7),
    "laminar_linear_bf16_ex": (c_int32, [c_void_p, c_int32, c_void_p,
                                         c_void_p, c_void_p, c_int32, c_int32,
                                         c_int32, c_void_p, c_size_t,
                                         c_void_p]),
    "laminar_linear_bf16_norm": (c_int32, [c_void_p, c_int32, c_void_p,
                                           c_void_p, c_void_p, c_void_p,
                                           ctypes.c_float, c_void_p, c_int32,
                                           c_int32, c_int32, c_void_p,
                                           c_size_t, c_void_p]),
    "laminar_linear_bf16_swiglu": (c_int32, [c_void_p, c_int32, c_void_p,
                                             c_void_p, c_void_p, c_int32,
                                             c_int32, c_int32, c_void_p,
                                             c_size_t, c_void_p]),
    "laminar_linear_bf16_rmsnorm": (c_int32, [c_void_p, c_void_p,
                                              ctypes.c_float, c_void_p,
                                              c_void_p, c_void_p, c_int32,
                                              c_int32, c_int32, c_void_p,
                                              c_size_t, c_void_p]),
    "laminar_rmsnorm": (c_int32, [c_void_p, c_void_p, c_void_p, c_int32,
                                  c_int32, ctypes.c_float, c_void_p]),
    "laminar_silu_mul": (c_int32, [c_void_p, c_void_p, c_int32, c_int32,
                                   c_void_p]),
    "laminar_linear_splits": (c_int32, [c_int32, c_int32, c_int32]),
    "laminar_linear_workspace_bytes": (c_size_t, [c_int32, c_int32, c_int32]),
    "laminar_linear": (c_int32, [c_void_p, c_void_p, c_void_p, c_int32, c_int32,
                                 c_int32, c_void_p, c_size_t, c_void_p]),
    "laminar_migrate_pages": (c_int32, [c_void_p, ctypes.c_int64, c_void_p,
                                        ctypes.c_int64, c_size_t, c_void_p,
                                        c_int32, c_void_p]),
}


def library_path() -> str:
    return os.environ.get("LAMINAR_LIB", LIB_PATH)


def lib() -> ctypes.CDLL:
    """The loaded HIP library; raises if it has not been built."""
    global _LIB
    if _LIB is None:
        path = library_path()
        if not os.path.exists(path):
            raise RuntimeError(
                f"HIP library {path} is missing: build it with "
                "`python -m paper_2510_12633_amd.build` (no CPU fallback)")
        handle = ctypes.CDLL(path)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _LIB = handle
    return _LIB


def _ptr(x):
    """Device or host address of a tensor / integer / None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if hasattr(x, "data_ptr"):
        return x.data_ptr()
    raise TypeError(f"cannot take the address of {type(x).__name__}")


def _check(status: int, where: str):
    if status != LAMINAR_OK:
        raise LaminarError(status, where)


def laminar_status_string(status: int) -> str:
    return lib().laminar_status_string(int(status)).decode()


def laminar_plan_create(desc: LaminarAttnDesc, seq_lens_host, num_cus: int):
    lens = np.ascontiguousarray(seq_lens_host, dtype=np.int32)
    out = c_void_p()
    st = lib().laminar_plan_create(
        ctypes.byref(desc), lens.ctypes.data_as(POINTER(c_int32)),
        int(num_cus), ctypes.byref(out))
    _check(st, "laminar_plan_create")
    return out.value


def laminar_plan_create_cascade(desc: LaminarAttnDesc, seq_lens_host,
                                group_of_host, group_pages_host, num_cus: int):
    lens = np.ascontiguousarray(seq_lens_host, dtype=np.int32)
    grp = np.ascontiguousarray(group_of_host, dtype=np.int32)
    pages = np.ascontiguousarray(group_pages_host, dtype=np.int32)
    out = c_void_p()
    st = lib().laminar_plan_create_cascade(
        ctypes.byref(desc), lens.ctypes.data_as(POINTER(c_int32)),
        grp.ctypes.data_as(POINTER(c_int32)), int(pages.size),
        pages.ctypes.data_as(POINTER(c_int32)), int(num_cus), ctypes.byref(out))
    _check(st, "laminar_plan_create_cascade")
    return out.value


def laminar_plan_workspace_bytes(plan) -> int:
    return int(lib().laminar_plan_workspace_bytes(plan))


def laminar_plan_bind_workspace(plan, workspace, nbytes: int, stream):
    _check(lib().laminar_plan_bind_workspace(plan, _ptr(workspace), int(nbytes),
                                             _ptr(stream)),
           "laminar_plan_bind_workspace")


def laminar_decode_attn(plan, q, k_pages, v_pages, block_table, seq_lens, out,
                        lse, stream):
    _check(lib().laminar_decode_attn(
        plan, _ptr(q), _ptr(k_pages), _ptr(v_pages), _ptr(block_table),
        _ptr(seq_lens), _ptr(out), _ptr(lse), _ptr(stream)),
        "laminar_decode_attn")


def laminar_decode_attn_partial(plan, q, k_pages, v_pages, block_table,
                                seq_lens, out, lse, stream):
    _check(lib().laminar_decode_attn_partial(
        plan, _ptr(q), _ptr(k_pages), _ptr(v_pages), _ptr(block_table),
        _ptr(seq_lens), _ptr(out), _ptr(lse), _ptr(stream)),
        "laminar_decode_attn_partial")


def laminar_decode_attn_merge(plan, out, lse, stream):
    _check(lib().laminar_decode_attn_merge(plan, _ptr(out), _ptr(lse),
                                           _ptr(stream)),
           "laminar_decode_attn_merge")


def laminar_decode_attn_static(plan, q, k_pages, v_pages, block_table,
                               seq_lens, out, lse, stream):
    _check(lib().laminar_decode_attn_static(
        plan, _ptr(q), _ptr(k_pages), _ptr(v_pages), _ptr(block_table),
        _ptr(seq_lens), _ptr(out), _ptr(lse), _ptr(stream)),
        "laminar_decode_attn_static")


def laminar_plan_num_items(plan) -> int:
    return int(lib().laminar_plan_num_items(plan))


def laminar_plan_num_merges(plan) -> int:
    return int(lib().laminar_plan_num_merges(plan))


def laminar_plan_pages_per_item(plan) -> int:
    return int(lib().laminar_plan_pages_per_item(plan))


def laminar_plan_waves_per_item(plan) -> int:
    return int(lib().laminar_plan_waves_per_item(plan))


def laminar_plan_items_copy(plan) -> np.ndarray:
    n = laminar_plan_num_items(plan)
    buf = np.zeros((max(n, 0), 4), dtype=np.int32)
    got = lib().laminar_plan_items_copy(
        plan, buf.ctypes.data_as(POINTER(c_int32)), n)
    assert got == n
    return buf


def laminar_plan_merges_copy(plan) -> np.ndarray:
    n = laminar_plan_num_merges(plan)
    buf = np.zeros((max(n, 0), 4), dtype=np.int32)
    got = lib().laminar_plan_merges_copy(
        plan, buf.ctypes.data_as(POINTER(c_int32)), n)
    assert got == n
    return buf


def laminar_plan_cascade_units_copy(plan) -> np.ndarray:
    n = int(lib().laminar_plan_num_cascade_units(plan))
    buf = np.zeros((max(n, 0), 4), dtype=np.int32)
    got = lib().laminar_plan_cascade_units_copy(
        plan, buf.ctypes.data_as(POINTER(c_int32)), n)
    assert got == n
    return buf


def laminar_plan_cascade_members_copy(plan) -> np.ndarray:
    n = int(lib().laminar_plan_num_cascade_members(plan))
    buf = np.zeros((max(n, 0), 2), dtype=np.int32)
    got = lib().laminar_plan_cascade_members_copy(
        plan, buf.ctypes.data_as(POINTER(c_int32)), n)
    assert got == n
    return buf


def laminar_plan_destroy(plan):
    lib().laminar_plan_destroy(plan)


def laminar_kv_append(desc: LaminarAttnDesc, k_new, v_new, block_table,
                      seq_lens, k_pages, v_pages, k_scale, v_scale, stream):
    _check(lib().laminar_kv_append(
        ctypes.byref(desc), _ptr(k_new), _ptr(v_new), _ptr(block_table),
        _ptr(seq_lens), _ptr(k_pages), _ptr(v_pages), _ptr(k_scale),
        _ptr(v_scale), _ptr(stream)), "laminar_kv_append")


def _i32p(a):
    return a.ctypes.data_as(POINTER(c_int32))


def laminar_repack_plan(kv_used, kv_prev, num_reqs, kv_max: int,
                        batch_max: int):
    """(source, destination) rollout pairs of the consolidation plan."""
    n = len(kv_used)
    states = (LaminarRolloutState * max(n, 1))()
    for i in range(n):
        states[i].kv_used = int(kv_used[i])
        states[i].kv_prev = int(kv_prev[i])
        states[i].num_reqs = int(num_reqs[i])
    src = np.zeros(max(n, 1), np.int32)
    dst = np.zeros(max(n, 1), np.int32)
    k = c_int32(0)
    _check(lib().laminar_repack_plan(states, n, int(kv_max), int(batch_max),
                                     _i32p(src), _i32p(dst), ctypes.byref(k)),
           "laminar_repack_plan")
    return [(int(a), int(b)) for a, b in zip(src[:k.value], dst[:k.value])]


def laminar_roofline_batch_bound(shape: LaminarModelShape, peak_flops: int,
                                 peak_bw: int) -> int:
    """Roofline batch bound B (0: no batch is compute-bound)."""
    out = c_int32()
    _check(lib().laminar_roofline_batch_bound(ctypes.byref(shape),
                                              int(peak_flops), int(peak_bw),
                                              ctypes.byref(out)),
           "laminar_roofline_batch_bound")
    return out.value


def laminar_roofline_step_seconds(shape: LaminarModelShape, batch: int,
                                  context: int, peak_flops: int,
                                  peak_bw: int) -> float:
    out = ctypes.c_double()
    _check(lib().laminar_roofline_step_seconds(
        ctypes.byref(shape), int(batch), int(context), int(peak_flops),
        int(peak_bw), ctypes.byref(out)), "laminar_roofline_step_seconds")
    return out.value


def laminar_migration_pairs(src_table, lens, dst_free, dst_width: int):
    """(dst_table [n, dst_width], pairs [k, 2], free pages used)."""
    src_table = np.ascontiguousarray(src_table, dtype=np.int32)
    lens = np.ascontiguousarray(lens, dtype=np.int32)
    dst_free = np.ascontiguousarray(dst_free, dtype=np.int32)
    n, width = src_table.shape
    dst_table = np.full((n, dst_width), -1, np.int32)
    cap = int(np.sum((lens.astype(np.int64) + 15) // 16))
    pairs = np.zeros((max(cap, 1), 2), np.int32)
    k, used = c_int32(0), c_int32(0)
    _check(lib().laminar_migration_pairs(
        _i32p(src_table), _i32p(lens), n, width, _i32p(dst_free),
        dst_free.size, _i32p(dst_table), dst_width, _i32p(pairs), cap,
        ctypes.byref(k), ctypes.byref(used)), "laminar_migration_pairs")
    return dst_table, pairs[:k.value].copy(), used.value


def laminar_migrate_pages(src_pool, src_pages: int, dst_pool, dst_pages: int,
                          page_bytes: int, pairs, num_pairs: int, stream):
    _check(lib().laminar_migrate_pages(
        _ptr(src_pool), int(src_pages), _ptr(dst_pool), int(dst_pages),
        int(page_bytes), _ptr(pairs), int(num_pairs), _ptr(stream)),
        "laminar_migrate_pages")


def laminar_linear_pack(w, w_packed, n: int, k: int, stream):
    _check(lib().laminar_linear_pack(_ptr(w), _ptr(w_packed), int(n), int(k),
                                     _ptr(stream)), "laminar_linear_pack")


def laminar_linear_splits(m: int, n: int, k: int) -> int:
    return int(lib().laminar_linear_splits(int(m), int(n), int(k)))


def laminar_linear_workspace_bytes(m: int, n: int, k: int) -> int:
    return int(lib().laminar_linear_workspace_bytes(int(m), int(n), int(k)))


def laminar_linear(x, w_packed, y, m: int, n: int, k: int, workspace,
                   workspace_bytes: int, stream):
    _check(lib().laminar_linear(_ptr(x), _ptr(w_packed), _ptr(y), int(m), int(n),
                                int(k), _ptr(workspace), int(workspace_bytes),
                                _ptr(stream)), "laminar_linear")


def laminar_linear_bf16(x, w_packed, y, residual, m: int, n: int, k: int,
                        workspace, workspace_bytes: int, stream):
    _check(lib().laminar_linear_bf16(_ptr(x), _ptr(w_packed), _ptr(y),
                                     _ptr(residual), int(m), int(n), int(k),
                                     _ptr(workspace), int(workspace_bytes),
                                     _ptr(stream)), "laminar_linear_bf16")


def laminar_linear_bf16_ex(x, x_kind: int, w_packed, y, residual, m: int,
                           n: int, k: int, workspace, workspace_bytes: int,
                           stream):
    _check(lib().laminar_linear_bf16_ex(_ptr(x), int(x_kind), _ptr(w_packed),
                                        _ptr(y), _ptr(residual), int(m),
                                        int(n), int(k), _ptr(workspace),
                                        int(workspace_bytes), _ptr(stream)),
           "laminar_linear_bf16_ex")


def laminar_linear_bf16_norm(x, x_kind: int, w_packed, y, residual,
                             norm_weight, eps: float, y_norm, m: int, n: int,
                             k: int, workspace, workspace_bytes: int, stream):
    _check(lib().laminar_linear_bf16_norm(
        _ptr(x), int(x_kind), _ptr(w_packed), _ptr(y), _ptr(residual),
        _ptr(norm_weight), float(eps), _ptr(y_norm), int(m), int(n), int(k),
        _ptr(workspace), int(workspace_bytes), _ptr(stream)),
        "laminar_linear_bf16_norm")


def laminar_linear_bf16_kv_append(x, x_kind: int, w_packed, y, m: int, n: int,
                                  k: int, workspace, workspace_bytes: int,
                                  kv_desc: LaminarAttnDesc, k_col: int,
                                  v_col: int, block_table, seq_lens, k_pages,
                                  v_pages, k_scale, v_scale, stream):
    _check(lib().laminar_linear_bf16_kv_append(
        _ptr(x), int(x_kind), _ptr(w_packed), _ptr(y), int(m), int(n), int(k),
        _ptr(workspace), int(workspace_bytes), ctypes.byref(kv_desc),
        int(k_col), int(v_col), _ptr(block_table), _ptr(seq_lens),
        _ptr(k_pages), _ptr(v_pages), _ptr(k_scale), _ptr(v_scale),
        _ptr(stream)), "laminar_linear_bf16_kv_append")


def laminar_linear_bf16_swiglu(x, x_kind: int, w_packed, y, y_act, m: int,
                               n: int, k: int, workspace, workspace_bytes: int,
                               stream):
    _check(lib().laminar_linear_bf16_swiglu(
        _ptr(x), int(x_kind), _ptr(w_packed), _ptr(y), _ptr(y_act), int(m),
        int(n), int(k), _ptr(workspace), int(workspace_bytes), _ptr(stream)),
        "laminar_linear_bf16_swiglu")


def laminar_linear_bf16_rmsnorm(x, norm_weight, eps: float, w_packed, y,
                                residual, m: int, n: int, k: int, workspace,
                                workspace_bytes: int, stream):
    _check(lib().laminar_linear_bf16_rmsnorm(
        _ptr(x), _ptr(norm_weight), float(eps), _ptr(w_packed), _ptr(y),
        _ptr(residual), int(m), int(n), int(k), _ptr(workspace),
        int(workspace_bytes), _ptr(stream)), "laminar_linear_bf16_rmsnorm")


def laminar_rmsnorm(x, weight, y, m: int, n: int, eps: float, stream):
    _check(lib().laminar_rmsnorm(_ptr(x), _ptr(weight), _ptr(y), int(m), int(n),
                                 float(eps), _ptr(stream)), "laminar_rmsnorm")


def laminar_silu_mul(gu, y, m: int, inter: int, stream):
    _check(lib().laminar_silu_mul(_ptr(gu), _ptr(y), int(m), int(inter),
                                  _ptr(stream)), "laminar_silu_mul")


def laminar_hbm_read_sink_floats() -> int:
    return int(lib().laminar_hbm_read_sink_floats())


def laminar_hbm_read(src, nbytes: int, sink, stream):
    _check(lib().laminar_hbm_read(_ptr(src), int(nbytes), _ptr(sink),
                                  _ptr(stream)), "laminar_hbm_read")


def laminar_hbm_copy(dst, src, nbytes: int, stream):
    _check(lib().laminar_hbm_copy(_ptr(dst), _ptr(src), int(nbytes),
                                  _ptr(stream)), "laminar_hbm_copy")


def laminar_hbm_gather_sink_words(n_idx: int, tile_bytes: int) -> int:
    return int(lib().laminar_hbm_gather_sink_words(int(n_idx), int(tile_bytes)))


def laminar_hbm_gather(src, src_bytes: int, tile_bytes: int, idx, n_idx: int,
                       sink, stream):
    _check(lib().laminar_hbm_gather(_ptr(src), int(src_bytes), int(tile_bytes),
                                    _ptr(idx), int(n_idx), _ptr(sink),
                                    _ptr(stream)), "laminar_hbm_gather")


def laminar_kv_pack(src, dst, num_tiles: int, head_dim: int, kv_dtype: int,
                    which: int, stream):
    _check(lib().laminar_kv_pack(_ptr(src), _ptr(dst), int(num_tiles),
                                 int(head_dim), int(kv_dtype), int(which),
                                 _ptr(stream)), "laminar_kv_pack")
