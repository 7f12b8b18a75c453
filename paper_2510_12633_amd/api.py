"""Owner object for one decode step's plan and workspace.

Holds the plan handle and a torch-allocated device workspace and forwards
calls to the C ABI. Argument marshalling and resource ownership only.
"""
from __future__ import annotations

from typing import Optional

import numpy as np
import torch

from . import _native as N

KV_DTYPES = {"bf16": N.LAMINAR_KV_BF16, "fp8_e4m3fn": N.LAMINAR_KV_FP8_E4M3FN}


def _stream_handle(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def num_cus(device=None) -> int:
    return torch.cuda.get_device_properties(
        device if device is not None else torch.cuda.current_device()
    ).multi_processor_count


class PagedDecodeAttention:
    """Plan + bound workspace for a batch with fixed trajectory lengths.

    ``seq_lens_host`` are the lengths the next calls will see. The plan is
    reusable by every layer of the decode step. With ``group_of`` (group
    index per trajectory, -1 for none) and ``group_pages`` (shared prefix
    pages per group) the plan decodes each group's shared pages once.
    """

    def __init__(self, *, batch: int, num_q_heads: int, num_kv_heads: int,
                 head_dim: int, num_pages: int, max_blocks_per_seq: int,
                 seq_lens_host, softmax_scale: float, kv_dtype: str = "bf16",
                 k_scale: Optional[torch.Tensor] = None,
                 v_scale: Optional[torch.Tensor] = None,
                 pages_per_item: int = 0, waves_per_item: int = 0,
                 cus: Optional[int] = None, device="cuda", stream=None,
                 group_of=None, group_pages=None, q_row_stride: int = 0):
        self.desc = N.LaminarAttnDesc(
            batch=batch, num_q_heads=num_q_heads, num_kv_heads=num_kv_heads,
            head_dim=head_dim, page_size=16, num_pages=num_pages,
            max_blocks_per_seq=max_blocks_per_seq,
            kv_dtype=KV_DTYPES[kv_dtype], softmax_scale=softmax_scale,
            k_scale=None if k_scale is None else k_scale.data_ptr(),
            v_scale=None if v_scale is None else v_scale.data_ptr(),
            pages_per_item=pages_per_item, waves_per_item=waves_per_item,
            input_row_stride=q_row_stride)
        self.device = torch.device(device)
        self.q_strides = (q_row_stride or num_q_heads * head_dim, head_dim, 1)
        self._scales = (k_scale, v_scale)        # keep alive
        if cus is None:
            cus = num_cus(self.device) if self.device.type == "cuda" else 256
        if group_of is None:
            self.plan = N.laminar_plan_create(self.desc,
                                              np.asarray(seq_lens_host), cus)
        else:
            self.plan = N.laminar_plan_create_cascade(
                self.desc, np.asarray(seq_lens_host), group_of, group_pages,
                cus)
        self.workspace_bytes = N.laminar_plan_workspace_bytes(self.plan)
        self.workspace = None
        if self.device.type == "cuda":
            self.bind(stream)

    def bind(self, stream=None):
        nbytes = max(self.workspace_bytes, 256)
        self.workspace = torch.empty(nbytes, dtype=torch.uint8,
                                     device=self.device)
        self._bind_stream = stream
        N.laminar_plan_bind_workspace(self.plan, self.workspace,
                                      self.workspace_bytes,
                                      _stream_handle(stream))

    def outputs(self, fill: Optional[float] = float("nan")):
        """New out [B, Hq, D] and lse [B, Hq] fp32 buffers, filled with
        ``fill`` (NaN by default, so that a row the kernels leave unwritten
        shows up instead of passing as a stale value; None leaves them
        uninitialised)."""
        d = self.desc
        shape_o = (d.batch, d.num_q_heads, d.head_dim)
        shape_l = (d.batch, d.num_q_heads)
        if fill is None:
            return (torch.empty(shape_o, dtype=torch.float32, device=self.device),
                    torch.empty(shape_l, dtype=torch.float32, device=self.device))
        return (torch.full(shape_o, fill, dtype=torch.float32, device=self.device),
                torch.full(shape_l, fill, dtype=torch.float32, device=self.device))

    def __call__(self, q, k_pages, v_pages, block_table, seq_lens, out=None,
                 lse=None, stream=None):
        if out is None or lse is None:
            out, lse = self.outputs()
        self._check_q(q)
        N.laminar_decode_attn(self.plan, q, k_pages, v_pages, block_table,
                              seq_lens, out, lse, _stream_handle(stream))
        return out, lse

    def _check_q(self, q):
        if q.shape[0] > 1 and tuple(q.stride()) != self.q_strides:
            raise ValueError(f"q strides {tuple(q.stride())} differ from the "
                             f"plan's {self.q_strides}")

    def partial(self, q, k_pages, v_pages, block_table, seq_lens, out, lse,
                stream=None):
        self._check_q(q)
        N.laminar_decode_attn_partial(self.plan, q, k_pages, v_pages,
                                      block_table, seq_lens, out, lse,
                                      _stream_handle(stream))

    def merge(self, out, lse, stream=None):
        N.laminar_decode_attn_merge(self.plan, out, lse, _stream_handle(stream))

    @property
    def num_items(self) -> int:
        return N.laminar_plan_num_items(self.plan)

    @property
    def num_merges(self) -> int:
        return N.laminar_plan_num_merges(self.plan)

    @property
    def pages_per_item(self) -> int:
        return N.laminar_plan_pages_per_item(self.plan)

    @property
    def waves_per_item(self) -> int:
        return N.laminar_plan_waves_per_item(self.plan)

    def items(self) -> np.ndarray:
        return N.laminar_plan_items_copy(self.plan)

    def merges(self) -> np.ndarray:
        return N.laminar_plan_merges_copy(self.plan)

    def close(self):
        """Destroy the plan once the stream has passed the table upload."""
        if getattr(self, "plan", None):
            if self.workspace is not None:
                torch.cuda.current_stream(self.device).synchronize() \
                    if self._bind_stream is None else self._bind_stream.synchronize()
            N.laminar_plan_destroy(self.plan)
            self.plan = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def kv_append(k_new, v_new, block_table, seq_lens, k_pages, v_pages,
              k_scale=None, v_scale=None, *, kv_dtype: str = "bf16",
              stream=None):
    """Append the current token's K/V ([B, Hkv, D] bf16) to the paged pools
    in place (pools [P, Hkv, 16*D]; fp8 scales [P, Hkv] updated too)."""
    b, hkv, d = k_new.shape
    # rows may be strided (views into a fused QKV output); heads and dims not
    if (k_new.stride()[1:] != (d, 1) or v_new.stride()[1:] != (d, 1)
            or k_new.stride(0) != v_new.stride(0)):
        raise ValueError("k_new and v_new need contiguous [heads, dim] rows "
                         "and one row stride")
    row = k_new.stride(0)
    desc = kv_append_desc(b, hkv, d, k_pages.shape[0], block_table.shape[1],
                          kv_dtype, input_row_stride=0 if row == hkv * d else row)
    N.laminar_kv_append(desc, k_new, v_new, block_table, seq_lens, k_pages,
                        v_pages, k_scale, v_scale, _stream_handle(stream))


def kv_append_desc(batch: int, num_kv_heads: int, head_dim: int,
                   num_pages: int, max_blocks: int, kv_dtype: str = "bf16",
                   input_row_stride: int = 0):
    """The description laminar_kv_append (and the projection that makes the
    append, SkinnyLinear.bf16_kv_append) reads: pools of num_pages pages of
    16 tokens, a block table of max_blocks entries per trajectory."""
    return N.LaminarAttnDesc(
        batch=batch, num_q_heads=num_kv_heads, num_kv_heads=num_kv_heads,
        head_dim=head_dim, page_size=16, num_pages=num_pages,
        max_blocks_per_seq=max_blocks, kv_dtype=KV_DTYPES[kv_dtype],
        softmax_scale=1.0, k_scale=None, v_scale=None, pages_per_item=0,
        waves_per_item=0, input_row_stride=input_row_stride)


def migrate(src_pools, dst_pools, pairs, stream=None):
    """Copy the pages listed in ``pairs`` (device int32 [n, 2]: source page,
    destination page) between matching pools of two rollouts, e.g.
    (k_pages, v_pages) or (k_pages, v_pages, k_scale, v_scale)."""
    n = int(pairs.shape[0])
    for s, d in zip(src_pools, dst_pools):
        if s is None:
            continue
        page_bytes = s[0].numel() * s.element_size()
        N.laminar_migrate_pages(s, s.shape[0], d, d.shape[0], page_bytes,
                                pairs, n, _stream_handle(stream))


class SkinnyLinear:
    """y = x w^T for decode batches (M <= 128): w [N, K] bf16 on the device is
    packed once into the kernel's tiled layout (a copy of the same size);
    owns that copy and the K-split workspace for up to max_m rows."""

    def __init__(self, weight, max_m: int = 128, stream=None):
        self.n, self.k = weight.shape
        self.w_packed = torch.empty_like(weight)
        N.laminar_linear_pack(weight, self.w_packed, self.n, self.k,
                              _stream_handle(stream))
        self.ws_bytes = max(N.laminar_linear_workspace_bytes(m, self.n, self.k)
                            for m in range(1, max_m + 1))
        # zeroed once: the K split's group counters start at zero and every
        # call leaves them there
        self.ws = (torch.zeros(self.ws_bytes, dtype=torch.uint8,
                               device=weight.device) if self.ws_bytes else None)

    def __call__(self, x, out=None, stream=None):
        m = x.shape[0]
        if out is None:
            out = torch.empty((m, self.n), dtype=torch.float32, device=x.device)
        N.laminar_linear(x, self.w_packed, out, m, self.n, self.k, self.ws,
                         self.ws_bytes, _stream_handle(stream))
        return out

    def bf16(self, x, out=None, residual=None, swiglu=False, norm_weight=None,
             eps: float = 1e-6, stream=None):
        """bf16(x w^T + residual) [M, N]; out may be the residual itself.
        fp32 x [M, K] is rounded to bf16 on load; with swiglu, x [M, 2K]
        bf16 holds gate then up and the operand is silu(gate) * up; with
        norm_weight [K] bf16 (at most 8 rows), the operand is
        rmsnorm(x, norm_weight, eps). Each equals the separate cast,
        laminar_silu_mul or laminar_rmsnorm followed by this call, bit for
        bit, in one launch."""
        m = x.shape[0]
        if norm_weight is not None:
            if (x.dtype != torch.bfloat16 or x.shape[1] != self.k or swiglu
                    or not x.is_contiguous()):
                raise ValueError(f"x must be contiguous bf16 [M, {self.k}] "
                                 "for the norm")
            if (norm_weight.dtype != torch.bfloat16
                    or tuple(norm_weight.shape) != (self.k,)
                    or not norm_weight.is_contiguous()):
                raise ValueError(f"norm_weight must be contiguous bf16 [{self.k}]")
            if out is None:
                out = torch.empty((m, self.n), dtype=torch.bfloat16,
                                  device=x.device)
            N.laminar_linear_bf16_rmsnorm(x, norm_weight, eps, self.w_packed,
                                          out, residual, m, self.n, self.k,
                                          self.ws, self.ws_bytes,
                                          _stream_handle(stream))
            return out
        if swiglu:
            kind = N.LAMINAR_X_SILU_MUL
            want = (torch.bfloat16, 2 * self.k)
        elif x.dtype == torch.float32:
            kind, want = N.LAMINAR_X_F32, (torch.float32, self.k)
        else:
            kind, want = N.LAMINAR_X_BF16, (torch.bfloat16, self.k)
        if (x.dtype, x.shape[1]) != want or not x.is_contiguous():
            raise ValueError(f"x must be contiguous {want[0]} [M, {want[1]}]")
        if out is None:
            out = torch.empty((m, self.n), dtype=torch.bfloat16, device=x.device)
        N.laminar_linear_bf16_ex(x, kind, self.w_packed, out, residual, m,
                                 self.n, self.k, self.ws, self.ws_bytes,
                                 _stream_handle(stream))
        return out

    def _kind(self, x, swiglu):
        if swiglu:
            kind, want = N.LAMINAR_X_SILU_MUL, (torch.bfloat16, 2 * self.k)
        elif x.dtype == torch.float32:
            kind, want = N.LAMINAR_X_F32, (torch.float32, self.k)
        else:
            kind, want = N.LAMINAR_X_BF16, (torch.bfloat16, self.k)
        if (x.dtype, x.shape[1]) != want or not x.is_contiguous():
            raise ValueError(f"x must be contiguous {want[0]} [M, {want[1]}]")
        return kind

    def bf16_norm(self, x, norm_weight, eps: float = 1e-6, out=None,
                  residual=None, out_norm=None, swiglu=False, stream=None):
        """(y, rmsnorm(y, norm_weight, eps)) with y = bf16(x w^T + residual)
        as bf16() computes it (x may be fp32 or, with swiglu, gate and up);
        the norm equals laminar_rmsnorm on y bit for bit and, where K is
        split (from 33 rows), comes from the same reduction launch."""
        m = x.shape[0]
        kind = self._kind(x, swiglu)
        if out is None:
            out = torch.empty((m, self.n), dtype=torch.bfloat16, device=x.device)
        if out_norm is None:
            out_norm = torch.empty((m, self.n), dtype=torch.bfloat16,
                                   device=x.device)
        N.laminar_linear_bf16_norm(x, kind, self.w_packed, out, residual,
                                   norm_weight, eps, out_norm, m, self.n,
                                   self.k, self.ws, self.ws_bytes,
                                   _stream_handle(stream))
        return out, out_norm

    def bf16_swiglu(self, x, out=None, out_act=None, stream=None):
        """(y, silu(y[:, :N/2]) * y[:, N/2:]) with y = bf16(x w^T); the
        second equals laminar_silu_mul on y bit for bit and, with the
        balanced split, comes from the same reduction launch."""
        m = x.shape[0]
        kind = self._kind(x, False)
        if out is None:
            out = torch.empty((m, self.n), dtype=torch.bfloat16, device=x.device)
        if out_act is None:
            out_act = torch.empty((m, self.n // 2), dtype=torch.bfloat16,
                                  device=x.device)
        N.laminar_linear_bf16_swiglu(x, kind, self.w_packed, out, out_act, m,
                                     self.n, self.k, self.ws, self.ws_bytes,
                                     _stream_handle(stream))
        return out, out_act

    def bf16_kv_append(self, x, kv_desc, k_col: int, v_col: int, block_table,
                       seq_lens, k_pages, v_pages, k_scale=None, v_scale=None,
                       out=None, swiglu=False, stream=None):
        """y = bf16(x w^T) as bf16() computes it, then the decode step's KV
        append of row m's new token (columns [k_col, k_col + Hkv D) and
        [v_col, ...) of y) into the pools, exactly laminar_kv_append on y;
        from 33 rows on bf16 pools the split's reduction launch stores them.
        kv_desc is a LaminarAttnDesc with batch = M."""
        m = x.shape[0]
        kind = self._kind(x, swiglu)
        if out is None:
            out = torch.empty((m, self.n), dtype=torch.bfloat16, device=x.device)
        N.laminar_linear_bf16_kv_append(
            x, kind, self.w_packed, out, m, self.n, self.k, self.ws,
            self.ws_bytes, kv_desc, k_col, v_col, block_table, seq_lens,
            k_pages, v_pages, k_scale, v_scale, _stream_handle(stream))
        return out


def rmsnorm(x, weight=None, eps: float = 1e-6, out=None, stream=None):
    """Row-wise RMS norm of bf16 x [M, N] (times weight [N]) -> bf16."""
    m, n = x.shape
    if out is None:
        out = torch.empty_like(x)
    N.laminar_rmsnorm(x, weight, out, m, n, eps, _stream_handle(stream))
    return out


def silu_mul(gu, out=None, stream=None):
    """silu(gate) * up for bf16 gu [M, 2I] (gate then up) -> bf16 [M, I]."""
    m, two_i = gu.shape
    if out is None:
        out = torch.empty((m, two_i // 2), dtype=gu.dtype, device=gu.device)
    N.laminar_silu_mul(gu, out, m, two_i // 2, _stream_handle(stream))
    return out
