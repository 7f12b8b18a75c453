"""Seeded synthetic inputs for paged decode attention.

This module is shared by the fp64 oracle's tests and by the GPU path's tests
and bench: it draws lengths, queries and KV values and lays them out in the
library's page format. It performs none of the attention arithmetic.

Readings of the workload text (the paper gives no attention inputs):
  * values are N(0, 1); q is rounded to bf16 with round-to-nearest-even;
  * draw order: lengths, q, pool permutation (on a CPU torch.Generator), then
    K, then V (on a generator of the device that will hold them, seeded the
    same); the same seed on the same device gives the same bytes;
  * the pool holds ceil(1.0625 x pages needed) pages unless fixed; logical
    blocks take pool indices in order from a seeded permutation;
  * shared-prefix groups are trajectories 8j..8j+7; block j < min(pages, 64)
    of each member maps to the group's j-th shared page;
  * slots no trajectory reads (the tail of a last page, unreferenced pages)
    hold NaN (bf16 0x7FC0, fp8 0x7F); unused block-table entries are -1;
  * fp8 KV (OCP e4m3fn): separate K and V scales per (page, kv-head),
    scale = amax / 448 over the valid slots (1 when amax is 0), stored byte =
    e4m3fn(clamp(x / scale, -448, 448)) with round-to-nearest-even.

Page format (one (page, kv-head) tile of 16 tokens x D dims, contiguous):
  K: with X = 16 bytes / element size, element (t, d) sits at
     ((d // X) * 16 + t) * X + d % X          -- [D/X][16][X]
  V: element (t, d) sits at ((t // 4) * D + d) * 4 + t % 4   -- [4][D][4]
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Optional, Sequence

import numpy as np
import torch

from .configs import PAGE_SIZE, LengthModel, WorkloadConfig, get_config

FP8_MAX = 448.0
FP8_NAN_BYTE = 0x7F


@dataclass
class Workload:
    cfg: WorkloadConfig
    seed: int
    seq_lens: np.ndarray          # int32 [B]
    block_table: np.ndarray       # int32 [B, max_blocks]; -1 = unused
    num_pages: int
    page_valid: np.ndarray        # int32 [num_pages]: valid slots per page
    q: torch.Tensor               # bf16 [B, Hq, D]
    k_pages: torch.Tensor         # bf16 or uint8 [num_pages, Hkv, 16*D]
    v_pages: torch.Tensor         # bf16 or uint8 [num_pages, Hkv, 16*D]
    k_scale: Optional[torch.Tensor]   # fp32 [num_pages, Hkv] (fp8 only)
    v_scale: Optional[torch.Tensor]
    softmax_scale: float
    # [num_pages, Hkv, 16, D] in storage dtype (bf16 / uint8), kept on request
    k_logical: Optional[torch.Tensor] = None
    v_logical: Optional[torch.Tensor] = None

    @property
    def batch(self) -> int:
        return int(self.seq_lens.shape[0])

    def kv_bytes_unique(self) -> int:
        """K+V bytes of valid tokens, each physical page counted once."""
        c = self.cfg
        return int(self.page_valid.astype(np.int64).sum()) * c.num_kv_heads \
            * c.head_dim * 2 * c.kv_elem_bytes

    def kv_bytes_logical(self) -> int:
        """K+V bytes of valid tokens as each trajectory sees them."""
        c = self.cfg
        return int(self.seq_lens.astype(np.int64).sum()) * c.num_kv_heads \
            * c.head_dim * 2 * c.kv_elem_bytes

    def algorithmic_bytes(self) -> int:
        """Bytes the method must move per call: unique KV, q, out, lse,
        block-table entries in use, seq_lens, and fp8 scales of used pages."""
        c = self.cfg
        b = self.batch
        pages = (self.seq_lens.astype(np.int64) + PAGE_SIZE - 1) // PAGE_SIZE
        n = self.kv_bytes_unique()
        n += b * c.num_q_heads * c.head_dim * 2           # q
        n += b * c.num_q_heads * c.head_dim * 4           # out
        n += b * c.num_q_heads * 4                        # lse
        n += int(pages.sum()) * 4 + b * 4                 # block table, lens
        if c.kv_dtype == "fp8_e4m3fn":
            used = int((self.page_valid > 0).sum())
            n += used * c.num_kv_heads * 2 * 4
        return n


def custom_config(lens: Sequence[int], num_q_heads: int, num_kv_heads: int,
                  head_dim: int, kv_dtype: str = "bf16",
                  pool_pages: Optional[int] = None, prefix_group: int = 0,
                  prefix_tokens: int = 0, name: str = "custom") -> WorkloadConfig:
    return WorkloadConfig(
        name=name, index=0, batch=len(lens), num_q_heads=num_q_heads,
        num_kv_heads=num_kv_heads, head_dim=head_dim, kv_dtype=kv_dtype,
        lengths=LengthModel(kind="fixed", values=tuple(int(x) for x in lens)),
        prefix_group=prefix_group, prefix_tokens=prefix_tokens,
        pool_pages=pool_pages)


def draw_lengths(cfg: WorkloadConfig, gen: torch.Generator) -> np.ndarray:
    lm = cfg.lengths
    b = cfg.batch
    if lm.kind == "fixed":
        out = np.asarray(lm.values, dtype=np.int64)
    elif lm.kind == "lognormal":
        z = torch.randn(b, generator=gen, dtype=torch.float64).numpy()
        out = np.rint(np.exp(math.log(lm.median) + lm.sigma * z))
        out = np.clip(out, lm.lo, lm.hi).astype(np.int64)
    elif lm.kind == "uniform":
        out = torch.randint(lm.lo, lm.hi + 1, (b,), generator=gen).numpy()
    elif lm.kind == "bimodal":
        n_long = int(round(lm.long_frac * b))
        perm = torch.randperm(b, generator=gen).numpy()
        is_long = np.zeros(b, dtype=bool)
        is_long[perm[:n_long]] = True
        short = torch.randint(lm.lo, lm.hi + 1, (b,), generator=gen).numpy()
        long_ = torch.randint(lm.long_lo, lm.long_hi + 1, (b,),
                              generator=gen).numpy()
        out = np.where(is_long, long_, short)
    else:
        raise ValueError(f"unknown length model {lm.kind!r}")
    return out.astype(np.int32)


def place_pages(cfg: WorkloadConfig, lens: np.ndarray, gen: torch.Generator):
    """Pool size, block table and per-page valid-slot counts."""
    b = lens.shape[0]
    pages = (lens.astype(np.int64) + PAGE_SIZE - 1) // PAGE_SIZE
    grp = cfg.prefix_group
    pre_pages = cfg.prefix_tokens // PAGE_SIZE if grp else 0
    shared = np.minimum(pages, pre_pages) if grp else np.zeros_like(pages)
    if grp:
        n_groups = -(-b // grp)
        group_need = np.zeros(n_groups, dtype=np.int64)
        np.maximum.at(group_need, np.arange(b) // grp, shared)
        needed = int(group_need.sum() + (pages - shared).sum())
    else:
        needed = int(pages.sum())
    if cfg.pool_pages is not None:
        num_pages = int(cfg.pool_pages)
        if num_pages < needed:
            raise ValueError(f"pool of {num_pages} pages < {needed} needed")
    else:
        num_pages = int(math.ceil(1.0625 * needed))
    num_pages = max(num_pages, 1)
    perm = torch.randperm(num_pages, generator=gen).numpy().astype(np.int64)

    width = max(cfg.max_blocks_per_seq, int(pages.max()) if b else 0, 1)
    table = np.full((b, width), -1, dtype=np.int32)
    valid = np.zeros(num_pages, dtype=np.int32)
    nxt = 0
    shared_map = {}
    for i in range(b):
        n = int(pages[i])
        if n == 0:
            continue
        ns = int(shared[i])
        for j in range(ns):
            key = (i // grp, j)
            if key not in shared_map:
                shared_map[key] = int(perm[nxt])
                nxt += 1
            table[i, j] = shared_map[key]
        priv = n - ns
        table[i, ns:n] = perm[nxt:nxt + priv]
        nxt += priv
        slots = np.minimum(PAGE_SIZE, int(lens[i]) - PAGE_SIZE * np.arange(n))
        np.maximum.at(valid, table[i, :n].astype(np.int64), slots.astype(np.int32))
    return num_pages, table, valid


def _kv_pool(num_pages: int, hkv: int, d: int, kv_dtype: str,
             page_valid: np.ndarray, gen: torch.Generator, device,
             which: str, keep_logical: bool):
    """Draw one K or V pool, poison unread slots, quantise for fp8.

    Returns (pages [P, Hkv, 16*D] in page format, scale [P, Hkv] or None,
    logical [P, Hkv, 16, D] or None)."""
    fp8 = kv_dtype == "fp8_e4m3fn"
    store = torch.uint8 if fp8 else torch.bfloat16
    pages = torch.empty((num_pages, hkv, PAGE_SIZE * d), dtype=store,
                        device=device)
    logical = torch.empty((num_pages, hkv, PAGE_SIZE, d), dtype=store,
                          device=device) if keep_logical else None
    scale = torch.empty((num_pages, hkv), dtype=torch.float32,
                        device=device) if fp8 else None
    pv = torch.as_tensor(page_valid, dtype=torch.int32, device=device)
    slot = torch.arange(PAGE_SIZE, device=device, dtype=torch.int32)
    chunk = max(1, (1 << 26) // (hkv * PAGE_SIZE * d))
    for p0 in range(0, num_pages, chunk):
        p1 = min(num_pages, p0 + chunk)
        x = torch.randn((p1 - p0, hkv, PAGE_SIZE, d), generator=gen,
                        device=device, dtype=torch.float32)
        ok = (slot[None, :] < pv[p0:p1, None])[:, None, :, None]
        if fp8:
            amax = torch.where(ok, x.abs(), torch.zeros_like(x)).amax(dim=(2, 3))
            s = amax / FP8_MAX
            s = torch.where(amax == 0, torch.ones_like(s), s)
            y = (x / s[:, :, None, None]).clamp(-FP8_MAX, FP8_MAX)
            y = y.to(torch.float8_e4m3fn).view(torch.uint8)
            y = torch.where(ok, y, torch.full_like(y, FP8_NAN_BYTE))
            scale[p0:p1] = s
        else:
            y = x.to(torch.bfloat16)
            y = torch.where(ok, y, torch.full_like(y, float("nan")))
        del x
        pages[p0:p1] = to_page_format(y, which)
        if keep_logical:
            logical[p0:p1] = y
    return pages, scale, logical


def to_page_format(logical: torch.Tensor, which: str) -> torch.Tensor:
    """[P, Hkv, 16, D] -> [P, Hkv, 16*D] in the library's K or V tile order."""
    p, h, t, d = logical.shape
    x = 16 // logical.element_size()
    if which == "k":
        y = logical.view(p, h, t, d // x, x).permute(0, 1, 3, 2, 4)
    elif which == "v":
        y = logical.view(p, h, t // 4, 4, d).permute(0, 1, 2, 4, 3)
    else:
        raise ValueError(which)
    return y.contiguous().view(p, h, t * d)


def make_workload(cfg, seed: Optional[int] = None, device="cpu",
                  keep_logical: bool = False,
                  lens: Optional[Sequence[int]] = None) -> Workload:
    cfg = get_config(cfg)
    seed = cfg.default_seed if seed is None else int(seed)
    device = torch.device(device)
    gen = torch.Generator(device="cpu").manual_seed(seed)
    if lens is None:
        seq_lens = draw_lengths(cfg, gen)
    else:
        seq_lens = np.asarray(lens, dtype=np.int32)
    b = seq_lens.shape[0]
    q = torch.randn((b, cfg.num_q_heads, cfg.head_dim), generator=gen,
                    dtype=torch.float32).to(torch.bfloat16).to(device)
    num_pages, table, valid = place_pages(cfg, seq_lens, gen)
    if device.type == "cpu":
        kv_gen = gen
    else:
        kv_gen = torch.Generator(device=device).manual_seed(seed)
    hkv, d = cfg.num_kv_heads, cfg.head_dim
    k_pages, k_scale, k_log = _kv_pool(num_pages, hkv, d, cfg.kv_dtype,
                                       valid, kv_gen, device, "k",
                                       keep_logical)
    v_pages, v_scale, v_log = _kv_pool(num_pages, hkv, d, cfg.kv_dtype,
                                       valid, kv_gen, device, "v",
                                       keep_logical)
    return Workload(cfg=cfg, seed=seed, seq_lens=seq_lens, block_table=table,
                    num_pages=num_pages, page_valid=valid, q=q,
                    k_pages=k_pages, v_pages=v_pages, k_scale=k_scale,
                    v_scale=v_scale, softmax_scale=1.0 / math.sqrt(d),
                    k_logical=k_log, v_logical=v_log)


def prefix_groups(wl: Workload):
    """(group_of [B], group_pages [G]) of a workload with shared prefixes:
    trajectory b belongs to group b // prefix_group, whose first
    prefix_tokens / 16 blocks are shared. (None, None) without sharing."""
    cfg = wl.cfg
    if not cfg.prefix_group:
        return None, None
    b = wl.batch
    group_of = (np.arange(b) // cfg.prefix_group).astype(np.int32)
    n_groups = -(-b // cfg.prefix_group)
    pages = np.full(n_groups, cfg.prefix_tokens // PAGE_SIZE, dtype=np.int32)
    return group_of, pages


def _bits(t: torch.Tensor) -> np.ndarray:
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    if t.dtype == torch.uint8:
        return t.numpy()
    return t.numpy()


def host_arrays(wl: Workload, seqs: Optional[Sequence[int]] = None) -> dict:
    """Raw host copies (bf16 as uint16 bits, fp8 as uint8) of the inputs of
    the trajectories ``seqs`` (all if None), with the pool cut down to the
    pages they reference and the block table renumbered to match."""
    b = wl.batch
    idx = np.arange(b) if seqs is None else np.asarray(seqs, dtype=np.int64)
    table = wl.block_table[idx]
    lens = wl.seq_lens[idx]
    used = np.unique(table[table >= 0]).astype(np.int64)
    if seqs is None:
        used = np.arange(wl.num_pages, dtype=np.int64)
    remap = np.full(wl.num_pages, -1, dtype=np.int64)
    remap[used] = np.arange(used.shape[0])
    new_table = np.where(table >= 0, remap[np.maximum(table, 0)], -1)
    sel = torch.as_tensor(used, device=wl.k_pages.device)
    pick = (lambda t: t) if seqs is None else (lambda t: t.index_select(0, sel))
    out = dict(
        q=_bits(wl.q[torch.as_tensor(idx, device=wl.q.device)]),
        k_pages=_bits(pick(wl.k_pages)),
        v_pages=_bits(pick(wl.v_pages)),
        block_table=new_table.astype(np.int32),
        seq_lens=lens.astype(np.int32),
        k_scale=None, v_scale=None,
        kv_dtype=wl.cfg.kv_dtype, head_dim=wl.cfg.head_dim,
        num_kv_heads=wl.cfg.num_kv_heads, softmax_scale=wl.softmax_scale,
    )
    if wl.k_scale is not None:
        out["k_scale"] = pick(wl.k_scale).cpu().numpy()
        out["v_scale"] = pick(wl.v_scale).cpu().numpy()
    return out
