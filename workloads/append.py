"""Seeded inputs for decode steps that append to a workload's KV cache.

Shared by the oracle's tests and by the GPU path's tests and bench. It draws
the new tokens' keys and values and gives every trajectory the pages its
next tokens need; it performs none of the cache arithmetic (no
quantisation, no scale update).

Readings (the paper gives no cache-write inputs):
  * one decode step appends one token to every trajectory of the batch, so
    before step i (0-based) trajectory b holds lens0[b] + i tokens and
    after it lens0[b] + i + 1;
  * blocks the longer trajectories need get fresh pool pages appended after
    the workload's pool, in a seeded random order; their slots hold NaN
    (bf16 0x7FC0, fp8 0x7F) and, for fp8, their scales NaN, so nothing may
    read a slot or scale before it is written;
  * new keys and values are bf16 (RNE) of N(0, 1) draws, optionally
    multiplied per (step, trajectory, kv-head, K|V) to reach the corners of
    fp8 encoding ("stress": x4, x2^-8, x0 or x300 next to x1; "ties": every
    token has amax 448 * 2^k and otherwise holds midpoints between adjacent
    E4M3FN magnitudes, times 2^k, so that x / 2^k falls exactly on ties);
  * workloads whose trajectories share prefix pages are refused: a shared
    last page would have to be copied before it is written.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional

import numpy as np
import torch

from .configs import PAGE_SIZE
from .generate import FP8_NAN_BYTE, Workload

MIXES = ("normal", "stress", "ties")


@dataclass
class DecodeRun:
    base: Workload
    steps: int
    lens0: np.ndarray                 # int32 [B], before the first append
    block_table: np.ndarray           # int32 [B, W], room for lens0 + steps
    num_pages: int
    k_pages: torch.Tensor             # pools with the fresh pages appended
    v_pages: torch.Tensor
    k_scale: Optional[torch.Tensor]   # fp32 [num_pages, Hkv] (fp8 only)
    v_scale: Optional[torch.Tensor]
    k_new: torch.Tensor               # bf16 [steps, B, Hkv, D]
    v_new: torch.Tensor

    def lens_after(self, step: int) -> np.ndarray:
        """Lengths including the token appended at ``step``."""
        return (self.lens0 + step + 1).astype(np.int32)


def _e4m3fn_midpoints() -> np.ndarray:
    """Midpoints between adjacent finite non-negative E4M3FN magnitudes."""
    mags = []
    for code in range(0x7F):
        e, m = code >> 3, code & 7
        mags.append(m * 2.0 ** -9 if e == 0 else (1 + m / 8) * 2.0 ** (e - 7))
    mags = np.asarray(mags)
    return (mags[:-1] + mags[1:]) / 2


def _draw_tokens(steps, b, hkv, d, mix, gen):
    x = torch.randn((2, steps, b, hkv, d), generator=gen, dtype=torch.float32)
    if mix == "normal":
        pass
    elif mix == "stress":
        choice = torch.multinomial(torch.tensor([0.6, 0.15, 0.1, 0.1, 0.05]),
                                   2 * steps * b * hkv, replacement=True,
                                   generator=gen)
        mult = torch.tensor([1.0, 4.0, 2.0 ** -8, 0.0, 300.0])[choice]
        x = x * mult.view(2, steps, b, hkv, 1)
    elif mix == "ties":
        mids = torch.as_tensor(_e4m3fn_midpoints(), dtype=torch.float32)
        pick = torch.randint(0, mids.numel(), x.shape, generator=gen)
        sign = torch.where(x < 0, -1.0, 1.0)
        k = torch.tensor([-8.0, -3.0, 0.0, 2.0])[
            torch.randint(0, 4, (2, 1, b, hkv, 1), generator=gen)]
        x = sign * mids[pick] * torch.exp2(k)
        x[..., 0] = 448.0 * torch.exp2(k[..., 0])     # the token's amax
    else:
        raise ValueError(f"mix must be one of {MIXES}")
    x = x.to(torch.bfloat16)
    return x[0], x[1]


def make_decode_run(wl: Workload, steps: int, seed: int = 7,
                    mix: str = "normal") -> DecodeRun:
    cfg = wl.cfg
    if cfg.prefix_group:
        raise ValueError("workloads with shared prefix pages are not appended to")
    b, hkv, d = wl.batch, cfg.num_kv_heads, cfg.head_dim
    device = wl.k_pages.device
    gen = torch.Generator().manual_seed(int(seed))
    lens0 = wl.seq_lens.astype(np.int64)
    pages0 = (lens0 + PAGE_SIZE - 1) // PAGE_SIZE
    pages1 = (lens0 + steps + PAGE_SIZE - 1) // PAGE_SIZE
    fresh = int((pages1 - pages0).sum())
    order = torch.randperm(max(fresh, 1), generator=gen).numpy()[:fresh]
    new_ids = wl.num_pages + order
    width = max(wl.block_table.shape[1], int(pages1.max()) if b else 0, 1)
    table = np.full((b, width), -1, dtype=np.int32)
    table[:, :wl.block_table.shape[1]] = wl.block_table
    nxt = 0
    for i in range(b):
        n = int(pages1[i] - pages0[i])
        table[i, pages0[i]:pages1[i]] = new_ids[nxt:nxt + n]
        nxt += n
    num_pages = wl.num_pages + fresh

    fp8 = cfg.kv_dtype == "fp8_e4m3fn"
    tile = wl.k_pages.shape[2]

    def grow(pool):
        extra = torch.empty((fresh, hkv, tile), dtype=pool.dtype, device=device)
        if fp8:
            extra.fill_(FP8_NAN_BYTE)
        else:
            extra.fill_(float("nan"))
        return torch.cat([pool, extra])

    def grow_scale(s):
        if s is None:
            return None
        return torch.cat([s, torch.full((fresh, hkv), float("nan"),
                                        dtype=s.dtype, device=device)])

    k_new, v_new = _draw_tokens(steps, b, hkv, d, mix, gen)
    return DecodeRun(base=wl, steps=steps, lens0=lens0.astype(np.int32),
                     block_table=table, num_pages=num_pages,
                     k_pages=grow(wl.k_pages), v_pages=grow(wl.v_pages),
                     k_scale=grow_scale(wl.k_scale),
                     v_scale=grow_scale(wl.v_scale),
                     k_new=k_new.to(device), v_new=v_new.to(device))
