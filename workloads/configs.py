"""The five named decode-attention workloads and the length models behind them.

Each workload is one layer's decode-attention call over a paged KV cache: one
query token per trajectory, trajectories of long-tail-skewed length. The paper
motivates the shapes (rollout decode is memory-bound and dominates the RL
iteration, §1 and §2.4; KV-cache capacity bounds the decode batch, §5.2; long
tails are ~10x the median, §2.2) but prints no attention shapes; the head
counts follow the Qwen2.5 7B/32B/72B models it trains (§8, "Models").

This module holds sizes only: no random draws and no attention arithmetic.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional, Tuple

PAGE_SIZE = 16


@dataclass(frozen=True)
class LengthModel:
    """How the per-trajectory KV lengths are drawn.

    kind:
      "fixed"     -- ``values`` verbatim.
      "lognormal" -- clip(rint(exp(ln(median) + sigma * z)), lo, hi), z ~ N(0, 1).
      "uniform"   -- integers uniform in [lo, hi], both ends inclusive.
      "bimodal"   -- exactly round(long_frac * B) trajectories (at seeded
                     positions) uniform in [long_lo, long_hi], the rest uniform
                     in [lo, hi].
    """

    kind: str
    values: Tuple[int, ...] = ()
    median: float = 0.0
    sigma: float = 0.0
    lo: int = 0
    hi: int = 0
    long_frac: float = 0.0
    long_lo: int = 0
    long_hi: int = 0

    def max_len(self) -> int:
        if self.kind == "fixed":
            return max(self.values) if self.values else 0
        if self.kind == "bimodal":
            return max(self.hi, self.long_hi)
        return self.hi


@dataclass(frozen=True)
class WorkloadConfig:
    name: str
    index: int                 # 1-based position in the list below
    batch: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    kv_dtype: str              # "bf16" or "fp8_e4m3fn"
    lengths: LengthModel
    prefix_group: int = 0      # trajectories per shared-prefix group (0: none)
    prefix_tokens: int = 0     # shared prompt tokens per group
    pool_pages: Optional[int] = None   # fixed pool size; None: 1.0625 x needed
    description: str = ""
    seed_of: int = 0           # draw with this workload's seed (0: own index)

    @property
    def group_size(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    @property
    def max_blocks_per_seq(self) -> int:
        return -(-self.lengths.max_len() // PAGE_SIZE)

    @property
    def default_seed(self) -> int:
        return 1000 + (self.seed_of or self.index)

    @property
    def kv_elem_bytes(self) -> int:
        return 1 if self.kv_dtype == "fp8_e4m3fn" else 2


CONFIGS = (
    WorkloadConfig(
        name="tiny", index=1, batch=4, num_q_heads=4, num_kv_heads=1,
        head_dim=64, kv_dtype="bf16",
        lengths=LengthModel(kind="fixed", values=(17, 64, 200, 513)),
        pool_pages=64,
        description="4 trajectories of 17/64/200/513 tokens, 4q/1kv heads, "
                    "head_dim 64, 64-page pool"),
    WorkloadConfig(
        name="7b_pre_repack", index=2, batch=256, num_q_heads=28,
        num_kv_heads=4, head_dim=128, kv_dtype="bf16",
        lengths=LengthModel(kind="lognormal", median=2048, sigma=1.0,
                            lo=16, hi=32768),
        description="256 trajectories, lognormal(median 2048, sigma 1.0) "
                    "lengths clipped to [16, 32768], 28q/4kv, bf16 KV"),
    WorkloadConfig(
        name="post_repack", index=3, batch=8, num_q_heads=28, num_kv_heads=4,
        head_dim=128, kv_dtype="bf16",
        lengths=LengthModel(kind="uniform", lo=20000, hi=65536),
        description="8 trajectories uniform in [20000, 65536] tokens, "
                    "28q/4kv, bf16 KV"),
    WorkloadConfig(
        name="32b_fp8", index=4, batch=128, num_q_heads=40, num_kv_heads=8,
        head_dim=128, kv_dtype="fp8_e4m3fn",
        lengths=LengthModel(kind="lognormal", median=4096, sigma=1.2,
                            lo=16, hi=32768),
        description="128 trajectories, lognormal(median 4096, sigma 1.2) "
                    "clipped to [16, 32768], 40q/8kv, fp8-e4m3fn KV with a "
                    "per-(page, kv-head) fp32 scale"),
    WorkloadConfig(
        name="agentic_mix", index=5, batch=512, num_q_heads=64,
        num_kv_heads=8, head_dim=128, kv_dtype="bf16",
        lengths=LengthModel(kind="bimodal", lo=256, hi=4096, long_frac=0.1,
                            long_lo=32768, long_hi=98304),
        prefix_group=8, prefix_tokens=1024,
        description="512 trajectories, 90% uniform in [256, 4096] and 10% "
                    "uniform in [32768, 98304]; groups of 8 share a "
                    "1024-token prompt prefix; 64q/8kv, bf16 KV"),
)

# One GPU's share of the two larger models under the tensor parallelism the
# paper rolls them out with (appendix, hyperparameter details: TP 4 for 32B,
# TP 8 for 72B, whose head counts the agentic mix uses): the same
# trajectories and lengths, the kv-heads split across GPUs with their query
# heads. Attention needs no exchange between the shares, so one GPU's call
# is exactly this.
_FULL = {c.name: c for c in CONFIGS}

TP_SHARES = (
    WorkloadConfig(
        name="32b_fp8_tp4", index=6, batch=128, num_q_heads=10,
        num_kv_heads=2, head_dim=128, kv_dtype="fp8_e4m3fn",
        lengths=_FULL["32b_fp8"].lengths, seed_of=_FULL["32b_fp8"].index,
        description="32b_fp8 on one GPU of four: 10q/2kv heads, the same "
                    "trajectory lengths"),
    WorkloadConfig(
        name="agentic_mix_tp8", index=7, batch=512, num_q_heads=8,
        num_kv_heads=1, head_dim=128, kv_dtype="bf16",
        lengths=_FULL["agentic_mix"].lengths, prefix_group=8, prefix_tokens=1024,
        seed_of=_FULL["agentic_mix"].index,
        description="agentic_mix on one GPU of eight: 8q/1kv heads, the "
                    "same trajectory lengths and shared prefixes"),
)

BY_NAME = {c.name: c for c in CONFIGS + TP_SHARES}


def get_config(key) -> WorkloadConfig:
    """Look a workload up by 1-based index or by name."""
    if isinstance(key, WorkloadConfig):
        return key
    if isinstance(key, int) or (isinstance(key, str) and key.isdigit()):
        return (CONFIGS + TP_SHARES)[int(key) - 1]
    return BY_NAME[key]
