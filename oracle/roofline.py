"""CPU oracle for the roofline batch bound of one decode step.

TEST INFRASTRUCTURE. Only the tests, the package smoke check and the bench's
CPU-baseline leg may import or call this module. The GPU library never does,
and this module imports nothing from the GPU path.

What it computes. Repacking bounds a destination's decode batch by B, the
largest batch decoded at nearly the latency of a small one: under the
roofline model it is where decoding turns from memory-bound to
compute-bound (§5.2, where B enters Algorithm 1; §2.4 and its
latency-versus-batch figure show the flat, memory-bound part). One decode
step of a dense decoder (L layers, hidden size h, Hq query and Hkv KV heads
of size D, gated MLP of width I, vocabulary V; weights of wb bytes,
activations of ab bytes, KV entries of kb bytes) over M trajectories that
each hold c cached tokens runs these operations:

  * projections, per layer QKV [h -> (Hq + 2 Hkv) D], O [Hq D -> h],
    gate and up [h -> 2 I], down [I -> h], and the LM head [h -> V]: a
    product [M, K] x [K, N] does 2 M N K flops and moves wb N K weight
    bytes plus ab M (K + N) activation bytes;
  * attention, per layer: 4 M c Hq D flops (QK^T and PV) and
    kb 2 Hkv D M (c + 1) KV bytes (c cached tokens read, one written).

Reading: B is the transition of the projections, the part of the step
whose cost does not grow with the batch while it is memory-bound:

    B = min { M >= 1 : sum 2 M N K / F >= sum (wb N K + ab M (K + N)) / BW }

for peak compute F (FLOP/s) and bandwidth BW (B/s). Attention's intensity
is Hq / (Hkv kb) flops per byte (7 for bf16 at GQA 7), far below any
matrix-core balance, so it stays memory-bound at every batch; its cost is
per trajectory and enters the step time, not the transition. The step time
of the model is the sum over operations of max(flops / F, bytes / BW). No
bound exists when activations outweigh the weights' compute gain
(2 sum N K / F <= ab sum (K + N) / BW). All arithmetic is exact (integers
and Fractions). Norms, biases, rotary embedding and the embedding row are
left out (a few MB against GBs of weights and KV).
"""
from __future__ import annotations

from dataclasses import dataclass
from fractions import Fraction
from typing import List, Optional, Tuple


@dataclass(frozen=True)
class ModelShape:
    layers: int
    hidden: int
    q_heads: int
    kv_heads: int
    head_dim: int
    intermediate: int
    vocab: int
    weight_bytes: int = 2
    act_bytes: int = 2
    kv_bytes: int = 2


# Qwen2.5-7B and -32B shapes (the paper's models, §8 "Models").
QWEN25_7B = ModelShape(28, 3584, 28, 4, 128, 18944, 152064)
QWEN25_32B = ModelShape(64, 5120, 40, 8, 128, 27648, 152064)


def projections(m: ModelShape) -> List[Tuple[int, int]]:
    """(K, N) of every projection of one decode step."""
    h, d = m.hidden, m.head_dim
    layer = [(h, (m.q_heads + 2 * m.kv_heads) * d), (m.q_heads * d, h),
             (h, 2 * m.intermediate), (m.intermediate, h)]
    return layer * m.layers + [(h, m.vocab)]


def params(m: ModelShape) -> int:
    return sum(k * n for k, n in projections(m))


def batch_bound(m: ModelShape, peak_flops: int, peak_bw: int) -> Optional[int]:
    """Smallest M >= 1 at which the projections are compute-bound."""
    nk = sum(k * n for k, n in projections(m))
    kn = sum(k + n for k, n in projections(m))
    gain = Fraction(2 * nk, peak_flops) - Fraction(m.act_bytes * kn, peak_bw)
    if gain <= 0:
        return None
    q = Fraction(m.weight_bytes * nk, peak_bw) / gain
    bound = q.numerator // q.denominator
    if bound < q:
        bound += 1
    return max(bound, 1)


def projections_compute_bound(m: ModelShape, batch: int, peak_flops: int,
                              peak_bw: int) -> bool:
    f = sum(Fraction(2 * batch * n * k, peak_flops) for k, n in projections(m))
    b = sum(Fraction(m.weight_bytes * n * k + m.act_bytes * batch * (k + n),
                     peak_bw) for k, n in projections(m))
    return f >= b


def step_time(m: ModelShape, batch: int, context: int, peak_flops: int,
              peak_bw: int) -> Fraction:
    """Roofline time of one decode step: each operation at its own bound."""
    t = Fraction(0)
    for k, n in projections(m):
        t += max(Fraction(2 * batch * n * k, peak_flops),
                 Fraction(m.weight_bytes * n * k
                          + m.act_bytes * batch * (k + n), peak_bw))
    att_f = 4 * batch * context * m.q_heads * m.head_dim
    att_b = m.kv_bytes * 2 * m.kv_heads * m.head_dim * batch * (context + 1)
    t += m.layers * max(Fraction(att_f, peak_flops), Fraction(att_b, peak_bw))
    return t
