"""The planner's decomposition is exact: evaluating every work item of a plan
in float64 with the oracle's attention (each item over its page range,
cascade items once per member row with the member's length as the limit and
the longest member's table row as the page source), then merging each merge
record's partials, reproduces the oracle's result to rounding. Host only:
the plan tables come from the library's planner, no GPU is touched.
"""
import numpy as np
import pytest

from oracle import decode_attention_from_host
from oracle.decode_attention import attend, bf16_bits_to_f64, gather_kv
from paper_2510_12633_amd import _native as N
from workloads import custom_config, host_arrays, make_workload, prefix_groups


def plan_tables(wl, ppi, waves, cascade):
    c = wl.cfg
    d = N.LaminarAttnDesc(
        batch=wl.batch, num_q_heads=c.num_q_heads, num_kv_heads=c.num_kv_heads,
        head_dim=c.head_dim, page_size=16, num_pages=wl.num_pages,
        max_blocks_per_seq=wl.block_table.shape[1], kv_dtype=0,
        softmax_scale=wl.softmax_scale, k_scale=None, v_scale=None,
        pages_per_item=ppi, waves_per_item=waves)
    if cascade:
        group_of, group_pages = prefix_groups(wl)
        p = N.laminar_plan_create_cascade(d, wl.seq_lens, group_of,
                                          group_pages, 256)
    else:
        p = N.laminar_plan_create(d, wl.seq_lens, 256)
    try:
        return (N.laminar_plan_items_copy(p), N.laminar_plan_merges_copy(p),
                N.laminar_plan_cascade_units_copy(p),
                N.laminar_plan_cascade_members_copy(p))
    finally:
        N.laminar_plan_destroy(p)


def evaluate_plan(wl, arrays, tables):
    items, merges, cunits, cmem = tables
    c = wl.cfg
    hkv, d = c.num_kv_heads, c.head_dim
    g = c.num_q_heads // hkv
    q = bf16_bits_to_f64(arrays["q"])
    lens = arrays["seq_lens"]
    out = np.full((wl.batch, c.num_q_heads, d), np.nan)
    lse = np.full((wl.batch, c.num_q_heads), np.nan)
    po, pl, kv = {}, {}, {}

    def partial(b, kvh, p0, p1, row, limit):
        if (row, kvh) not in kv:
            kv[(row, kvh)] = gather_kv(arrays["k_pages"], arrays["v_pages"],
                                       arrays["block_table"][row],
                                       int(lens[row]), kvh, d, "bf16")
        k, v = kv[(row, kvh)]
        lo, hi = 16 * p0, min(16 * p1, limit)
        heads = slice(kvh * g, kvh * g + g)
        if hi <= lo:
            return np.zeros((g, d)), np.full(g, -np.inf)
        return attend(q[b, heads], k[lo:hi], v[lo:hi], wl.softmax_scale)

    for unit, p0, p1, slot in items:
        if unit >= 0:
            b, kvh = divmod(int(unit), hkv)
            o, l = partial(b, kvh, p0, p1, b, int(lens[b]))
            if slot < 0:
                out[b, kvh * g:(kvh + 1) * g] = o
                lse[b, kvh * g:(kvh + 1) * g] = l
            else:
                po[int(slot)], pl[int(slot)] = o, l
        else:
            row, cnt, moff, kvh = cunits[-unit - 1]
            for b, s0 in cmem[moff:moff + cnt]:
                o, l = partial(int(b), int(kvh), p0, p1, int(row), int(lens[b]))
                po[int(s0 + slot)], pl[int(s0 + slot)] = o, l
    for unit, s0, n, _ in merges:
        b, kvh = divmod(int(unit), hkv)
        L = np.stack([pl[s] for s in range(s0, s0 + n)])
        O = np.stack([po[s] for s in range(s0, s0 + n)])
        m = L.max(axis=0)
        with np.errstate(invalid="ignore"):
            tot = np.where(np.isinf(m), -np.inf,
                           m + np.log(np.exp(L - m).sum(axis=0)))
            w = np.where(np.isinf(tot), 0.0, np.exp(L - tot))
        out[b, kvh * g:(kvh + 1) * g] = (w[:, :, None] * O).sum(axis=0)
        lse[b, kvh * g:(kvh + 1) * g] = tot
    return out, lse


SHAPES = [
    ("plain_ragged", custom_config([0, 1, 17, 300, 1000, 33], 8, 2, 64), False),
    ("cascade_16members", custom_config(
        [0, 5, 511, 512, 513, 1024, 3000, 77, 600, 512, 9000, 1, 256, 700,
         2048, 40, 1200, 300], 32, 4, 64, prefix_group=16, prefix_tokens=512),
     True),
    ("cascade_g5", custom_config([100, 257, 3000, 20, 256, 999, 0], 15, 3, 64,
                                 prefix_group=3, prefix_tokens=256), True),
    ("cascade_mha", custom_config([50, 700, 130, 129, 128, 1000], 2, 2, 64,
                                  prefix_group=6, prefix_tokens=128), True),
]


@pytest.mark.parametrize("name,cfg,cascade", SHAPES, ids=[s[0] for s in SHAPES])
def test_plan_evaluates_to_the_oracle(name, cfg, cascade):
    wl = make_workload(cfg, seed=17)
    arrays = host_arrays(wl)
    ro, rl = decode_attention_from_host(arrays)
    fin = np.isfinite(rl)
    for ppi, waves in ((0, 4), (2, 1), (5, 2)):
        o, l = evaluate_plan(wl, arrays, plan_tables(wl, ppi, waves, cascade))
        assert np.array_equal(np.isneginf(l), np.isneginf(rl)), (ppi, waves)
        assert np.abs(o - ro).max() <= 1e-12, (name, ppi, waves)
        assert np.abs(l[fin] - rl[fin]).max() <= 1e-12, (name, ppi, waves)
