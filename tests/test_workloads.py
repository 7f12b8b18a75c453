"""Checks of the seeded input generator (CPU)."""
import math

import numpy as np
import torch

from workloads import CONFIGS, custom_config, get_config, make_workload
from workloads.generate import draw_lengths, place_pages


def _layout(cfg, seed=None):
    cfg = get_config(cfg)
    gen = torch.Generator().manual_seed(cfg.default_seed if seed is None else seed)
    lens = draw_lengths(cfg, gen)
    torch.randn((cfg.batch, cfg.num_q_heads, cfg.head_dim), generator=gen)
    return cfg, lens, place_pages(cfg, lens, gen)


def test_length_models_match_config_text():
    for cfg in CONFIGS:
        _, lens, _ = _layout(cfg)
        assert lens.shape == (cfg.batch,) and lens.dtype == np.int32
    assert list(_layout(1)[1]) == [17, 64, 200, 513]
    l2 = _layout(2)[1]
    assert l2.min() >= 16 and l2.max() <= 32768
    l3 = _layout(3)[1]
    assert l3.min() >= 20000 and l3.max() <= 65536
    l4 = _layout(4)[1]
    assert l4.min() >= 16 and l4.max() <= 32768
    l5 = _layout(5)[1]
    long_ = l5 >= 32768
    assert long_.sum() == 51
    assert l5[~long_].min() >= 256 and l5[~long_].max() <= 4096
    assert l5[long_].max() <= 98304


def test_tensor_parallel_shares_keep_the_batch():
    """A TP share is the parent's batch with 1/TP of its heads."""
    for share, parent, tp in (("32b_fp8_tp4", 4, 4), ("agentic_mix_tp8", 5, 8)):
        s, p = get_config(share), get_config(parent)
        assert np.array_equal(_layout(s)[1], _layout(p)[1])
        assert (s.num_q_heads * tp, s.num_kv_heads * tp) == (p.num_q_heads,
                                                            p.num_kv_heads)
        assert (s.kv_dtype, s.prefix_group, s.prefix_tokens) == (
            p.kv_dtype, p.prefix_group, p.prefix_tokens)


def test_page_counts_and_pool_occupancy():
    for idx in (1, 2, 3, 4):
        cfg, lens, (num_pages, table, valid) = _layout(idx)
        pages = -(-lens.astype(np.int64) // 16)
        needed = int(pages.sum())
        if cfg.pool_pages:
            assert num_pages == cfg.pool_pages
        else:
            assert num_pages == math.ceil(1.0625 * needed)
        used = table[table >= 0]
        assert used.size == needed and np.unique(used).size == needed
        assert used.min() >= 0 and used.max() < num_pages
        for b in range(cfg.batch):
            assert (table[b, :pages[b]] >= 0).all()
            assert (table[b, pages[b]:] == -1).all()
        assert int(valid.sum()) == int(lens.sum())
        assert int((valid > 0).sum()) == needed


def test_prefix_aliasing_structure_config5():
    cfg, lens, (num_pages, table, valid) = _layout(5)
    pages = -(-lens.astype(np.int64) // 16)
    for grp in range(cfg.batch // 8):
        members = range(8 * grp, 8 * grp + 8)
        rows = [table[b, :min(64, pages[b])] for b in members]
        longest = max(rows, key=len)
        for r in rows:
            assert np.array_equal(r, longest[:len(r)])
        # private pages are not shared with anyone
    priv = np.concatenate([table[b, 64:pages[b]] for b in range(cfg.batch)])
    assert np.unique(priv).size == priv.size
    shared = np.unique(np.concatenate(
        [table[b, :min(64, pages[b])] for b in range(cfg.batch)]))
    assert np.intersect1d(shared, priv).size == 0


def test_nan_poison_only_in_unread_slots():
    cfg = custom_config([1, 17, 31, 5, 64, 3, 100, 2], 8, 2, 64,
                        prefix_group=4, prefix_tokens=64)
    wl = make_workload(cfg, seed=3, keep_logical=True)
    k = wl.k_logical.float()
    nan_slot = torch.isnan(k).all(dim=-1).all(dim=1)          # [P, 16]
    any_nan = torch.isnan(k).any(dim=-1).any(dim=1)
    assert torch.equal(nan_slot, any_nan)
    expect = torch.arange(16)[None, :] >= torch.as_tensor(wl.page_valid)[:, None]
    assert torch.equal(nan_slot, expect)
    # every slot a trajectory reads is finite
    for b in range(wl.batch):
        for t in range(int(wl.seq_lens[b])):
            p = wl.block_table[b, t // 16]
            assert not nan_slot[p, t % 16]


def test_fp8_scales_and_codes():
    cfg = custom_config([5, 40, 16], 4, 2, 64, kv_dtype="fp8_e4m3fn")
    wl = make_workload(cfg, seed=4, keep_logical=True)
    for p in range(wl.num_pages):
        n = int(wl.page_valid[p])
        for h in range(2):
            codes = wl.k_logical[p, h]
            if n == 0:
                assert (codes == 0x7F).all() and wl.k_scale[p, h] == 1.0
                continue
            vals = codes[:n].view(torch.float8_e4m3fn).float()
            assert torch.isfinite(vals).all()
            assert vals.abs().max() == 448.0          # amax maps to the max code
            assert (codes[n:] == 0x7F).all()
            assert wl.k_scale[p, h] > 0 and wl.v_scale[p, h] > 0


def test_same_seed_same_bytes():
    a = make_workload(custom_config([100, 7], 4, 2, 64, kv_dtype="fp8_e4m3fn"),
                      seed=21)
    b = make_workload(custom_config([100, 7], 4, 2, 64, kv_dtype="fp8_e4m3fn"),
                      seed=21)
    c = make_workload(custom_config([100, 7], 4, 2, 64, kv_dtype="fp8_e4m3fn"),
                      seed=22)
    assert torch.equal(a.k_pages, b.k_pages) and torch.equal(a.v_pages, b.v_pages)
    assert torch.equal(a.q.view(torch.int16), b.q.view(torch.int16))
    assert np.array_equal(a.block_table, b.block_table)
    assert not torch.equal(a.k_pages, c.k_pages)


def test_algorithmic_bytes_accounting():
    wl = make_workload(1, seed=1001)
    kv = int(wl.seq_lens.sum()) * 1 * 64 * 2 * 2
    assert wl.kv_bytes_unique() == wl.kv_bytes_logical() == kv
    assert wl.kv_bytes_unique() == 203264
    pages = int((-(-wl.seq_lens.astype(np.int64) // 16)).sum())
    assert wl.algorithmic_bytes() == kv + 4 * 4 * 64 * 6 + 4 * 4 * 4 \
        + pages * 4 + 4 * 4
