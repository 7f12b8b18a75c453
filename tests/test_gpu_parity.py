"""GPU parity: the HIP library through its C ABI against the fp64 oracle.

Bar: fp32 out and lse within max-abs 1e-3 of the oracle on every case.
Identities that hold exactly on the GPU (page permutation, prefix aliasing,
run-to-run) are checked bitwise.
"""
import math
import os

import numpy as np
import pytest
import torch

from oracle import decode_attention_from_host
from workloads import (custom_config, get_config, host_arrays, make_workload,
                       prefix_groups)

pytestmark = pytest.mark.gpu

TOL = 1e-3


def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")


def _say(msg):
    print(f"[gpu-parity] {msg}", flush=True)


def run_gpu(wl, pages_per_item=0, waves_per_item=0, block_table=None,
            k_pages=None, v_pages=None, two_phase=False, cascade=False):
    from paper_2510_12633_amd.api import PagedDecodeAttention
    c = wl.cfg
    dev = wl.q.device
    bt_np = wl.block_table if block_table is None else block_table
    bt = torch.as_tensor(bt_np, device=dev)
    lens = torch.as_tensor(wl.seq_lens, device=dev)
    att = PagedDecodeAttention(
        batch=wl.batch, num_q_heads=c.num_q_heads, num_kv_heads=c.num_kv_heads,
        head_dim=c.head_dim, num_pages=(wl.num_pages if k_pages is None
                                        else k_pages.shape[0]),
        max_blocks_per_seq=bt_np.shape[1], seq_lens_host=wl.seq_lens,
        softmax_scale=wl.softmax_scale, kv_dtype=c.kv_dtype,
        k_scale=wl.k_scale, v_scale=wl.v_scale,
        pages_per_item=pages_per_item, waves_per_item=waves_per_item,
        **(dict(zip(("group_of", "group_pages"), prefix_groups(wl)))
           if cascade else {}))
    if cascade and (waves_per_item or 4) * (16 // (c.num_q_heads //
                                                   c.num_kv_heads)) >= 2:
        # one item holds waves x (16 / g) members; a chunk needs two
        assert N_cascade_units(att) > 0, "the cascade plan decodes no prefix"
    kp = wl.k_pages if k_pages is None else k_pages
    vp = wl.v_pages if v_pages is None else v_pages
    # NaN-filled outputs: a row the kernels skip cannot pass as a stale value
    out, lse = att.outputs(fill=float("nan"))
    if two_phase:
        att.partial(wl.q, kp, vp, bt, lens, out, lse)
        att.merge(out, lse)
    else:
        att(wl.q, kp, vp, bt, lens, out, lse)
    torch.cuda.synchronize()
    res = out.cpu().numpy(), lse.cpu().numpy()
    att.close()
    return res


def N_cascade_units(att):
    from paper_2510_12633_amd import _native as N
    return int(N.lib().laminar_plan_num_cascade_units(att.plan))


def check(gpu, ref, what, seqs=None):
    out, lse = gpu
    ro, rl = ref
    if seqs is not None:
        out, lse = out[seqs], lse[seqs]
    assert np.isfinite(out).all() and np.isfinite(lse[np.isfinite(rl)]).all(), what
    eo = np.abs(out - ro).max() if out.size else 0.0
    fin = np.isfinite(rl)
    assert np.array_equal(np.isneginf(lse), np.isneginf(rl)), what
    el = np.abs(lse[fin] - rl[fin]).max() if fin.any() else 0.0
    _say(f"{what}: max|out err| {eo:.2e}  max|lse err| {el:.2e}")
    assert eo <= TOL and el <= TOL, (what, eo, el)
    return eo, el


CUSTOM = [
    ("g7_d128_ragged", custom_config([1, 15, 16, 17, 31, 32, 33, 1000, 4097, 9],
                                     28, 4, 128)),
    ("g5_d128_fp8", custom_config([1, 5, 16, 17, 250, 700, 3001], 40, 8, 128,
                                  kv_dtype="fp8_e4m3fn")),
    ("g16_d64", custom_config([3, 64, 100, 513], 32, 2, 64)),
    ("g1_d128_mha", custom_config([40, 7, 300], 4, 4, 128)),
    ("g8_d128_prefix", custom_config([10, 400, 1500, 64, 3, 2000, 1100, 90],
                                     16, 2, 128, prefix_group=4,
                                     prefix_tokens=1024)),
    ("g4_d64_fp8_empty", custom_config([0, 17, 0, 64], 8, 2, 64,
                                       kv_dtype="fp8_e4m3fn")),
    ("g8_d64_odd_pages", custom_config([16 * 3, 16 * 5 + 1, 16 * 7 - 1], 8, 1, 64)),
]


CASCADE = [
    ("g8_d128_prefix1024", custom_config([10, 400, 1500, 64, 3, 2000, 1100, 90],
                                         16, 2, 128, prefix_group=4,
                                         prefix_tokens=1024)),
    ("g8_d128_16members", custom_config(
        [0, 5, 511, 512, 513, 1024, 3000, 77, 600, 512, 9000, 1, 256, 700,
         2048, 40, 1200, 300], 32, 4, 128, prefix_group=16, prefix_tokens=512)),
    ("g5_d128_fp8", custom_config([100, 257, 3000, 20, 256, 999], 40, 8, 128,
                                  kv_dtype="fp8_e4m3fn", prefix_group=3,
                                  prefix_tokens=256)),
    ("g16_d64", custom_config([64, 300, 31, 800, 2000, 65, 5], 16, 1, 64,
                              prefix_group=6, prefix_tokens=320)),
    ("g1_d64_mha", custom_config([50, 700, 130, 129, 128, 1000], 2, 2, 64,
                                 prefix_group=6, prefix_tokens=128)),
    ("g7_d128", custom_config([2100, 2048, 100, 5000, 2047, 4000, 2049, 1],
                              28, 4, 128, prefix_group=8, prefix_tokens=2048)),
]


@pytest.mark.parametrize("name,cfg", CASCADE, ids=[c[0] for c in CASCADE])
def test_cascade_shapes(name, cfg):
    """Shared prefixes decoded once per group: members shorter than, equal
    to and longer than the prefix, empty members, groups larger than one
    item, prefix pieces split. Against the oracle at the bar, and against
    the plain plan within 1e-5."""
    _need_gpu()
    wl = make_workload(cfg, seed=17, device="cuda")
    ref = decode_attention_from_host(host_arrays(wl), workers=4)
    plain = run_gpu(wl)
    for ppi in (0, 2, 6):
        for waves in (1, 2, 4):
            o, l = run_gpu(wl, pages_per_item=ppi, waves_per_item=waves,
                           cascade=True)
            check((o, l), ref,
                  f"{name} cascade waves={waves} pages_per_item={ppi}")
            fin = np.isfinite(plain[1])
            assert np.abs(o - plain[0]).max() <= 1e-5
            assert np.abs(l[fin] - plain[1][fin]).max() <= 1e-5


def test_cascade_run_to_run_bitwise():
    _need_gpu()
    wl = make_workload(CASCADE[1][1], seed=3, device="cuda")
    a = run_gpu(wl, cascade=True)
    b = run_gpu(wl, cascade=True)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_dynamic_tail_repeated_launches_bitwise():
    """One plan launched five times: the tail counter is reset by each
    launch's last pull, so every launch computes every item once and the
    results are bitwise identical (the items' arithmetic does not depend on
    which workgroup runs them)."""
    from paper_2510_12633_amd import _native as N
    from paper_2510_12633_amd.api import PagedDecodeAttention
    _need_gpu()
    wl = make_workload(get_config(2), device="cuda")
    c = wl.cfg
    att = PagedDecodeAttention(
        batch=wl.batch, num_q_heads=c.num_q_heads, num_kv_heads=c.num_kv_heads,
        head_dim=c.head_dim, num_pages=wl.num_pages,
        max_blocks_per_seq=wl.block_table.shape[1], seq_lens_host=wl.seq_lens,
        softmax_scale=wl.softmax_scale)
    assert N.lib().laminar_plan_num_dynamic_items(att.plan) > 0
    bt = torch.as_tensor(wl.block_table, device="cuda")
    lens = torch.as_tensor(wl.seq_lens, device="cuda")
    runs = []
    out, lse = att.outputs()
    for _ in range(5):
        # every launch starts from NaN: an item a launch skipped would show
        out.fill_(float("nan"))
        lse.fill_(float("nan"))
        att(wl.q, wl.k_pages, wl.v_pages, bt, lens, out, lse)
        torch.cuda.synchronize()
        runs.append((out.cpu().numpy(), lse.cpu().numpy()))
        assert np.isfinite(runs[-1][0]).all() and np.isfinite(runs[-1][1]).all()
    for o, l in runs[1:]:
        assert np.array_equal(o, runs[0][0]) and np.array_equal(l, runs[0][1])
    ref = decode_attention_from_host(host_arrays(wl), workers=_host_workers())
    check(runs[-1], ref, "7b_pre_repack dynamic tail, 5th launch, all trajectories")
    att.close()


@pytest.mark.parametrize("cascade", [False, True])
def test_strided_q_equals_contiguous(cascade):
    """q read as a view into a fused QKV projection's output (rows
    (Hq + 2 Hkv) D elements apart) gives bit-identical out and lse."""
    from paper_2510_12633_amd.api import PagedDecodeAttention
    _need_gpu()
    name, cfg = CASCADE[1] if cascade else CUSTOM[0]
    wl = make_workload(cfg, seed=11, device="cuda")
    c = wl.cfg
    hq, hkv, d = c.num_q_heads, c.num_kv_heads, c.head_dim
    row = (hq + 2 * hkv) * d
    qkv = torch.full((wl.batch, row), float("nan"), dtype=torch.bfloat16,
                     device="cuda")
    qkv[:, :hq * d] = wl.q.reshape(wl.batch, hq * d)
    q_view = qkv[:, :hq * d].view(wl.batch, hq, d)
    bt = torch.as_tensor(wl.block_table, device="cuda")
    lens = torch.as_tensor(wl.seq_lens, device="cuda")
    res = []
    for q, stride in ((wl.q, 0), (q_view, row)):
        att = PagedDecodeAttention(
            batch=wl.batch, num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
            num_pages=wl.num_pages, max_blocks_per_seq=wl.block_table.shape[1],
            seq_lens_host=wl.seq_lens, softmax_scale=wl.softmax_scale,
            q_row_stride=stride,
            **(dict(zip(("group_of", "group_pages"), prefix_groups(wl)))
               if cascade else {}))
        out, lse = att(q, wl.k_pages, wl.v_pages, bt, lens)
        torch.cuda.synchronize()
        res.append((out.cpu().numpy(), lse.cpu().numpy()))
        att.close()
    assert np.array_equal(res[0][0], res[1][0]), name
    assert np.array_equal(res[0][1], res[1][1]), name


def test_distinct_plans_on_two_streams():
    """Two plans with their own workspaces, bound and run on two streams at
    once (the staging ring of the uploads is shared), give the same bits as
    running them one after the other."""
    from paper_2510_12633_amd.api import PagedDecodeAttention
    _need_gpu()
    wls = [make_workload(CUSTOM[0][1], seed=21, device="cuda"),
           make_workload(CUSTOM[1][1], seed=22, device="cuda")]

    def make(wl, stream):
        c = wl.cfg
        return PagedDecodeAttention(
            batch=wl.batch, num_q_heads=c.num_q_heads,
            num_kv_heads=c.num_kv_heads, head_dim=c.head_dim,
            num_pages=wl.num_pages, max_blocks_per_seq=wl.block_table.shape[1],
            seq_lens_host=wl.seq_lens, softmax_scale=wl.softmax_scale,
            kv_dtype=c.kv_dtype, k_scale=wl.k_scale, v_scale=wl.v_scale,
            pages_per_item=2, stream=stream)

    def run(wl, att, stream):
        bt = torch.as_tensor(wl.block_table, device="cuda")
        lens = torch.as_tensor(wl.seq_lens, device="cuda")
        return att(wl.q, wl.k_pages, wl.v_pages, bt, lens, stream=stream)

    seq = []
    for wl in wls:
        att = make(wl, None)
        o, l = run(wl, att, None)
        torch.cuda.synchronize()
        seq.append((o.cpu().numpy(), l.cpu().numpy()))
        att.close()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for rep in range(3):
        atts = [make(wl, s) for wl, s in zip(wls, streams)]
        outs = [run(wl, att, s) for wl, att, s in zip(wls, atts, streams)]
        torch.cuda.synchronize()
        for (o, l), (so, sl) in zip(outs, seq):
            assert np.array_equal(o.cpu().numpy(), so)
            assert np.array_equal(l.cpu().numpy(), sl)
        for att in atts:
            att.close()


def test_empty_batches():
    """batch 0 is a no-op; a batch whose trajectories are all empty gives
    out = 0 and lse = -inf (the merge identity) for every head."""
    from paper_2510_12633_amd import _native as N
    from paper_2510_12633_amd.api import PagedDecodeAttention
    _need_gpu()
    att = PagedDecodeAttention(
        batch=0, num_q_heads=8, num_kv_heads=2, head_dim=128, num_pages=1,
        max_blocks_per_seq=1, seq_lens_host=np.zeros(0, np.int32),
        softmax_scale=0.1)
    assert att.num_items == 0
    N.laminar_decode_attn(att.plan, None, None, None, None, None, None, None,
                          torch.cuda.current_stream().cuda_stream)
    att.close()
    wl = make_workload(custom_config([0, 0, 0], 16, 2, 64), device="cuda")
    o, l = run_gpu(wl)
    assert np.array_equal(o, np.zeros_like(o)) and np.isneginf(l).all()
    o, l = run_gpu(wl, pages_per_item=1, waves_per_item=1)
    assert np.array_equal(o, np.zeros_like(o)) and np.isneginf(l).all()


def test_tiny_config_all_outputs():
    _need_gpu()
    wl = make_workload(1, device="cuda")
    ref = decode_attention_from_host(host_arrays(wl))
    for ppi in (0, 1, 4, 64):
        for waves in (1, 2, 4):
            check(run_gpu(wl, pages_per_item=ppi, waves_per_item=waves), ref,
                  f"tiny waves={waves} pages_per_item={ppi}")
    check(run_gpu(wl, two_phase=True), ref, "tiny partial+merge")


@pytest.mark.parametrize("name,cfg", CUSTOM, ids=[c[0] for c in CUSTOM])
def test_custom_shapes(name, cfg):
    _need_gpu()
    wl = make_workload(cfg, seed=31, device="cuda")
    ref = decode_attention_from_host(host_arrays(wl), workers=4)
    for ppi in (0, 2, 5):
        for waves in (1, 2, 4):
            check(run_gpu(wl, pages_per_item=ppi, waves_per_item=waves), ref,
                  f"{name} waves={waves} pages_per_item={ppi}")


def test_forced_split_independence():
    _need_gpu()
    wl = make_workload(custom_config([5000, 777, 12000, 33], 28, 4, 128),
                       seed=5, device="cuda")
    base = run_gpu(wl, pages_per_item=100000)
    for waves in (1, 4):
        for ppi in (1, 2, 7, 64):
            o, l = run_gpu(wl, pages_per_item=ppi, waves_per_item=waves)
            eo = np.abs(o - base[0]).max()
            el = np.abs(l - base[1]).max()
            _say(f"waves {waves} split {ppi} vs unsplit: {eo:.2e} {el:.2e}")
            assert eo <= 1e-5 and el <= 1e-5


def test_no_rescale_drift_on_long_single_wave_items():
    """One wavefront over thousands of pages: the running-max rescale must be
    exactly 1 while the max is unchanged, or lse drifts by ~n_pairs * 2e-7
    (out cancels, lse does not). Bound far tighter than the 1e-3 bar."""
    _need_gpu()
    wl = make_workload(custom_config([12000, 5000], 28, 4, 128), seed=5,
                       device="cuda")
    ro, rl = decode_attention_from_host(host_arrays(wl), workers=4)
    for kw in (dict(waves_per_item=1), dict(waves_per_item=4)):
        o, l = run_gpu(wl, pages_per_item=1 << 20, **kw)
        el = np.abs(l - rl).max()
        eo = np.abs(o - ro).max()
        _say(f"unsplit single wave {kw}: lse err {el:.2e} out err {eo:.2e}")
        assert el <= 5e-6 and eo <= 2e-5


def test_page_permutation_bitwise():
    _need_gpu()
    wl = make_workload(custom_config([33, 200, 513, 16, 3000], 28, 4, 128),
                       seed=2, device="cuda")
    base = run_gpu(wl)
    p = wl.num_pages
    perm = torch.randperm(p, generator=torch.Generator().manual_seed(0))
    kp = torch.empty_like(wl.k_pages)
    vp = torch.empty_like(wl.v_pages)
    kp[perm.to(kp.device)] = wl.k_pages
    vp[perm.to(vp.device)] = wl.v_pages
    permn = perm.numpy()
    bt = wl.block_table
    bt2 = np.where(bt >= 0, permn[np.maximum(bt, 0)], -1).astype(np.int32)
    o2, l2 = run_gpu(wl, block_table=bt2, k_pages=kp, v_pages=vp)
    assert np.array_equal(base[0], o2) and np.array_equal(base[1], l2)


def test_prefix_alias_equals_copy_bitwise():
    _need_gpu()
    cfg = custom_config([10, 400, 1500, 64, 3, 2000, 1100, 90], 16, 2, 128,
                        prefix_group=4, prefix_tokens=1024)
    wl = make_workload(cfg, seed=13, device="cuda")
    base = run_gpu(wl)
    bt = wl.block_table.copy()
    extra = []
    nxt = wl.num_pages
    seen = set()
    for b in range(bt.shape[0]):
        for j in range(bt.shape[1]):
            p = int(bt[b, j])
            if p < 0:
                continue
            if p in seen:
                extra.append(p)
                bt[b, j] = nxt
                nxt += 1
            seen.add(p)
    idx = torch.as_tensor(extra, device=wl.k_pages.device)
    kp = torch.cat([wl.k_pages, wl.k_pages[idx]])
    vp = torch.cat([wl.v_pages, wl.v_pages[idx]])
    o2, l2 = run_gpu(wl, block_table=bt, k_pages=kp, v_pages=vp)
    assert np.array_equal(base[0], o2) and np.array_equal(base[1], l2)


def test_run_to_run_bitwise():
    _need_gpu()
    wl = make_workload(custom_config([5000, 777, 33, 12000], 40, 8, 128,
                                     kv_dtype="fp8_e4m3fn"), seed=8,
                       device="cuda")
    a = run_gpu(wl)
    b = run_gpu(wl)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_single_long_trajectory():
    """B = 1 with the longest length of the agentic mix (98304 tokens)."""
    _need_gpu()
    wl = make_workload(custom_config([98304], 64, 8, 128), seed=17,
                       device="cuda")
    ref = decode_attention_from_host(host_arrays(wl), workers=8)
    check(run_gpu(wl), ref, "B=1 n=98304 auto split")
    check(run_gpu(wl, pages_per_item=1 << 20, waves_per_item=4), ref,
          "B=1 n=98304 unsplit, 4 waves")
    check(run_gpu(wl, pages_per_item=1 << 20, waves_per_item=1), ref,
          "B=1 n=98304 unsplit, 1 wave")


def test_invalid_arguments_return_status():
    _need_gpu()
    from paper_2510_12633_amd import _native as N
    from paper_2510_12633_amd.api import PagedDecodeAttention
    wl = make_workload(1, device="cuda")
    bt = torch.as_tensor(wl.block_table, device="cuda")
    lens = torch.as_tensor(wl.seq_lens, device="cuda")
    att = PagedDecodeAttention(
        batch=4, num_q_heads=4, num_kv_heads=1, head_dim=64, num_pages=64,
        max_blocks_per_seq=bt.shape[1], seq_lens_host=wl.seq_lens,
        softmax_scale=wl.softmax_scale)
    out, lse = att.outputs()
    with pytest.raises(N.LaminarError) as e:
        N.laminar_decode_attn(att.plan, None, wl.k_pages, wl.v_pages, bt, lens,
                              out, lse, 0)
    assert e.value.status == N.LAMINAR_ERR_INVALID_ARG
    with pytest.raises(N.LaminarError) as e:
        N.laminar_decode_attn(None, wl.q, wl.k_pages, wl.v_pages, bt, lens,
                              out, lse, 0)
    assert e.value.status == N.LAMINAR_ERR_INVALID_ARG
    small = torch.empty(64, dtype=torch.uint8, device="cuda")
    with pytest.raises(N.LaminarError) as e:
        N.laminar_plan_bind_workspace(att.plan, small, 64, 0)
    assert e.value.status == N.LAMINAR_ERR_WORKSPACE
    # an unbound plan refuses to launch
    plan = N.laminar_plan_create(att.desc, wl.seq_lens, 256)
    with pytest.raises(N.LaminarError) as e:
        N.laminar_decode_attn(plan, wl.q, wl.k_pages, wl.v_pages, bt, lens,
                              out, lse, 0)
    assert e.value.status == N.LAMINAR_ERR_WORKSPACE
    N.laminar_plan_destroy(plan)
    att.close()


def _host_workers():
    return max(1, min(16, len(os.sched_getaffinity(0))))


@pytest.mark.parametrize("idx,cascade", [(2, False), (3, False), (4, False),
                                         (5, False), (5, True), (6, False),
                                         (7, True), (7, False)])
def test_full_size_config_every_trajectory(idx, cascade):
    """Full-size batch in the bench's launch configuration (automatic split,
    four wavefronts per item, cascade plan where the workload shares
    prefixes), outputs NaN-filled before the launch, and every trajectory
    and head compared with the fp64 oracle at the bar."""
    _need_gpu()
    cfg = get_config(idx)
    _say(f"generating {cfg.name}")
    wl = make_workload(cfg, device="cuda")
    out, lse = run_gpu(wl, cascade=cascade)
    _say(f"{cfg.name}: oracle over all {wl.batch} trajectories, "
         f"{_host_workers()} threads")
    ref = decode_attention_from_host(host_arrays(wl), workers=_host_workers())
    check((out, lse), ref, f"{cfg.name}{' cascade' if cascade else ''} "
          f"all {wl.batch} trajectories")
    del wl
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name,cfg", [
    ("g7_d128_bf16", custom_config([1, 17, 300, 5000, 40000], 28, 4, 128)),
    ("g5_d128_fp8", custom_config([2, 33, 999, 7000], 40, 8, 128,
                                  kv_dtype="fp8_e4m3fn")),
    ("g16_d64_bf16", custom_config([5, 64, 2500], 32, 2, 64)),
], ids=lambda v: v if isinstance(v, str) else "")
def test_extreme_score_ranges(name, cfg):
    """Scores far outside exp's fp32 range (q scaled by 100: |s| up to a
    few hundred, a sharply peaked softmax) and all-zero scores (q = 0: the
    softmax is uniform, out is the mean of V and lse = ln n exactly)."""
    _need_gpu()
    wl = make_workload(cfg, seed=23, device="cuda")
    q0 = wl.q.clone()
    for factor in (100.0, 0.0):
        wl.q.copy_((q0.float() * factor).to(wl.q.dtype))
        ref = decode_attention_from_host(host_arrays(wl), workers=8)
        out, lse = run_gpu(wl)
        check((out, lse), ref, f"{name} q x {factor:g}")
        if factor == 0.0:
            n = np.repeat(wl.seq_lens.astype(np.float64), cfg.num_q_heads)
            assert np.allclose(lse.reshape(-1), np.log(n), atol=1e-4, rtol=0)


def _random_case(seed):
    """A seeded random decode-attention problem: batch, head layout,
    head_dim, dtype, ragged lengths with the page-boundary and empty cases,
    forced split size, wavefronts per item and, for some, shared prefixes."""
    rng = np.random.default_rng(1000 + seed)
    hkv = int(rng.choice([1, 2, 4, 8]))
    g = int(rng.integers(1, 17))
    d = int(rng.choice([64, 128]))
    kv = "fp8_e4m3fn" if rng.random() < 0.4 else "bf16"
    b = int(rng.integers(1, 33))
    special = [0, 1, 15, 16, 17, 31, 32, 33, 255, 256, 257]
    lens = [int(rng.choice(special)) if rng.random() < 0.35
            else int(rng.integers(1, 2500)) for _ in range(b)]
    prefix = {}
    if rng.random() < 0.35 and b >= 2:
        prefix = dict(prefix_group=int(rng.integers(2, min(b, 9) + 1)),
                      prefix_tokens=16 * int(rng.integers(1, 40)))
    cfg = custom_config(lens, g * hkv, hkv, d, kv_dtype=kv, **prefix)
    ppi = int(rng.choice([0, 0, 1, 2, 3, 8, 33]))
    waves = int(rng.choice([0, 1, 2, 4]))
    return cfg, ppi, waves, bool(prefix)


@pytest.mark.parametrize("seed", range(24))
def test_random_shapes(seed):
    """Seeded random problems (see _random_case) through the C ABI into
    NaN-filled outputs, every trajectory and head against the oracle at the
    bar; problems with shared prefixes also through the cascade plan."""
    _need_gpu()
    cfg, ppi, waves, has_prefix = _random_case(seed)
    _say(f"random {seed}: B={cfg.batch} Hq={cfg.num_q_heads} Hkv={cfg.num_kv_heads} "
         f"D={cfg.head_dim} {cfg.kv_dtype} ppi={ppi} waves={waves} "
         f"prefix={has_prefix}")
    wl = make_workload(cfg, seed=seed, device="cuda")
    ref = decode_attention_from_host(host_arrays(wl), workers=_host_workers())
    check(run_gpu(wl, pages_per_item=ppi, waves_per_item=waves), ref,
          f"random {seed}")
    if has_prefix:
        check(run_gpu(wl, pages_per_item=ppi, waves_per_item=waves,
                      cascade=True), ref, f"random {seed} cascade")
