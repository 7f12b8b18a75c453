"""The allocation-free entry point (laminar_decode_attn_static, the
library's static per-GPU workspace) against laminar_decode_attn with a
bound, caller-allocated workspace: the same plans, NaN-filled outputs, two
calls in a row (the second on a smaller batch, whose tables and partial
results overwrite only the front of what the first left), results equal
bit for bit and within the bar of the fp64 oracle."""
import os

import numpy as np
import pytest
import torch

from oracle import decode_attention_from_host
from paper_2510_12633_amd import _native as N
from paper_2510_12633_amd.api import PagedDecodeAttention
from workloads import (custom_config, get_config, host_arrays, make_workload,
                       prefix_groups)

pytestmark = pytest.mark.gpu

TOL = 1e-3


def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")


def _both(wl, cascade=False):
    """(out, lse) of laminar_decode_attn on a bound plan and of
    laminar_decode_attn_static on an unbound plan of the same batch."""
    c = wl.cfg
    kw = dict(zip(("group_of", "group_pages"), prefix_groups(wl))) if cascade else {}
    att = PagedDecodeAttention(
        batch=wl.batch, num_q_heads=c.num_q_heads, num_kv_heads=c.num_kv_heads,
        head_dim=c.head_dim, num_pages=wl.num_pages,
        max_blocks_per_seq=wl.block_table.shape[1], seq_lens_host=wl.seq_lens,
        softmax_scale=wl.softmax_scale, kv_dtype=c.kv_dtype,
        k_scale=wl.k_scale, v_scale=wl.v_scale, **kw)
    bt = torch.as_tensor(wl.block_table, device="cuda")
    lens = torch.as_tensor(wl.seq_lens, device="cuda")
    h = torch.cuda.current_stream().cuda_stream
    o1, l1 = att.outputs()
    N.laminar_decode_attn(att.plan, wl.q, wl.k_pages, wl.v_pages, bt, lens,
                          o1, l1, h)
    if cascade:
        plan = N.laminar_plan_create_cascade(att.desc, wl.seq_lens, kw["group_of"],
                                             kw["group_pages"], 256)
    else:
        plan = N.laminar_plan_create(att.desc, wl.seq_lens, 256)
    assert N.laminar_plan_workspace_bytes(plan) <= 64 << 20
    o2, l2 = att.outputs()
    N.laminar_decode_attn_static(plan, wl.q, wl.k_pages, wl.v_pages, bt, lens,
                                 o2, l2, h)
    torch.cuda.synchronize()
    N.laminar_plan_destroy(plan)
    att.close()
    return ((o1.cpu().numpy(), l1.cpu().numpy()),
            (o2.cpu().numpy(), l2.cpu().numpy()))


def _check(wl, cascade, what):
    print(f"[no-alloc] {what}: batch {wl.batch}", flush=True)
    (o1, l1), (o2, l2) = _both(wl, cascade)
    assert np.isfinite(o2).all(), what
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2), what
    ro, rl = decode_attention_from_host(
        host_arrays(wl), workers=max(1, min(16, len(os.sched_getaffinity(0)))))
    fin = np.isfinite(rl)
    assert np.array_equal(np.isneginf(l2), np.isneginf(rl)), what
    eo = float(np.abs(o2 - ro).max())
    el = float(np.abs(l2[fin] - rl[fin]).max()) if fin.any() else 0.0
    print(f"[no-alloc] {what}: max|out err| {eo:.2e}  max|lse err| {el:.2e}",
          flush=True)
    assert eo <= TOL and el <= TOL, (what, eo, el)


def test_static_workspace_two_calls_second_smaller():
    """7b_pre_repack (dynamic tail: the counter comes in with the tables),
    then a small fp8 batch with empty trajectories."""
    _need_gpu()
    _check(make_workload(get_config(2), device="cuda"), False, "7b_pre_repack")
    _check(make_workload(custom_config([0, 5, 17, 250, 0, 3001], 40, 8, 128,
                                       kv_dtype="fp8_e4m3fn"), seed=41,
                         device="cuda"), False, "fp8 ragged")


def test_static_workspace_cascade_then_tiny():
    """A cascade plan (shared-prefix tables) of the TP-8 agentic share,
    then the tiny workload."""
    _need_gpu()
    _check(make_workload(get_config("agentic_mix_tp8"), device="cuda"), True,
           "agentic_mix_tp8 cascade")
    _check(make_workload(get_config(1), device="cuda"), False, "tiny")


def test_static_workspace_refuses_a_plan_too_large():
    """A plan whose workspace exceeds the static maximum returns WORKSPACE
    before any launch."""
    d = N.LaminarAttnDesc(batch=1, num_q_heads=16, num_kv_heads=1, head_dim=128,
                          page_size=16, num_pages=1 << 20,
                          max_blocks_per_seq=1 << 14, kv_dtype=N.LAMINAR_KV_BF16,
                          softmax_scale=0.1, k_scale=None, v_scale=None,
                          pages_per_item=1, waves_per_item=0, input_row_stride=0)
    plan = N.laminar_plan_create(d, np.array([16 << 14], np.int32), 256)
    try:
        assert N.laminar_plan_workspace_bytes(plan) > 64 << 20
        st = N.lib().laminar_decode_attn_static(plan, *([4096] * 7), None)
        assert st == N.LAMINAR_ERR_WORKSPACE
    finally:
        N.laminar_plan_destroy(plan)
