"""GPU parity of the KV append: the HIP kernel through its C ABI against the
CPU oracle.

Bar: bit-exact pools and scales (the append is byte work; fp32 decides the
fp8 codes on both sides with the same operations). Then attention over the
appended pools is checked against the attention oracle at the 1e-3 bar.
"""
import numpy as np
import pytest
import torch

from oracle import decode_attention, kv_append
from workloads import custom_config, get_config, make_decode_run, make_workload

pytestmark = pytest.mark.gpu

TOL = 1e-3


def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")


def _say(msg):
    print(f"[gpu-append] {msg}", flush=True)


def host(t):
    if t is None:
        return None
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def gpu_append(run, step, kp, vp, ks, vs):
    from paper_2510_12633_amd.api import kv_append as gpu_kv_append
    dev = kp.device
    bt = torch.as_tensor(run.block_table, device=dev)
    lens = torch.as_tensor(run.lens_after(step), device=dev)
    gpu_kv_append(run.k_new[step], run.v_new[step], bt, lens, kp, vp, ks, vs,
                  kv_dtype=run.base.cfg.kv_dtype)


def oracle_steps(run, steps, arrays):
    kp, vp, ks, vs = arrays
    bt = run.block_table
    c = run.base.cfg
    for i in steps:
        kp, vp, ks, vs = kv_append(
            kp, vp, ks, vs, bt, run.lens_after(i), host(run.k_new[i]),
            host(run.v_new[i]), head_dim=c.head_dim,
            num_kv_heads=c.num_kv_heads, kv_dtype=c.kv_dtype)
    return kp, vp, ks, vs


def assert_same(got, want, what):
    got, want = np.asarray(got), np.asarray(want)
    if got.dtype == np.float32:                  # scales: NaN poison equal too
        same = (got.view(np.uint32) == want.view(np.uint32))
    else:
        same = got == want
    bad = np.argwhere(~same)
    assert bad.size == 0, f"{what}: {bad.shape[0]} differing elements, first {bad[:3]}"


CASES = [
    ("bf16_d64_g4", custom_config([0, 1, 15, 16, 17, 40, 200], 4, 1, 64)),
    ("bf16_d128_hkv4", custom_config([3, 16, 31, 33, 500], 28, 4, 128)),
    ("fp8_d128_hkv8", custom_config([0, 1, 5, 16, 17, 250, 700], 40, 8, 128,
                                    kv_dtype="fp8_e4m3fn")),
    ("fp8_d64_hkv2", custom_config([2, 14, 15, 16, 48, 100], 4, 2, 64,
                                   kv_dtype="fp8_e4m3fn")),
]


@pytest.mark.parametrize("mix", ["normal", "stress", "ties"])
@pytest.mark.parametrize("name,cfg", CASES, ids=[c[0] for c in CASES])
def test_append_bit_exact_over_a_decode_run(name, cfg, mix):
    """40 decode steps (pages fill, new pages start, fp8 scales grow and
    re-encode), compared in full after steps 1, 17 and 40."""
    _need_gpu()
    if cfg.kv_dtype == "bf16" and mix != "normal":
        pytest.skip("bf16 appends copy codes; the mixes only matter for fp8")
    _say(f"case {name} mix {mix}")
    wl = make_workload(cfg, seed=21, device="cuda")
    run = make_decode_run(wl, steps=40, seed=5, mix=mix)
    kp, vp = run.k_pages.clone(), run.v_pages.clone()
    ks = None if run.k_scale is None else run.k_scale.clone()
    vs = None if run.v_scale is None else run.v_scale.clone()
    ref = (host(kp), host(vp), host(ks), host(vs))
    done = 0
    for upto in (1, 17, 40):
        for i in range(done, upto):
            gpu_append(run, i, kp, vp, ks, vs)
        torch.cuda.synchronize()
        ref = oracle_steps(run, range(done, upto), ref)
        done = upto
        assert_same(host(kp), ref[0], f"{name}/{mix} K after {upto}")
        assert_same(host(vp), ref[1], f"{name}/{mix} V after {upto}")
        if ks is not None:
            assert_same(host(ks), ref[2], f"{name}/{mix} K scale after {upto}")
            assert_same(host(vs), ref[3], f"{name}/{mix} V scale after {upto}")
    _say(f"{name}/{mix}: bit-exact after 40 steps")


@pytest.mark.parametrize("mix", ["normal", "stress"])
@pytest.mark.parametrize("name,cfg", CASES[1:3], ids=[c[0] for c in CASES[1:3]])
def test_attention_after_appends_matches_oracle(name, cfg, mix):
    """append x 20 on the GPU, then decode attention on the GPU, against the
    oracle's appends followed by the attention oracle.

    Bar: 1e-3 for N(0, 1) values. The stress mix scales some tokens by 300,
    so outputs reach the hundreds; there the kernel's P (fp32, times the fp8
    V scale, carried as a bf16 hi + lo pair: 16 significant bits) bounds the
    error by about 2^-16 * max|V| per output, and the bar is
    max(1e-3, 2^-14 * max|V|)."""
    from paper_2510_12633_amd.api import PagedDecodeAttention
    _need_gpu()
    wl = make_workload(cfg, seed=3, device="cuda")
    run = make_decode_run(wl, steps=20, seed=8, mix=mix)
    kp, vp = run.k_pages.clone(), run.v_pages.clone()
    ks = None if run.k_scale is None else run.k_scale.clone()
    vs = None if run.v_scale is None else run.v_scale.clone()
    ref = (host(kp), host(vp), host(ks), host(vs))
    for i in range(run.steps):
        gpu_append(run, i, kp, vp, ks, vs)
    ref = oracle_steps(run, range(run.steps), ref)
    lens = run.lens_after(run.steps - 1)
    c = cfg
    att = PagedDecodeAttention(
        batch=wl.batch, num_q_heads=c.num_q_heads, num_kv_heads=c.num_kv_heads,
        head_dim=c.head_dim, num_pages=run.num_pages,
        max_blocks_per_seq=run.block_table.shape[1], seq_lens_host=lens,
        softmax_scale=wl.softmax_scale, kv_dtype=c.kv_dtype, k_scale=ks,
        v_scale=vs)
    out, lse = att(wl.q, kp, vp, torch.as_tensor(run.block_table, device="cuda"),
                   torch.as_tensor(lens, device="cuda"))
    torch.cuda.synchronize()
    ro, rl = decode_attention(host(wl.q), ref[0], ref[1], run.block_table, lens,
                              head_dim=c.head_dim, num_kv_heads=c.num_kv_heads,
                              kv_dtype=c.kv_dtype, softmax_scale=wl.softmax_scale,
                              k_scale=ref[2], v_scale=ref[3])
    eo = np.abs(out.cpu().numpy() - ro).max()
    el = np.abs(lse.cpu().numpy() - rl).max()
    vmax = float(np.abs(run.v_new.float().cpu().numpy()).max())
    tol = TOL if mix == "normal" else max(TOL, 2.0 ** -14 * vmax)
    _say(f"{name}/{mix}: attention after appends max|out err| {eo:.2e} "
         f"max|lse err| {el:.2e} (out bar {tol:.1e})")
    assert eo <= tol and el <= TOL
    att.close()


def _sub_run_arrays(run, kp, vp, ks, vs, seqs):
    """Host copies of the pages the trajectories ``seqs`` use (through the
    end of the run), with their block-table rows renumbered."""
    table = run.block_table[seqs]
    used = np.unique(table[table >= 0]).astype(np.int64)
    remap = np.full(run.num_pages, -1, np.int64)
    remap[used] = np.arange(used.size)
    sub = np.where(table >= 0, remap[np.maximum(table, 0)], -1).astype(np.int32)
    sel = torch.as_tensor(used, device=kp.device)
    pick = lambda t: None if t is None else host(t.index_select(0, sel))
    return (pick(kp), pick(vp), pick(ks), pick(vs)), sub, used


@pytest.mark.parametrize("config", ["32b_fp8", "7b_pre_repack"])
def test_append_full_size_every_trajectory(config):
    """Three decode steps on a full-size pool in one launch per step; the
    oracle replays them for every trajectory, and every page any trajectory
    references (K, V and fp8 scales) must match bit for bit."""
    _need_gpu()
    wl = make_workload(get_config(config), device="cuda")
    run = make_decode_run(wl, steps=3, seed=1, mix="stress")
    del wl
    kp, vp = run.k_pages, run.v_pages
    ks, vs = run.k_scale, run.v_scale
    seqs = np.arange(run.lens0.size)
    before, sub_table, used = _sub_run_arrays(run, kp, vp, ks, vs, seqs)
    for i in range(run.steps):
        gpu_append(run, i, kp, vp, ks, vs)
    torch.cuda.synchronize()
    after, _, _ = _sub_run_arrays(run, kp, vp, ks, vs, seqs)

    k_new = run.k_new[:, seqs]
    v_new = run.v_new[:, seqs]
    c = run.base.cfg
    kp_r, vp_r, ks_r, vs_r = before
    for i in range(run.steps):
        kp_r, vp_r, ks_r, vs_r = kv_append(
            kp_r, vp_r, ks_r, vs_r, sub_table, run.lens_after(i)[seqs],
            host(k_new[i]), host(v_new[i]), head_dim=c.head_dim,
            num_kv_heads=c.num_kv_heads, kv_dtype=c.kv_dtype)
    assert_same(after[0], kp_r, f"{config} K")
    assert_same(after[1], vp_r, f"{config} V")
    if ks_r is not None:
        assert_same(after[2], ks_r, f"{config} K scale")
        assert_same(after[3], vs_r, f"{config} V scale")
    _say(f"{config}: {seqs.size} trajectories bit-exact after {run.steps} steps")


def test_append_argument_errors_on_gpu():
    from paper_2510_12633_amd import _native as N
    _need_gpu()
    cfg = custom_config([5], 4, 1, 64, kv_dtype="fp8_e4m3fn")
    wl = make_workload(cfg, device="cuda")
    run = make_decode_run(wl, steps=1)
    d = N.LaminarAttnDesc(batch=1, num_q_heads=4, num_kv_heads=1, head_dim=64,
                          page_size=16, num_pages=run.num_pages,
                          max_blocks_per_seq=run.block_table.shape[1],
                          kv_dtype=N.LAMINAR_KV_FP8_E4M3FN, softmax_scale=1.0,
                          k_scale=None, v_scale=None, pages_per_item=0,
                          waves_per_item=0)
    bt = torch.as_tensor(run.block_table, device="cuda")
    lens = torch.as_tensor(run.lens_after(0), device="cuda")
    with pytest.raises(N.LaminarError) as e:
        N.laminar_kv_append(d, run.k_new[0], run.v_new[0], bt, lens,
                            run.k_pages, run.v_pages, None, run.v_scale, None)
    assert e.value.status == N.LAMINAR_ERR_INVALID_ARG
    N.laminar_kv_append(d, run.k_new[0], run.v_new[0], bt, lens, run.k_pages,
                        run.v_pages, run.k_scale, run.v_scale, None)
    torch.cuda.synchronize()


@pytest.mark.parametrize("name,cfg", CASES, ids=[c[0] for c in CASES])
def test_strided_rows_equal_contiguous(name, cfg):
    """k_new and v_new read as views into a fused QKV projection's output
    (rows input_row_stride elements apart) give bit-identical pools and
    scales to the contiguous call."""
    from paper_2510_12633_amd.api import kv_append as gpu_kv_append
    _need_gpu()
    wl = make_workload(cfg, seed=5, device="cuda")
    run = make_decode_run(wl, steps=3)
    c = wl.cfg
    hq, hkv, d = c.num_q_heads, c.num_kv_heads, c.head_dim
    bt = torch.as_tensor(run.block_table, device="cuda")

    def state():
        return [t.clone() if t is not None else None
                for t in (run.k_pages, run.v_pages, run.k_scale, run.v_scale)]

    plain, strided = state(), state()
    for step in range(run.steps):
        lens = torch.as_tensor(run.lens_after(step), device="cuda")
        b = run.k_new[step].shape[0]
        qkv = torch.full((b, (hq + 2 * hkv) * d), float("nan"),
                         dtype=torch.bfloat16, device="cuda")
        qkv[:, hq * d:(hq + hkv) * d] = run.k_new[step].reshape(b, hkv * d)
        qkv[:, (hq + hkv) * d:] = run.v_new[step].reshape(b, hkv * d)
        k_view = qkv[:, hq * d:(hq + hkv) * d].view(b, hkv, d)
        v_view = qkv[:, (hq + hkv) * d:].view(b, hkv, d)
        assert k_view.stride(0) == (hq + 2 * hkv) * d
        gpu_kv_append(run.k_new[step], run.v_new[step], bt, lens, *plain,
                      kv_dtype=c.kv_dtype)
        gpu_kv_append(k_view, v_view, bt, lens, *strided, kv_dtype=c.kv_dtype)
    torch.cuda.synchronize()
    for got, want, what in zip(strided, plain, ("K", "V", "K scale", "V scale")):
        if want is not None:
            assert_same(host(got), host(want), f"{name} strided {what}")
