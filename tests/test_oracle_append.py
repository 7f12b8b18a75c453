"""Pins of the KV-append oracle against things other than itself.

The rounding step is pinned to torch's float8_e4m3fn cast (a library
routine) over every code, every tie and random values; the page writes to
the workload generator's independent layout code and batch quantisation;
the scale update to a closed form (doubling re-encodes by one exponent step)
and to the batch definition of the scale; the re-encoding error to the
format's rounding bound.
"""
import numpy as np
import pytest
import torch

from oracle import (E4M3FN_TABLE, decode_attention, e4m3fn_round, kv_append,
                    quantize)
from oracle.kv_append import append_scale
from workloads import (custom_config, host_arrays, make_decode_run,
                       make_workload, to_page_format)
from workloads.generate import FP8_MAX


def bits16(t):
    return t.contiguous().view(torch.int16).numpy().view(np.uint16)


def torch_e4m3fn(y):
    return torch.as_tensor(np.asarray(y, np.float32)).to(
        torch.float8_e4m3fn).view(torch.uint8).numpy()


# ------------------------------------------------------------ rounding

def test_round_matches_torch_on_codes_ties_and_random():
    finite = E4M3FN_TABLE[np.isfinite(E4M3FN_TABLE)].astype(np.float32)
    mags = np.unique(np.abs(finite))
    mids = ((mags[:-1].astype(np.float64) + mags[1:]) / 2).astype(np.float32)
    rng = np.random.default_rng(0)
    rand = np.concatenate([
        rng.uniform(-448, 448, 20000), rng.normal(0, 1, 20000),
        rng.normal(0, 2 ** -8, 20000), rng.uniform(-2 ** -6, 2 ** -6, 20000),
    ]).astype(np.float32)
    for y in (finite, mids, -mids, rand, np.array([0.0, -0.0, 448, -448],
                                                   np.float32)):
        np.testing.assert_array_equal(e4m3fn_round(y), torch_e4m3fn(y))
    # every code's own value rounds back to that code (0x80 is -0)
    codes = np.arange(256)
    ok = np.isfinite(E4M3FN_TABLE)
    np.testing.assert_array_equal(
        e4m3fn_round(E4M3FN_TABLE[ok].astype(np.float32)), codes[ok])


def test_quantize_clamps_before_rounding():
    s = np.float32(0.5)
    x = np.array([224.0, 230.0, 1000.0, -1e6], np.float32)
    np.testing.assert_array_equal(quantize(x, s), [0x7E, 0x7E, 0x7E, 0xFE])


# ------------------------------------------------------------ bf16 pages

def test_bf16_appends_rebuild_the_generators_pages():
    """Appending every token of a few trajectories one at a time into
    poisoned pages gives the pool the generator lays out directly."""
    lens = [0, 1, 15, 16, 17, 40, 64]
    for hkv, d in ((1, 64), (2, 128)):
        cfg = custom_config(lens, num_q_heads=2 * hkv, num_kv_heads=hkv,
                            head_dim=d)
        wl = make_workload(cfg, seed=5, keep_logical=True)
        arrays = host_arrays(wl)
        kp = np.full_like(arrays["k_pages"], 0x7FC0)
        vp = np.full_like(arrays["v_pages"], 0x7FC0)
        bt = arrays["block_table"]
        k_log = wl.k_logical                                   # [P, Hkv, 16, D]
        v_log = wl.v_logical
        for step in range(max(lens)):
            cur = np.array([min(step + 1, n) for n in lens], np.int32)
            grow = np.array([step < n for n in lens])
            t = np.maximum(cur - 1, 0)
            pages = bt[np.arange(len(lens)), t // 16].astype(np.int64)
            k_new = bits16(k_log[pages, :, t % 16])             # [B, Hkv, D]
            v_new = bits16(v_log[pages, :, t % 16])
            run_lens = np.where(grow, cur, 0).astype(np.int32)
            kp, vp, _, _ = kv_append(kp, vp, None, None, bt, run_lens, k_new,
                                     v_new, head_dim=d, num_kv_heads=hkv,
                                     kv_dtype="bf16")
        want_k = bits16(to_page_format(k_log, "k"))
        want_v = bits16(to_page_format(v_log, "v"))
        valid = wl.page_valid
        for p in range(wl.num_pages):
            if valid[p] == 0:
                continue
            for h in range(hkv):
                # valid slots only: the generator poisons the rest
                np.testing.assert_array_equal(
                    _valid_elems(kp[p, h], valid[p], d, "k", 2),
                    _valid_elems(want_k[p, h], valid[p], d, "k", 2))
                np.testing.assert_array_equal(
                    _valid_elems(vp[p, h], valid[p], d, "v", 2),
                    _valid_elems(want_v[p, h], valid[p], d, "v", 2))


def _layout(d, which, elem_bytes):
    """Storage position -> logical index (t * D + dim) of one tile, found by
    running the generator's layout code on index tensors of the pool's
    element size (two byte planes for fp8)."""
    idx = torch.arange(16 * d, dtype=torch.int64)
    if elem_bytes == 2:
        pos = to_page_format(idx.to(torch.int16).view(1, 1, 16, d), which)
        return pos.view(-1).numpy().astype(np.int64)
    lo = to_page_format((idx & 0xFF).to(torch.uint8).view(1, 1, 16, d), which)
    hi = to_page_format((idx >> 8).to(torch.uint8).view(1, 1, 16, d), which)
    return (lo.view(-1).numpy().astype(np.int64)
            + 256 * hi.view(-1).numpy().astype(np.int64))


def _valid_elems(tile, n_valid, d, which, elem_bytes):
    """[n_valid, D] elements of the first n_valid slots of a tile."""
    lay = _layout(d, which, elem_bytes)           # storage i holds logical lay[i]
    logical = np.empty(16 * d, dtype=np.asarray(tile).dtype)
    logical[lay] = np.asarray(tile).reshape(-1)
    return logical.reshape(16, d)[:n_valid]


# ------------------------------------------------------------ fp8 pages

def batch_quantize(x):
    """Whole-page quantisation as the workload generator states it, with
    torch ops: scale = amax / 448 (1 if 0), code = e4m3fn(clamp(x / s))."""
    x = torch.as_tensor(x, dtype=torch.float32)
    amax = x.abs().amax()
    s = amax / FP8_MAX if amax > 0 else torch.tensor(1.0)
    y = (x / s).clamp(-FP8_MAX, FP8_MAX).to(torch.float8_e4m3fn)
    return y.view(torch.uint8).numpy(), np.float32(s)


def fp8_single_page(d=64, seed=0):
    cfg = custom_config([16], num_q_heads=1, num_kv_heads=1, head_dim=d,
                        kv_dtype="fp8_e4m3fn")
    wl = make_workload(cfg, seed=seed)
    return host_arrays(wl)


@pytest.mark.parametrize("seed", range(4))
def test_fp8_appends_match_batch_quantisation_when_token0_is_largest(seed):
    d = 64
    arrays = fp8_single_page(d, seed)
    rng = np.random.default_rng(seed)
    xk = torch.as_tensor(rng.normal(size=(16, d)), dtype=torch.float32)
    xv = torch.as_tensor(rng.normal(size=(16, d)), dtype=torch.float32)
    for x in (xk, xv):
        x[0, 3] = 2 * x.abs().max() + 1              # token 0 holds the amax
    xk, xv = xk.to(torch.bfloat16), xv.to(torch.bfloat16)
    kp = np.full_like(arrays["k_pages"], 0x7F)
    vp = np.full_like(arrays["v_pages"], 0x7F)
    ks = np.full_like(arrays["k_scale"], np.nan)
    vs = np.full_like(arrays["v_scale"], np.nan)
    bt = arrays["block_table"]
    for t in range(16):
        kp, vp, ks, vs = kv_append(
            kp, vp, ks, vs, bt, np.array([t + 1], np.int32),
            bits16(xk[t])[None, None], bits16(xv[t])[None, None],
            head_dim=d, num_kv_heads=1, kv_dtype="fp8_e4m3fn")
    p = int(bt[0, 0])
    for pool, sc, x, which in ((kp, ks, xk, "k"), (vp, vs, xv, "v")):
        codes, s = batch_quantize(x.float())
        want = to_page_format(torch.as_tensor(codes).view(1, 1, 16, d), which)
        np.testing.assert_array_equal(pool[p, 0], want.view(-1).numpy())
        assert sc[p, 0] == s


def test_fp8_doubling_recodes_by_one_exponent_step():
    """Old codes with exponent field >= 2, then a token with twice the amax:
    the scale doubles exactly and every old code drops one exponent step,
    so dequantised old values are unchanged."""
    d = 64
    arrays = fp8_single_page(d)
    rng = np.random.default_rng(3)
    u = 9
    old = rng.integers(0x10, 0x7F, size=(u, d)).astype(np.uint8)
    old[0, 0] = 0x7E                                   # the old amax code
    old |= (rng.integers(0, 2, size=(u, d)) << 7).astype(np.uint8)
    s_old = np.float32(2.0 ** -5)
    kp = np.full_like(arrays["k_pages"], 0x7F)
    vp = np.full_like(arrays["v_pages"], 0x7F)
    p = int(arrays["block_table"][0, 0])
    kp[p, 0] = to_page_format(
        torch.as_tensor(np.concatenate([old, np.full((16 - u, d), 0x7F, np.uint8)]))
        .view(1, 1, 16, d), "k").view(-1).numpy()
    ks = np.full_like(arrays["k_scale"], s_old)
    vs = np.full_like(arrays["v_scale"], 1.0)
    a_old = np.float32(448 * s_old)
    x_new = np.zeros(d, np.float32)
    x_new[5] = -2 * a_old
    new_bits = bits16(torch.as_tensor(x_new).to(torch.bfloat16))
    kp2, _, ks2, _ = kv_append(kp, vp, ks, vs, arrays["block_table"],
                               np.array([u + 1], np.int32),
                               new_bits[None, None], new_bits[None, None],
                               head_dim=d, num_kv_heads=1,
                               kv_dtype="fp8_e4m3fn")
    assert ks2[p, 0] == 2 * s_old
    got = _valid_elems(kp2[p, 0], u + 1, d, "k", 1)
    want_old = old - np.uint8(0x08)                    # exponent field - 1
    np.testing.assert_array_equal(got[:u], want_old)
    np.testing.assert_array_equal(
        E4M3FN_TABLE[got[:u]] * ks2[p, 0], E4M3FN_TABLE[old] * s_old)
    assert got[u, 5] == 0xFE and np.all(got[u, np.arange(d) != 5] == 0)


def test_fp8_scale_is_the_batch_scale_and_recoding_error_is_bounded():
    """Random appends with growing magnitudes: the scale always equals
    fl(max |x| / 448) over the page's appended values, and each old value
    is off by at most one rounding per re-encoding (3-bit mantissa:
    relative 2^-4, plus the subnormal step 2^-10 * s)."""
    d = 64
    arrays = fp8_single_page(d, 1)
    rng = np.random.default_rng(11)
    p = int(arrays["block_table"][0, 0])
    kp = np.full_like(arrays["k_pages"], 0x7F)
    vp = np.full_like(arrays["v_pages"], 0x7F)
    ks = np.full_like(arrays["k_scale"], np.nan)
    vs = np.full_like(arrays["v_scale"], np.nan)
    xs, recodes = [], np.zeros(16, int)
    for t in range(16):
        x = rng.normal(size=d) * 2.0 ** rng.integers(-4, 6)
        xb = torch.as_tensor(x, dtype=torch.float32).to(torch.bfloat16)
        xs.append(xb.float().numpy())
        before = ks[p, 0]
        kp, vp, ks, vs = kv_append(kp, vp, ks, vs, arrays["block_table"],
                                   np.array([t + 1], np.int32),
                                   bits16(xb)[None, None], bits16(xb)[None, None],
                                   head_dim=d, num_kv_heads=1,
                                   kv_dtype="fp8_e4m3fn")
        if t > 0 and ks[p, 0] != before:
            recodes[:t] += 1
        amax = np.float32(np.abs(np.array(xs)).max())
        assert ks[p, 0] == np.float32(amax / np.float32(448))
        assert vs[p, 0] == ks[p, 0]
    s = np.float64(ks[p, 0])
    got = E4M3FN_TABLE[_valid_elems(kp[p, 0], 16, d, "k", 1)] * s
    x = np.array(xs, np.float64)
    bound = (recodes[:, None] + 1) * (2.0 ** -4 * np.abs(x) + 2.0 ** -10 * s)
    assert np.all(np.abs(got - x) <= bound)


def test_fp8_zero_page_takes_the_first_nonzero_scale():
    """A page whose valid codes are all zero has scale 1; the next token
    with a magnitude sets the scale afresh (no re-encoding of the zeros)."""
    d = 64
    arrays = fp8_single_page(d, 2)
    kp = np.full_like(arrays["k_pages"], 0x7F)
    vp = np.full_like(arrays["v_pages"], 0x7F)
    ks = np.full_like(arrays["k_scale"], np.nan)
    vs = np.full_like(arrays["v_scale"], np.nan)
    bt = arrays["block_table"]
    p = int(bt[0, 0])
    zero = np.zeros((1, 1, d), np.uint16)
    for t in range(3):
        kp, vp, ks, vs = kv_append(kp, vp, ks, vs, bt, np.array([t + 1], np.int32),
                                   zero, zero, head_dim=d, num_kv_heads=1,
                                   kv_dtype="fp8_e4m3fn")
        assert ks[p, 0] == 1.0
    x = np.full(d, 0.01, np.float32)
    xb = bits16(torch.as_tensor(x).to(torch.bfloat16))[None, None]
    kp, vp, ks, vs = kv_append(kp, vp, ks, vs, bt, np.array([4], np.int32), xb,
                               xb, head_dim=d, num_kv_heads=1,
                               kv_dtype="fp8_e4m3fn")
    xf = torch.as_tensor(x).to(torch.bfloat16).float().numpy()
    assert ks[p, 0] == np.float32(np.float32(np.abs(xf).max()) / np.float32(448))
    got = _valid_elems(kp[p, 0], 4, d, "k", 1)
    assert np.all(got[:3] == 0) and np.all(got[3] == 0x7E)


def test_append_scale_special_cases():
    empty = np.zeros((0, 8), np.uint8)
    x = np.array([0.5, -3.0], np.float32)
    assert append_scale(empty, np.float32(np.nan), x) == (np.float32(3.0) / np.float32(448), False)
    assert append_scale(empty, np.float32(7), np.zeros(2, np.float32)) == (1.0, False)
    old = np.array([[0x10, 0x90]], np.uint8)
    s, recode = append_scale(old, np.float32(1.0), x)
    assert s == 1.0 and not recode                # 1.0 >= 3/448 and not empty
    s, recode = append_scale(old, np.float32(1e-3), x)
    assert s == np.float32(3.0) / np.float32(448) and recode


# ------------------------------------------------------------ edges, runs

def test_no_append_for_empty_or_unmapped_trajectories():
    cfg = custom_config([0, 5, 20], num_q_heads=2, num_kv_heads=1, head_dim=64)
    arrays = host_arrays(make_workload(cfg, seed=9))
    bt = arrays["block_table"].copy()
    bt[1, 0] = -1                                 # unmapped block
    bt[2, 1] = 10 ** 6                            # outside the pool
    new = np.ones((3, 1, 64), np.uint16)
    kp, vp, _, _ = kv_append(arrays["k_pages"], arrays["v_pages"], None, None,
                             bt, np.array([0, 5, 20], np.int32), new, new,
                             head_dim=64, num_kv_heads=1, kv_dtype="bf16")
    np.testing.assert_array_equal(kp, arrays["k_pages"])
    np.testing.assert_array_equal(vp, arrays["v_pages"])
    wide = np.array([[0]], np.int32)              # block index past the width
    kp, _, _, _ = kv_append(arrays["k_pages"], arrays["v_pages"], None, None,
                            wide, np.array([17], np.int32), new[:1], new[:1],
                            head_dim=64, num_kv_heads=1, kv_dtype="bf16")
    np.testing.assert_array_equal(kp, arrays["k_pages"])


def test_decode_run_then_attention_equals_attention_on_the_appended_tokens():
    """bf16: after a decode run the attention oracle over the appended pool
    equals torch float64 SDPA over the original tokens followed by the
    appended ones (gathered without the oracle's addressing)."""
    cfg = custom_config([3, 16, 30], num_q_heads=4, num_kv_heads=2,
                        head_dim=64)
    wl = make_workload(cfg, seed=4, keep_logical=True)
    run = make_decode_run(wl, steps=21, seed=2)
    kp = bits16(run.k_pages)
    vp = bits16(run.v_pages)
    for i in range(run.steps):
        kp, vp, _, _ = kv_append(kp, vp, None, None, run.block_table,
                                 run.lens_after(i), bits16(run.k_new[i]),
                                 bits16(run.v_new[i]), head_dim=64,
                                 num_kv_heads=2, kv_dtype="bf16")
    lens = run.lens_after(run.steps - 1)
    out, lse = decode_attention(bits16(wl.q), kp, vp, run.block_table, lens,
                                head_dim=64, num_kv_heads=2, kv_dtype="bf16",
                                softmax_scale=wl.softmax_scale)
    g = 2
    for b in range(3):
        n0 = int(run.lens0[b])
        t = torch.arange(n0)
        pages = torch.as_tensor(wl.block_table[b].astype(np.int64))[t // 16]
        for h in range(2):
            k = torch.cat([wl.k_logical[pages, h, t % 16].double(),
                           run.k_new[:, b, h].double()])
            v = torch.cat([wl.v_logical[pages, h, t % 16].double(),
                           run.v_new[:, b, h].double()])
            qh = wl.q[b, h * g:(h + 1) * g].double()[:, None, :]
            o = torch.nn.functional.scaled_dot_product_attention(
                qh, k[None].expand(g, -1, -1), v[None].expand(g, -1, -1),
                scale=wl.softmax_scale)[:, 0]
            s = wl.softmax_scale * (qh[:, 0] @ k.T)
            np.testing.assert_allclose(out[b, h * g:(h + 1) * g], o.numpy(),
                                       atol=1e-12)
            np.testing.assert_allclose(lse[b, h * g:(h + 1) * g],
                                       torch.logsumexp(s, 1).numpy(), atol=1e-12)
