"""Pins of the fp64 oracle against things other than itself.

Each test fixes the oracle against a library routine (torch float64 SDPA and
torch dtype casts), brute force, closed forms or invariants of softmax
attention, chosen so that a plausible slip (a dropped scale, a wrong log base,
a swapped head mapping, a transposed tile index, a K/V scale mix-up, a masking
off-by-one) fails at least one of them.
"""
import math
import os

import numpy as np
import pytest
import torch

from oracle import (E4M3FN_TABLE, bf16_bits_to_f64, decode_attention,
                    decode_attention_from_host, e4m3fn_bytes_to_f64)
from workloads import custom_config, host_arrays, make_workload, to_page_format

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ------------------------------------------------------------------ helpers

def logical_kv(wl, b, kvh):
    """K, V of trajectory b / kv-head kvh as float64 [n, D], read from the
    generator's logical pool with torch casts (independent of the oracle's
    decoders and tile addressing)."""
    n = int(wl.seq_lens[b])
    t = torch.arange(n)
    pages = torch.as_tensor(wl.block_table[b].astype(np.int64))[t // 16]
    slot = t % 16
    k = wl.k_logical[pages, kvh, slot]          # [n, D] storage dtype
    v = wl.v_logical[pages, kvh, slot]
    if wl.cfg.kv_dtype == "fp8_e4m3fn":
        k = k.view(torch.float8_e4m3fn).to(torch.float64) \
            * wl.k_scale[pages, kvh].to(torch.float64)[:, None]
        v = v.view(torch.float8_e4m3fn).to(torch.float64) \
            * wl.v_scale[pages, kvh].to(torch.float64)[:, None]
    else:
        k = k.to(torch.float64)
        v = v.to(torch.float64)
    return k, v


def torch_reference(wl):
    """torch float64 scaled_dot_product_attention + logsumexp, GQA by
    repeating each kv-head over its group of query heads."""
    c = wl.cfg
    g = c.num_q_heads // c.num_kv_heads
    out = np.zeros((wl.batch, c.num_q_heads, c.head_dim))
    lse = np.zeros((wl.batch, c.num_q_heads))
    qf = wl.q.to(torch.float64)
    for b in range(wl.batch):
        ks, vs = zip(*[logical_kv(wl, b, h) for h in range(c.num_kv_heads)])
        k = torch.stack(ks).repeat_interleave(g, dim=0)      # [Hq, n, D]
        v = torch.stack(vs).repeat_interleave(g, dim=0)
        qb = qf[b][:, None, :]                                # [Hq, 1, D]
        o = torch.nn.functional.scaled_dot_product_attention(
            qb, k, v, scale=wl.softmax_scale)
        s = (qb @ k.transpose(1, 2))[:, 0, :] * wl.softmax_scale
        out[b] = o[:, 0, :].numpy()
        lse[b] = torch.logsumexp(s, dim=-1).numpy()
    return out, lse


def run_oracle(arrays, **over):
    a = dict(arrays)
    a.update(over)
    return decode_attention_from_host(a)


# ----------------------------------------------------------------- decoders

def test_bf16_decoder_exhaustive():
    codes = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ref = torch.from_numpy(codes.view(np.int16).copy()).view(
        torch.bfloat16).to(torch.float64).numpy()
    got = bf16_bits_to_f64(codes)
    assert np.array_equal(np.isnan(ref), np.isnan(got))
    ok = ~np.isnan(ref)
    assert np.array_equal(ref[ok], got[ok])


def test_e4m3fn_decoder_exhaustive():
    codes = np.arange(256, dtype=np.uint8)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(
        torch.float64).numpy()
    got = e4m3fn_bytes_to_f64(codes)
    assert np.array_equal(np.isnan(ref), np.isnan(got))
    assert np.isnan(E4M3FN_TABLE[0x7F]) and np.isnan(E4M3FN_TABLE[0xFF])
    ok = ~np.isnan(ref)
    assert np.array_equal(ref[ok], got[ok])
    assert got[0x7E] == 448.0 and got[0x01] == 2.0 ** -9


# ----------------------------------------------------- library cross-check

CASES = [
    ("tiny", None),
    ("gqa7_d128", custom_config([1, 15, 16, 17, 300, 1000], 28, 4, 128)),
    ("fp8_g5", custom_config([5, 16, 33, 250, 700], 10, 2, 128,
                             kv_dtype="fp8_e4m3fn")),
    ("prefix", custom_config([10, 40, 100, 64, 3, 200, 65, 90], 8, 2, 64,
                             prefix_group=4, prefix_tokens=64)),
    ("mha_d64", custom_config([7, 129], 3, 3, 64)),
]


@pytest.mark.parametrize("name,cfg", CASES, ids=[c[0] for c in CASES])
def test_matches_torch_sdpa_float64(name, cfg):
    wl = make_workload(cfg if cfg is not None else 1, seed=7,
                       keep_logical=True)
    out, lse = decode_attention_from_host(host_arrays(wl))
    ref_out, ref_lse = torch_reference(wl)
    assert np.isfinite(out).all() and np.isfinite(lse).all()
    np.testing.assert_allclose(out, ref_out, rtol=0, atol=1e-10)
    np.testing.assert_allclose(lse, ref_lse, rtol=0, atol=1e-10)


def test_bruteforce_python_loops():
    """Direct summation with math.exp over decoded values (torch casts)."""
    wl = make_workload(custom_config([3, 18], 4, 2, 64), seed=3,
                       keep_logical=True)
    out, lse = decode_attention_from_host(host_arrays(wl))
    q = wl.q.to(torch.float64).tolist()
    for b in range(2):
        for h in range(4):
            k, v = logical_kv(wl, b, h // 2)
            k, v = k.tolist(), v.tolist()
            s = [wl.softmax_scale * sum(qi * ki for qi, ki in zip(q[b][h], kt))
                 for kt in k]
            z = sum(math.exp(x) for x in s)
            assert abs(lse[b, h] - math.log(z)) < 1e-12
            for d in range(64):
                o = sum(math.exp(x) / z * vt[d] for x, vt in zip(s, v))
                assert abs(out[b, h, d] - o) < 1e-12


def test_golden_two_token_example():
    vals = {}
    with open(os.path.join(GOLDEN, "two_token_example.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                k, v = line.split()
                vals[k] = float(v)
    d = 16
    one = 0x3F80                     # bf16 code of 1.0
    two = 0x4000                     # bf16 code of 2.0
    q = np.zeros((1, 1, d), np.uint16)
    q[0, 0, 0] = one
    klog = np.zeros((1, 1, 16, d), np.uint16)
    vlog = np.zeros((1, 1, 16, d), np.uint16)
    klog[0, 0, 0, 0] = two
    vlog[0, 0, 0, 0] = one
    vlog[0, 0, 1, 1] = one
    as_t = lambda a: torch.from_numpy(a.view(np.int16)).view(torch.bfloat16)
    kp = to_page_format(as_t(klog), "k").view(torch.int16).numpy().view(np.uint16)
    vp = to_page_format(as_t(vlog), "v").view(torch.int16).numpy().view(np.uint16)
    out, lse = decode_attention(q, kp, vp, np.array([[0]], np.int32),
                                np.array([2], np.int32), head_dim=d,
                                num_kv_heads=1, kv_dtype="bf16",
                                softmax_scale=0.25)
    assert abs(lse[0, 0] - vals["lse"]) < 1e-15
    assert abs(out[0, 0, 0] - vals["out0"]) < 1e-15
    assert abs(out[0, 0, 1] - vals["out1"]) < 1e-15
    assert np.all(out[0, 0, 2:] == 0)


# ------------------------------------------------------------- closed forms

def test_single_token_returns_v():
    wl = make_workload(custom_config([1, 1], 4, 2, 128), seed=11,
                       keep_logical=True)
    out, lse = decode_attention_from_host(host_arrays(wl))
    qf = wl.q.to(torch.float64)
    for b in range(2):
        for h in range(4):
            k, v = logical_kv(wl, b, h // 2)
            np.testing.assert_array_equal(out[b, h], v[0].numpy())
            s0 = wl.softmax_scale * float(qf[b, h] @ k[0])
            assert abs(lse[b, h] - s0) < 1e-12


def test_zero_query_gives_mean_v_and_ln_n():
    wl = make_workload(custom_config([5, 77, 300], 6, 3, 64), seed=5,
                       keep_logical=True)
    a = host_arrays(wl)
    a["q"] = np.zeros_like(a["q"])
    out, lse = decode_attention_from_host(a)
    for b in range(3):
        n = int(wl.seq_lens[b])
        for h in range(6):
            _, v = logical_kv(wl, b, h // 2)
            np.testing.assert_allclose(out[b, h], v.mean(0).numpy(),
                                       rtol=0, atol=1e-13)
            assert abs(lse[b, h] - math.log(n)) < 1e-13


def test_constant_keys_give_mean_v_and_s_plus_ln_n():
    cfg = custom_config([9, 50, 257], 4, 1, 64)
    wl = make_workload(cfg, seed=9, keep_logical=True)
    kc = torch.randn(64, generator=torch.Generator().manual_seed(1)).to(
        torch.bfloat16)
    klog = wl.k_logical.clone()
    klog[:] = kc
    a = host_arrays(wl)
    a["k_pages"] = to_page_format(klog, "k").view(torch.int16).numpy().view(
        np.uint16)
    out, lse = decode_attention_from_host(a)
    qf = wl.q.to(torch.float64)
    for b in range(3):
        n = int(wl.seq_lens[b])
        _, v = logical_kv(wl, b, 0)
        for h in range(4):
            s = wl.softmax_scale * float(qf[b, h] @ kc.to(torch.float64))
            assert abs(lse[b, h] - (s + math.log(n))) < 1e-12
            np.testing.assert_allclose(out[b, h], v.mean(0).numpy(),
                                       rtol=0, atol=1e-13)


def test_empty_sequence_is_merge_identity():
    wl = make_workload(custom_config([0, 20], 2, 1, 64), seed=1)
    out, lse = decode_attention_from_host(host_arrays(wl))
    assert np.all(out[0] == 0) and np.all(lse[0] == -np.inf)
    assert np.isfinite(lse[1]).all()


# --------------------------------------------------------------- invariants

def test_page_permutation_invariance_bitwise():
    wl = make_workload(custom_config([33, 200, 513, 16], 8, 2, 128), seed=2)
    a = host_arrays(wl)
    out, lse = decode_attention_from_host(a)
    p = a["k_pages"].shape[0]
    perm = np.random.default_rng(0).permutation(p)
    b = dict(a)
    b["k_pages"] = np.empty_like(a["k_pages"])
    b["v_pages"] = np.empty_like(a["v_pages"])
    b["k_pages"][perm] = a["k_pages"]
    b["v_pages"][perm] = a["v_pages"]
    bt = a["block_table"]
    b["block_table"] = np.where(bt >= 0, perm[np.maximum(bt, 0)], -1).astype(
        np.int32)
    out2, lse2 = decode_attention_from_host(b)
    assert np.array_equal(out, out2) and np.array_equal(lse, lse2)


def test_split_then_lse_merge_equals_unsplit():
    wl = make_workload(custom_config([513, 1000, 47], 6, 2, 64), seed=4)
    a = host_arrays(wl)
    out, lse = decode_attention_from_host(a)
    for cut_pages in (1, 3, 16):
        cut = 16 * cut_pages
        lens = a["seq_lens"]
        first = np.minimum(lens, cut).astype(np.int32)
        second = np.maximum(lens - cut, 0).astype(np.int32)
        bt2 = np.full_like(a["block_table"], -1)
        w = a["block_table"].shape[1] - cut_pages
        bt2[:, :w] = a["block_table"][:, cut_pages:]
        o1, l1 = run_oracle(a, seq_lens=first)
        o2, l2 = run_oracle(a, seq_lens=second, block_table=bt2)
        big = np.maximum(l1, l2)
        L = big + np.log(np.exp(l1 - big) + np.exp(l2 - big))
        o = np.exp(l1 - L)[..., None] * o1 + np.exp(l2 - L)[..., None] * o2
        np.testing.assert_allclose(L, lse, rtol=0, atol=1e-12)
        np.testing.assert_allclose(o, out, rtol=0, atol=1e-12)


def test_gqa_equals_mha_with_repeated_kv_heads():
    wl = make_workload(custom_config([40, 300], 12, 3, 64), seed=6)
    a = host_arrays(wl)
    out, lse = decode_attention_from_host(a)
    g = 4
    b = dict(a)
    b["k_pages"] = np.repeat(a["k_pages"], g, axis=1)
    b["v_pages"] = np.repeat(a["v_pages"], g, axis=1)
    b["num_kv_heads"] = 12
    out2, lse2 = decode_attention_from_host(b)
    np.testing.assert_allclose(out2, out, rtol=0, atol=1e-15)
    np.testing.assert_allclose(lse2, lse, rtol=0, atol=1e-15)


def test_linear_in_v():
    cfg = custom_config([30, 100], 4, 2, 64)
    wl = make_workload(cfg, seed=8, keep_logical=True)
    gen = torch.Generator().manual_seed(3)
    shape = wl.v_logical.shape
    v1 = torch.randint(-4, 5, shape, generator=gen).to(torch.bfloat16)
    v2 = torch.randint(-4, 5, shape, generator=gen).to(torch.bfloat16)
    bits = lambda t: to_page_format(t, "v").view(torch.int16).numpy().view(
        np.uint16)
    a = host_arrays(wl)
    o1, l1 = run_oracle(a, v_pages=bits(v1))
    o2, l2 = run_oracle(a, v_pages=bits(v2))
    o12, l12 = run_oracle(a, v_pages=bits(v1 + v2))   # exact: |sum| <= 8
    np.testing.assert_allclose(o12, o1 + o2, rtol=0, atol=1e-12)
    assert np.array_equal(l1, l12)


def test_batch_permutation_equivariance():
    wl = make_workload(custom_config([3, 99, 17, 260, 64], 4, 1, 64), seed=10)
    a = host_arrays(wl)
    out, lse = decode_attention_from_host(a)
    perm = np.array([3, 0, 4, 1, 2])
    b = dict(a)
    b["q"] = a["q"][perm]
    b["block_table"] = a["block_table"][perm]
    b["seq_lens"] = a["seq_lens"][perm]
    out2, lse2 = decode_attention_from_host(b)
    assert np.array_equal(out2, out[perm]) and np.array_equal(lse2, lse[perm])


def test_nan_poison_never_reaches_output():
    for cfg in (1, custom_config([1, 17, 31, 5, 64, 3, 100, 2], 8, 2, 64,
                                 prefix_group=4, prefix_tokens=64),
                custom_config([3, 33], 4, 2, 64, kv_dtype="fp8_e4m3fn")):
        wl = make_workload(cfg, seed=12)
        a = host_arrays(wl)
        assert np.isnan(bf16_bits_to_f64(a["k_pages"])).any() or \
            (a["k_pages"] == 0x7F).any()
        out, lse = decode_attention_from_host(a)
        assert np.isfinite(out).all() and np.isfinite(lse).all()


def test_prefix_aliasing_equals_copied_prefix():
    cfg = custom_config([10, 40, 100, 64, 3, 200, 65, 90], 8, 2, 64,
                        prefix_group=4, prefix_tokens=64)
    wl = make_workload(cfg, seed=13)
    a = host_arrays(wl)
    out, lse = decode_attention_from_host(a)
    # give every trajectory private copies of the pages it shares
    bt = a["block_table"].copy()
    kp, vp = [a["k_pages"]], [a["v_pages"]]
    nxt = a["k_pages"].shape[0]
    seen = set()
    for b in range(bt.shape[0]):
        for j in range(bt.shape[1]):
            p = bt[b, j]
            if p < 0:
                continue
            if p in seen:
                kp.append(a["k_pages"][p:p + 1])
                vp.append(a["v_pages"][p:p + 1])
                bt[b, j] = nxt
                nxt += 1
            seen.add(p)
    assert nxt > a["k_pages"].shape[0]
    out2, lse2 = run_oracle(a, k_pages=np.concatenate(kp),
                            v_pages=np.concatenate(vp), block_table=bt)
    assert np.array_equal(out, out2) and np.array_equal(lse, lse2)


def test_threaded_equals_serial():
    wl = make_workload(custom_config([100, 2000, 5, 700], 8, 2, 128), seed=14)
    a = host_arrays(wl)
    o1, l1 = decode_attention_from_host(a, workers=1)
    o4, l4 = decode_attention_from_host(a, workers=4)
    assert np.array_equal(o1, o4) and np.array_equal(l1, l4)
