"""GPU parity of the decode step's element-wise kernels and of the bf16
projection epilogue against the fp64 oracle.

Bar: every bf16 output within one bf16 unit in the last place of the fp64
value (the kernels round an fp32 result once; fp32 error can move that
rounding by one step), plus, for the projection, the fp32 accumulation
bound 4 (K/32 + 32) 2^-24 sum_k |x w| of the fp32 kernel."""
import numpy as np
import pytest
import torch

from oracle.decoder import rmsnorm as rmsnorm_ref, silu_mul as silu_mul_ref
from oracle.linear import bf16_to_f64, linear, linear_abs

pytestmark = pytest.mark.gpu


def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")


def bits(t):
    return t.detach().cpu().view(torch.int16).numpy().view(np.uint16)


def ulp_bound(ref):
    """One bf16 step at the magnitude of ref (8 significant bits)."""
    a = np.abs(ref)
    e = np.floor(np.log2(np.maximum(a, 2.0 ** -126)))
    return 2.0 ** (e - 7)


def rand_bf16(g, shape, scale=1.0):
    return (torch.randn(shape, generator=g, device="cuda") * scale).to(torch.bfloat16)


@pytest.mark.parametrize("m,n,weighted", [(1, 3584, True), (7, 5120, False),
                                          (64, 18944, True), (3, 8, True)])
def test_rmsnorm_matches_oracle(m, n, weighted):
    from paper_2510_12633_amd.api import rmsnorm
    _need_gpu()
    g = torch.Generator(device="cuda").manual_seed(m + n)
    x = rand_bf16(g, (m, n), 3.0)
    w = rand_bf16(g, (n,)) if weighted else None
    y = rmsnorm(x, w, eps=1e-6)
    torch.cuda.synchronize()
    ref = rmsnorm_ref(bits(x), bits(w) if weighted else None, eps=1e-6)
    err = np.abs(bf16_to_f64(bits(y)) - ref)
    print(f"[gpu-step] rmsnorm m={m} n={n}: max err/ulp "
          f"{(err / ulp_bound(ref)).max():.3f}", flush=True)
    assert np.all(err <= ulp_bound(ref))


@pytest.mark.parametrize("m,inter", [(1, 18944), (16, 27648), (64, 8)])
def test_silu_mul_matches_oracle(m, inter):
    from paper_2510_12633_amd.api import silu_mul
    _need_gpu()
    g = torch.Generator(device="cuda").manual_seed(m * 7 + inter)
    gu = rand_bf16(g, (m, 2 * inter), 4.0)
    y = silu_mul(gu)
    torch.cuda.synchronize()
    ref = silu_mul_ref(bits(gu))
    err = np.abs(bf16_to_f64(bits(y)) - ref)
    print(f"[gpu-step] silu_mul m={m} I={inter}: max err/ulp "
          f"{(err / ulp_bound(ref)).max():.3f}", flush=True)
    assert np.all(err <= ulp_bound(ref) + 2.0 ** -133)


@pytest.mark.parametrize("m,n,k,in_place", [(1, 3584, 3584, False),
                                            (16, 3584, 18944, True),
                                            (33, 4608, 3584, False),
                                            (5, 96, 640, True),
                                            (128, 3584, 3584, True)])
def test_linear_bf16_with_residual(m, n, k, in_place):
    from paper_2510_12633_amd.api import SkinnyLinear
    _need_gpu()
    g = torch.Generator(device="cuda").manual_seed(m + n + k)
    x = rand_bf16(g, (m, k))
    w = rand_bf16(g, (n, k), k ** -0.5)
    res = rand_bf16(g, (m, n))
    res_bits = bits(res)
    lin = SkinnyLinear(w)
    y = lin.bf16(x, out=res if in_place else None, residual=res)
    y_plain = lin.bf16(x)
    torch.cuda.synchronize()
    xb, wb = bits(x), bits(w)
    acc = 4 * (k / 32 + 32) * 2.0 ** -24 * linear_abs(xb, wb)
    for got, r in ((y, bf16_to_f64(res_bits)), (y_plain, 0.0)):
        ref = linear(xb, wb) + r
        err = np.abs(bf16_to_f64(bits(got)) - ref)
        print(f"[gpu-step] linear_bf16 m={m} n={n} k={k}: max err/bound "
              f"{(err / (acc + ulp_bound(ref))).max():.3f}", flush=True)
        assert np.all(err <= acc + ulp_bound(ref))


def test_decode_step_argument_errors():
    from paper_2510_12633_amd import _native as N
    _need_gpu()
    s = torch.cuda.current_stream().cuda_stream
    x = torch.zeros((4, 64), dtype=torch.bfloat16, device="cuda")
    y = torch.empty_like(x)
    for args in ((x, None, y, 4, 60, 1e-6), (x, None, y, 0, 64, 1e-6),
                 (x, None, y, 4, 64, -1.0), (x, None, None, 4, 64, 1e-6)):
        with pytest.raises(N.LaminarError) as e:
            N.laminar_rmsnorm(*args, s)
        assert e.value.status == N.LAMINAR_ERR_INVALID_ARG
    with pytest.raises(N.LaminarError) as e:
        N.laminar_silu_mul(x, y, 4, 12, s)
    assert e.value.status == N.LAMINAR_ERR_INVALID_ARG


@pytest.mark.parametrize("m", [1, 3, 4])
def test_fused_decode_step_equals_unfused(m):
    """A two-layer decoder step (RMS norm, QKV, KV append, paged attention,
    O with the residual, norm, gate+up, SwiGLU, down with the residual, LM
    head) run once with every norm, cast and SwiGLU as its own launch and
    once with all of them made on load in the projections: logits, the
    residual stream and the KV pages agree bit for bit."""
    from paper_2510_12633_amd.api import (PagedDecodeAttention, SkinnyLinear,
                                          kv_append, rmsnorm, silu_mul)
    _need_gpu()
    print(f"[gpu-decode-step] fused vs unfused m={m}", flush=True)
    L, h, hq, hkv, d, inter, vocab = 2, 512, 8, 2, 64, 1024, 2048
    g = torch.Generator(device="cuda").manual_seed(41 + m)
    bf = torch.bfloat16

    def lin(k, n):
        return SkinnyLinear(rand_bf16(g, (n, k), k ** -0.5))

    layers = [(lin(h, (hq + 2 * hkv) * d), lin(hq * d, h), lin(h, 2 * inter),
               lin(inter, h)) for _ in range(L)]
    head = lin(h, vocab)
    norms = (1 + 0.1 * torch.randn((2 * L + 1, h), generator=g,
                                   device="cuda")).to(bf)
    ctx = 40
    pages = -(-(ctx + 1) // 16)
    kp0 = rand_bf16(g, (m * pages, hkv, 16 * d))
    vp0 = rand_bf16(g, (m * pages, hkv, 16 * d))
    table = torch.arange(m * pages, dtype=torch.int32, device="cuda").view(m, pages)
    lens_host = np.full(m, ctx + 1, np.int32)
    lens = torch.as_tensor(lens_host, device="cuda")
    att = PagedDecodeAttention(
        batch=m, num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
        num_pages=m * pages, max_blocks_per_seq=pages, seq_lens_host=lens_host,
        softmax_scale=d ** -0.5, q_row_stride=(hq + 2 * hkv) * d)
    out, lse = att.outputs()
    x0 = rand_bf16(g, (m, h))

    def step(fused):
        kp, vp = kp0.clone(), vp0.clone()
        x = x0.clone()
        for li, (wqkv, wo, wgu, wd) in enumerate(layers):
            if fused:
                qkv = wqkv.bf16(x, norm_weight=norms[2 * li])
            else:
                qkv = wqkv.bf16(rmsnorm(x, norms[2 * li]))
            q = qkv[:, :hq * d].view(m, hq, d)
            k_new = qkv[:, hq * d:(hq + hkv) * d].view(m, hkv, d)
            v_new = qkv[:, (hq + hkv) * d:].view(m, hkv, d)
            kv_append(k_new, v_new, table, lens, kp, vp)
            att(q, kp, vp, table, lens, out, lse)
            a = out.view(m, hq * d)
            wo.bf16(a if fused else a.to(bf), out=x, residual=x)
            if fused:
                gu = wgu.bf16(x, norm_weight=norms[2 * li + 1])
                wd.bf16(gu, out=x, residual=x, swiglu=True)
            else:
                gu = wgu.bf16(rmsnorm(x, norms[2 * li + 1]))
                wd.bf16(silu_mul(gu), out=x, residual=x)
        if fused:
            logits = head.bf16(x, norm_weight=norms[2 * L])
        else:
            logits = head.bf16(rmsnorm(x, norms[2 * L]))
        torch.cuda.synchronize()
        return logits, x, kp, vp

    a, b = step(False), step(True)
    for ta, tb in zip(a, b):
        assert torch.equal(ta.view(torch.int16), tb.view(torch.int16))
    assert torch.isfinite(a[0].float()).all()
    att.close()


@pytest.mark.parametrize("m", [40, 64])
def test_reduction_fused_decode_step_equals_unfused(m):
    """The same two-layer step from 33 rows on, where K is split and a
    second kernel adds the ranges: once with every norm, SwiGLU and the KV
    append as its own launch, once with each made by the preceding
    projection's reduction (laminar_linear_bf16_kv_append for QKV,
    laminar_linear_bf16_norm for O and down, laminar_linear_bf16_swiglu for
    gate+up on the balanced split: 258 groups of 128 columns). Logits, the
    residual stream and the KV pages agree bit for bit."""
    from paper_2510_12633_amd import _native as N
    from paper_2510_12633_amd.api import (PagedDecodeAttention, SkinnyLinear,
                                          kv_append, kv_append_desc, rmsnorm,
                                          silu_mul)
    _need_gpu()
    print(f"[gpu-decode-step] reduction-fused vs unfused m={m}", flush=True)
    L, h, hq, hkv, d, inter, vocab = 2, 512, 8, 2, 64, 16512, 2048
    g = torch.Generator(device="cuda").manual_seed(77 + m)
    bf = torch.bfloat16

    def lin(k, n):
        return SkinnyLinear(rand_bf16(g, (n, k), k ** -0.5))

    layers = [(lin(h, (hq + 2 * hkv) * d), lin(hq * d, h), lin(h, 2 * inter),
               lin(inter, h)) for _ in range(L)]
    head = lin(h, vocab)
    # the reductions this step relies on do run at this size
    assert N.laminar_linear_splits(m, (hq + 2 * hkv) * d, h) > 1
    assert N.laminar_linear_splits(m, h, hq * d) > 1
    assert N.laminar_linear_splits(m, h, inter) > 1
    assert N.laminar_linear_workspace_bytes(m, 2 * inter, h) > 0     # balanced
    norms = (1 + 0.1 * torch.randn((2 * L + 1, h), generator=g,
                                   device="cuda")).to(bf)
    ctx = 40
    pages = -(-(ctx + 1) // 16)
    kp0 = rand_bf16(g, (m * pages, hkv, 16 * d))
    vp0 = rand_bf16(g, (m * pages, hkv, 16 * d))
    table = torch.randperm(m * pages, generator=g, device="cuda").to(torch.int32)
    table = table.view(m, pages).contiguous()
    lens_host = np.full(m, ctx + 1, np.int32)
    lens = torch.as_tensor(lens_host, device="cuda")
    att = PagedDecodeAttention(
        batch=m, num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
        num_pages=m * pages, max_blocks_per_seq=pages, seq_lens_host=lens_host,
        softmax_scale=d ** -0.5, q_row_stride=(hq + 2 * hkv) * d)
    out, lse = att.outputs()
    x0 = rand_bf16(g, (m, h))
    desc = kv_append_desc(m, hkv, d, m * pages, pages)

    def step(fused):
        kp, vp = kp0.clone(), vp0.clone()
        x = x0.clone()
        xn = rmsnorm(x, norms[0])
        for li, (wqkv, wo, wgu, wd) in enumerate(layers):
            if fused:
                qkv = wqkv.bf16_kv_append(xn, desc, hq * d, (hq + hkv) * d,
                                          table, lens, kp, vp)
            else:
                qkv = wqkv.bf16(xn)
                kv_append(qkv[:, hq * d:(hq + hkv) * d].view(m, hkv, d),
                          qkv[:, (hq + hkv) * d:].view(m, hkv, d), table,
                          lens, kp, vp)
            att(qkv[:, :hq * d].view(m, hq, d), kp, vp, table, lens, out, lse)
            a = out.view(m, hq * d)
            if fused:
                x, xn = wo.bf16_norm(a, norms[2 * li + 1], out=x, residual=x)
                _, act = wgu.bf16_swiglu(xn)
                x, xn = wd.bf16_norm(act, norms[2 * li + 2], out=x, residual=x)
            else:
                wo.bf16(a, out=x, residual=x)
                act = silu_mul(wgu.bf16(rmsnorm(x, norms[2 * li + 1])))
                wd.bf16(act, out=x, residual=x)
                xn = rmsnorm(x, norms[2 * li + 2])
        logits = head.bf16(xn)
        torch.cuda.synchronize()
        return logits, x, kp, vp

    a, b = step(False), step(True)
    for name, ta, tb in zip(("logits", "x", "k pages", "v pages"), a, b):
        assert torch.equal(ta.view(torch.int16), tb.view(torch.int16)), name
    assert torch.isfinite(a[0].float()).all()
    att.close()
