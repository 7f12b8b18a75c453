"""GPU parity of the skinny projection kernel against the fp64 oracle.

Bar: |y - y_ref| <= 4 (K/32 + 32) 2^-24 sum_k |x w| per output (fp32
accumulation of exact bf16 products, one rounding per matrix-core step of
32 and per accumulation), plus determinism and untouched padding rows."""
import numpy as np
import pytest
import torch

from oracle.linear import linear, linear_abs

pytestmark = pytest.mark.gpu


def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")


def bits(t):
    return t.detach().cpu().view(torch.int16).numpy().view(np.uint16)


SHAPES = [(1, 16, 128), (7, 48, 256), (16, 4608, 3584), (17, 3584, 3584),
          (33, 256, 1024), (64, 3584, 18944), (2, 37888, 3584),
          (1, 152064, 3584), (48, 96, 640), (65, 4608, 3584),
          (128, 3584, 18944), (100, 208, 512),
          # K split over the wavefronts of a workgroup (M <= 4): ragged
          # step counts per wavefront, 7B and 32B shapes
          (4, 48, 640), (1, 3584, 3584), (3, 3584, 18944), (2, 7168, 5120),
          (4, 5120, 20480),
          # the balanced split: a full round and 40 groups left over (7B
          # gate and up), 2 groups left over in 6 steps over 256 workgroups
          # (most of them get none), one step of K, 128 rows
          (64, 37888, 3584), (33, 33024, 384), (17, 37888, 128),
          (128, 37888, 256)]


@pytest.mark.parametrize("m,n,k", SHAPES)
def test_linear_matches_oracle(m, n, k):
    from paper_2510_12633_amd.api import SkinnyLinear
    _need_gpu()
    print(f"[gpu-linear] m={m} n={n} k={k}", flush=True)
    g = torch.Generator(device="cuda").manual_seed(m * 1000 + n + k)
    x = torch.randn((m, k), generator=g, device="cuda").to(torch.bfloat16)
    w = (torch.randn((n, k), generator=g, device="cuda") / k ** 0.5).to(torch.bfloat16)
    lin = SkinnyLinear(w)
    y = torch.full((m + 3, n), float("nan"), device="cuda")
    lin(x, out=y[:m])
    y2 = lin(x)
    torch.cuda.synchronize()
    got = y[:m].cpu().numpy().astype(np.float64)
    # sample rows of w for the oracle on the big shapes
    cols = np.arange(n) if n <= 8192 else np.random.default_rng(0).choice(n, 4096, replace=False)
    xb, wb = bits(x), bits(w)[cols]
    ref = linear(xb, wb)
    bound = 4 * (k / 32 + 32) * 2.0 ** -24 * linear_abs(xb, wb)
    err = np.abs(got[:, cols] - ref)
    print(f"[gpu-linear] max err {err.max():.2e}, max err/bound {(err / bound).max():.3f}",
          flush=True)
    assert np.all(err <= bound)
    assert torch.equal(y[:m], y2)                          # deterministic
    assert torch.isnan(y[m:]).all()                        # padding untouched


@pytest.mark.parametrize("n,k", [(16, 128), (48, 384), (4608, 3584)])
def test_pack_is_the_documented_permutation(n, k):
    """packed[((n/16)(K/8) + k/8) 16 + n%16][k%8] = w[n][k], bit for bit."""
    from paper_2510_12633_amd import _native as N
    _need_gpu()
    g = torch.Generator(device="cuda").manual_seed(n + k)
    w = torch.randint(-2 ** 15, 2 ** 15, (n, k), generator=g, device="cuda",
                      dtype=torch.int32).to(torch.int16)
    p = torch.empty_like(w)
    N.laminar_linear_pack(w, p, n, k, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    ref = (w.cpu().numpy().reshape(n // 16, 16, k // 8, 8)
           .transpose(0, 2, 1, 3).reshape(n, k))
    assert np.array_equal(p.cpu().numpy(), ref)


def test_linear_errors():
    from paper_2510_12633_amd import _native as N
    _need_gpu()
    x = torch.zeros((4, 256), dtype=torch.bfloat16, device="cuda")
    w = torch.zeros((32, 256), dtype=torch.bfloat16, device="cuda")
    y = torch.zeros((4, 32), device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    with pytest.raises(N.LaminarError) as e:
        N.laminar_linear(x, w, y, 129, 32, 256, None, 0, s)
    assert e.value.status == N.LAMINAR_ERR_UNSUPPORTED
    with pytest.raises(N.LaminarError) as e:
        N.laminar_linear(x, w, y, 4, 32, 200, None, 0, s)
    assert e.value.status == N.LAMINAR_ERR_UNSUPPORTED
    with pytest.raises(N.LaminarError) as e:
        N.laminar_linear_pack(w, w, 32, 256, s)
    assert e.value.status == N.LAMINAR_ERR_INVALID_ARG
    with pytest.raises(N.LaminarError) as e:
        N.laminar_linear_pack(w, y, 24, 256, s)
    assert e.value.status == N.LAMINAR_ERR_UNSUPPORTED
    need = N.laminar_linear_workspace_bytes(4, 32, 256)
    N.laminar_linear(x, w, y, 4, 32, 256,
                     torch.empty(max(need, 1), dtype=torch.uint8, device="cuda"),
                     need, s)
    torch.cuda.synchronize()


FUSED_SHAPES = [(1, 3584, 3584), (4, 3584, 3584), (3, 5120, 5120),
                (2, 3584, 18944), (4, 48, 640), (5, 4608, 3584),
                (17, 256, 1024), (64, 3584, 18944), (128, 208, 512),
                # the balanced split (x made in registers against x copied
                # into LDS as it is)
                (64, 37888, 512), (40, 33024, 384)]


@pytest.mark.parametrize("m,n,k", FUSED_SHAPES)
def test_fused_inputs_equal_the_separate_launches(m, n, k):
    """fp32 x rounded on load equals a cast then the bf16-x call, and gate
    and up combined on load equal laminar_silu_mul then the call, bit for
    bit, with and without the residual (in place). The shapes cover the
    split over wavefronts (M <= 4 and at most 256 or 512 tiles), the split
    over workgroups and no split."""
    from paper_2510_12633_amd.api import SkinnyLinear, silu_mul
    _need_gpu()
    print(f"[gpu-linear-fused] m={m} n={n} k={k}", flush=True)
    g = torch.Generator(device="cuda").manual_seed(7 * m + n + k)
    w = (torch.randn((n, k), generator=g, device="cuda") / k ** 0.5).to(torch.bfloat16)
    lin = SkinnyLinear(w)
    x32 = torch.randn((m, k), generator=g, device="cuda") * 3
    gu = (torch.randn((m, 2 * k), generator=g, device="cuda") * 4).to(torch.bfloat16)
    res = torch.randn((m, n), generator=g, device="cuda").to(torch.bfloat16)
    for fused, separate in ((lambda **kw: lin.bf16(x32, **kw),
                             lambda **kw: lin.bf16(x32.to(torch.bfloat16), **kw)),
                            (lambda **kw: lin.bf16(gu, swiglu=True, **kw),
                             lambda **kw: lin.bf16(silu_mul(gu), **kw))):
        a, b = fused(), separate()
        ra, rb = res.clone(), res.clone()
        fused(out=ra, residual=ra)
        separate(out=rb, residual=rb)
        torch.cuda.synchronize()
        assert torch.equal(bits_t(a), bits_t(b))
        assert torch.equal(bits_t(ra), bits_t(rb))
        assert torch.isfinite(a.float()).all()


def bits_t(t):
    return t.view(torch.int16)


NORM_SHAPES = [(1, 4608, 3584), (4, 37888, 3584), (3, 48, 640),
               (2, 7168, 5120), (4, 256, 1024), (2, 3584, 20608),
               (3, 208, 20608), (5, 4608, 3584), (8, 37888, 3584),
               (7, 208, 5120)]


@pytest.mark.parametrize("m,n,k", NORM_SHAPES)
def test_fused_norm_equals_rmsnorm_then_linear(m, n, k):
    """The RMS norm done on load equals laminar_rmsnorm followed by the
    bf16 call bit for bit (same summation order, same roundings), with and
    without the residual. Shapes: split over wavefronts (K of 640 to 5120
    chunks, one to three passes of the row sum), no split (gate+up), a
    split over workgroups (161 steps of K), one whose last workgroup has
    wavefronts past the last tile (13 tiles), and 5-8 rows (two rows per
    wavefront)."""
    from paper_2510_12633_amd.api import SkinnyLinear, rmsnorm
    _need_gpu()
    print(f"[gpu-linear-norm] m={m} n={n} k={k}", flush=True)
    g = torch.Generator(device="cuda").manual_seed(11 * m + n + k)
    w = (torch.randn((n, k), generator=g, device="cuda") / k ** 0.5).to(torch.bfloat16)
    lin = SkinnyLinear(w)
    x = (torch.randn((m, k), generator=g, device="cuda") * 5).to(torch.bfloat16)
    nw = (1 + 0.2 * torch.randn((k,), generator=g, device="cuda")).to(torch.bfloat16)
    res = torch.randn((m, n), generator=g, device="cuda").to(torch.bfloat16)
    for eps in (1e-6, 0.0):
        a = lin.bf16(x, norm_weight=nw, eps=eps)
        b = lin.bf16(rmsnorm(x, nw, eps=eps))
        ra, rb = res.clone(), res.clone()
        lin.bf16(x, out=ra, residual=ra, norm_weight=nw, eps=eps)
        lin.bf16(rmsnorm(x, nw, eps=eps), out=rb, residual=rb)
        torch.cuda.synchronize()
        assert torch.equal(bits_t(a), bits_t(b))
        assert torch.equal(bits_t(ra), bits_t(rb))
        assert torch.isfinite(a.float()).all()


@pytest.mark.parametrize("m,n,k", [(16, 4608, 3584), (64, 3584, 18944),
                                   (64, 37888, 512), (5, 3584, 3584)])
def test_back_to_back_calls_share_the_workspace(m, n, k):
    """Calls queued back to back on one stream reuse one workspace: the
    partial sums of a K split and the per-group counters. Each of six calls
    with different x (and the fused kinds in between) must equal its own
    product: a partial sum left from the call before, or a counter not
    returned to zero, would show up as a wrong output."""
    from paper_2510_12633_amd.api import SkinnyLinear
    _need_gpu()
    print(f"[gpu-linear-reuse] m={m} n={n} k={k}", flush=True)
    g = torch.Generator(device="cuda").manual_seed(5 * m + n + k)
    w = (torch.randn((n, k), generator=g, device="cuda") / k ** 0.5).to(torch.bfloat16)
    lin = SkinnyLinear(w)
    xs = [torch.randn((m, k), generator=g, device="cuda").to(torch.bfloat16)
          for _ in range(6)]
    ys = [torch.full((m, n), float("nan"), device="cuda") for _ in xs]
    refs = []
    for i, (x, y) in enumerate(zip(xs, ys)):
        lin(x, out=y)
        if i % 2:
            lin.bf16(x.float())                   # fp32 x, same workspace
    torch.cuda.synchronize()
    for x, y in zip(xs, ys):
        ref = (x.float() @ w.float().t())
        tol = 1e-5 * (x.float().abs() @ w.float().abs().t()) + 1e-6
        assert bool(((y - ref).abs() <= tol).all()), (m, n, k)
    assert torch.equal(ys[0], lin(xs[0]))


@pytest.mark.parametrize("n,k", [(4608, 3584), (3584, 18944), (37888, 512)])
def test_calls_of_every_batch_size_share_the_workspace(n, k):
    """One weight called at batch sizes in turn, as a decode step's
    projection is when the batch changes: every path of the split (inside
    the workgroup, finished by a group's last range, added by a second
    kernel, balanced) on one workspace, sized for the largest. Each call
    must equal its own product: a call whose partial sums covered the
    group counters of another batch size would leave that size's later
    calls with no last range, their outputs unwritten (NaN here). The next
    norm and SwiGLU ride along on some calls."""
    from paper_2510_12633_amd.api import SkinnyLinear, rmsnorm, silu_mul
    _need_gpu()
    print(f"[gpu-linear-mixed-m] n={n} k={k}", flush=True)
    g = torch.Generator(device="cuda").manual_seed(n + 3 * k)
    w = (torch.randn((n, k), generator=g, device="cuda") / k ** 0.5).to(torch.bfloat16)
    lin = SkinnyLinear(w)
    nw = (1 + 0.2 * torch.randn((n,), generator=g, device="cuda")).to(torch.bfloat16)
    for i, m in enumerate((16, 64, 8, 32, 128, 3, 16, 40, 64, 8, 17, 128, 32)):
        x = torch.randn((m, k), generator=g, device="cuda").to(torch.bfloat16)
        y = torch.full((m, n), float("nan"), device="cuda")
        lin(x, out=y)
        ref = x.float() @ w.float().t()
        tol = 1e-5 * (x.float().abs() @ w.float().abs().t()) + 1e-6
        torch.cuda.synchronize()
        assert bool(((y - ref).abs() <= tol).all()), (m, n, k, i)
        if i % 3 == 1:
            ya, za = lin.bf16_norm(x, nw, 1e-6)
            zb = rmsnorm(lin.bf16(x), nw, eps=1e-6)
            torch.cuda.synchronize()
            assert torch.equal(bits_t(ya), bits_t(y.to(torch.bfloat16))), (m, i)
            assert torch.equal(bits_t(za), bits_t(zb)), (m, n, k, i)
        elif i % 3 == 2:
            ya, act = lin.bf16_swiglu(x)
            torch.cuda.synchronize()
            assert torch.equal(bits_t(ya), bits_t(y.to(torch.bfloat16))), (m, i)
            assert torch.equal(bits_t(act), bits_t(silu_mul(ya))), (m, n, k, i)


@pytest.mark.parametrize("m,n,k", [(16, 4608, 3584), (32, 3584, 18944),
                                   (64, 37888, 512), (64, 3584, 3584)])
def test_graph_replays_equal_the_eager_call(m, n, k):
    """The product captured in a HIP graph and replayed four times, with
    eager calls on the same workspace between the replays: every replay
    equals the eager result bit for bit (the K split's counters return to
    zero in every call, so a replay starts from the state the capture saw;
    nothing in the call is a memset)."""
    from paper_2510_12633_amd.api import SkinnyLinear
    _need_gpu()
    print(f"[gpu-linear-graph] m={m} n={n} k={k}", flush=True)
    g = torch.Generator(device="cuda").manual_seed(3 * m + n + k)
    w = (torch.randn((n, k), generator=g, device="cuda") / k ** 0.5).to(torch.bfloat16)
    lin = SkinnyLinear(w)
    x = torch.randn((m, k), generator=g, device="cuda").to(torch.bfloat16)
    x2 = torch.randn((m, k), generator=g, device="cuda").to(torch.bfloat16)
    res = torch.randn((m, n), generator=g, device="cuda").to(torch.bfloat16)
    eager = lin.bf16(x, residual=res)
    torch.cuda.synchronize()
    out = torch.empty_like(eager)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        lin.bf16(x, out=out, residual=res)            # warm on the side stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        lin.bf16(x, out=out, residual=res)
    for i in range(4):
        out.fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(bits_t(out), bits_t(eager)), (m, n, k, i)
        other = lin.bf16(x2, residual=res)           # eager, same workspace
        torch.cuda.synchronize()
        assert torch.isfinite(other.float()).all()


POST_SHAPES = [(64, 3584, 3584), (40, 3584, 18944), (128, 4608, 3584),
               (16, 3584, 3584), (4, 3584, 3584), (3, 48, 640),
               (64, 37888, 512), (33, 33024, 384), (64, 32768, 256),
               (16, 37888, 512)]


@pytest.mark.parametrize("m,n,k", POST_SHAPES)
def test_norm_and_swiglu_outputs_equal_the_separate_launches(m, n, k):
    """laminar_linear_bf16_norm and _swiglu against the product followed by
    laminar_rmsnorm / laminar_silu_mul, bit for bit, on every path: the K
    split whose second kernel carries the step (33 rows and more), the K
    split finished inside the kernel, no split, the split over wavefronts,
    and the balanced split with and without groups left over; x in bf16,
    fp32 and gate-and-up form, the residual in place, with and without a
    norm weight."""
    from paper_2510_12633_amd.api import SkinnyLinear, rmsnorm, silu_mul
    _need_gpu()
    print(f"[gpu-linear-post] m={m} n={n} k={k}", flush=True)
    g = torch.Generator(device="cuda").manual_seed(13 * m + n + k)
    w = (torch.randn((n, k), generator=g, device="cuda") / k ** 0.5).to(torch.bfloat16)
    lin = SkinnyLinear(w)
    x = (torch.randn((m, k), generator=g, device="cuda") * 2).to(torch.bfloat16)
    x32 = torch.randn((m, k), generator=g, device="cuda") * 2
    gu = (torch.randn((m, 2 * k), generator=g, device="cuda") * 3).to(torch.bfloat16)
    res = torch.randn((m, n), generator=g, device="cuda").to(torch.bfloat16)
    nw = (1 + 0.2 * torch.randn((n,), generator=g, device="cuda")).to(torch.bfloat16)
    for xin, sw in ((x, False), (x32, False), (gu, True)):
        for weight, eps in ((nw, 1e-6), (None, 0.0)):
            ra, rb = res.clone(), res.clone()
            ya, za = lin.bf16_norm(xin, weight, eps, out=ra, residual=ra, swiglu=sw)
            yb = lin.bf16(xin, out=rb, residual=rb, swiglu=sw)
            zb = rmsnorm(yb, weight, eps=eps)
            torch.cuda.synchronize()
            assert torch.equal(bits_t(ya), bits_t(yb)), (m, n, k, sw)
            assert torch.equal(bits_t(za), bits_t(zb)), (m, n, k, sw)
            assert torch.isfinite(za.float()).all()
    ya, act_a = lin.bf16_swiglu(x)
    yb = lin.bf16(x)
    act_b = silu_mul(yb)
    torch.cuda.synchronize()
    assert torch.equal(bits_t(ya), bits_t(yb)), (m, n, k)
    assert torch.equal(bits_t(act_a), bits_t(act_b)), (m, n, k)
    assert torch.isfinite(act_a.float()).all()


APPEND_SHAPES = [
    # (M, Hq, Hkv, D, K, pool dtype): QKV of 7B at 64 rows and of 32B at 40
    # (the split's reduction stores K and V), at 16 rows (the split finished
    # in the kernel) and 3 rows (the split over wavefronts), where the append
    # is its own launch, and an fp8 pool (its own launch at any size)
    (64, 28, 4, 128, 3584, "bf16"), (40, 40, 8, 128, 5120, "bf16"),
    (16, 28, 4, 128, 3584, "bf16"), (3, 28, 4, 128, 3584, "bf16"),
    (48, 8, 2, 64, 1024, "bf16"), (64, 28, 4, 128, 3584, "fp8_e4m3fn")]


@pytest.mark.parametrize("m,hq,hkv,d,k,kv_dtype", APPEND_SHAPES)
def test_qkv_with_kv_append_equals_the_separate_launches(m, hq, hkv, d, k,
                                                         kv_dtype):
    """laminar_linear_bf16_kv_append against laminar_linear_bf16_ex followed
    by laminar_kv_append on y's K and V columns: y, both pools and the fp8
    scales bit for bit, with a trajectory of length 0, one whose block lies
    past the table and one whose table entry is -1 (nothing stored for any
    of them), on fresh pools of random codes."""
    from paper_2510_12633_amd.api import SkinnyLinear, kv_append, kv_append_desc
    _need_gpu()
    print(f"[gpu-linear-append] m={m} hq={hq} hkv={hkv} d={d} k={k} {kv_dtype}",
          flush=True)
    n = (hq + 2 * hkv) * d
    g = torch.Generator(device="cuda").manual_seed(m + n + k)
    w = (torch.randn((n, k), generator=g, device="cuda") / k ** 0.5).to(torch.bfloat16)
    lin = SkinnyLinear(w)
    x = torch.randn((m, k), generator=g, device="cuda").to(torch.bfloat16)
    blocks = 6
    pages = m * blocks
    table = torch.randperm(pages, generator=g, device="cuda").to(torch.int32)
    table = table.view(m, blocks).contiguous()
    lens = torch.randint(1, blocks * 16 + 1, (m,), generator=g, device="cuda",
                         dtype=torch.int32)
    lens[0] = 0
    lens[1] = blocks * 16 + 5                   # block past the table
    t2 = int(lens[2].item()) - 1
    table[2, t2 // 16] = -1                     # no page
    fp8 = kv_dtype != "bf16"
    if fp8:
        kp = torch.randint(0, 0x78, (pages, hkv, 16 * d), generator=g,
                           device="cuda", dtype=torch.uint8)
        ks = (0.5 + torch.rand((pages, hkv), generator=g, device="cuda"))
    else:
        kp = torch.randn((pages, hkv, 16 * d), generator=g,
                         device="cuda").to(torch.bfloat16)
        ks = None
    vp = kp.flip(0).contiguous()
    vs = None if ks is None else ks.flip(0).contiguous()
    kp2, vp2 = kp.clone(), vp.clone()
    ks2 = None if ks is None else ks.clone()
    vs2 = None if vs is None else vs.clone()
    desc = kv_append_desc(m, hkv, d, pages, blocks, kv_dtype)
    ya = lin.bf16_kv_append(x, desc, hq * d, (hq + hkv) * d, table, lens, kp,
                            vp, ks, vs)
    yb = lin.bf16(x)
    kv_append(yb[:, hq * d:(hq + hkv) * d].view(m, hkv, d),
              yb[:, (hq + hkv) * d:].view(m, hkv, d), table, lens, kp2, vp2,
              ks2, vs2, kv_dtype=kv_dtype)
    torch.cuda.synchronize()
    assert torch.equal(bits_t(ya), bits_t(yb)), (m, n, k)
    assert torch.equal(kp.view(torch.uint8), kp2.view(torch.uint8)), "K pool"
    assert torch.equal(vp.view(torch.uint8), vp2.view(torch.uint8)), "V pool"
    if fp8:
        assert torch.equal(ks.view(torch.int32), ks2.view(torch.int32))
        assert torch.equal(vs.view(torch.int32), vs2.view(torch.int32))
    # the append did happen: the last trajectory's token is in its page
    # (trajectories 0-2 store nothing)
    t = int(lens[-1].item()) - 1
    page = int(table[-1, t // 16].item())
    if not fp8 and m > 3:
        # V element (t, dim) of a tile at ((t / 4) D + dim) 4 + t % 4
        vt = vp[page, 0]
        got = vt[((t % 16) // 4) * d * 4 + (t % 4)::4][:d]
        assert torch.equal(bits_t(got), bits_t(ya[-1, (hq + hkv) * d:(hq + hkv + 1) * d]))
