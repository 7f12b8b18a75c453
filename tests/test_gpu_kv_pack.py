"""laminar_kv_pack: row-major (page, kv-head) tiles into the attention
kernels' K and V tile orders, bit for bit against the oracle's tile
addressing, and attention over packed pools equal to attention over the
generator's pools."""
import numpy as np
import pytest
import torch

from oracle.decode_attention import k_tile_offsets, v_tile_offsets
from paper_2510_12633_amd import _native as N
from paper_2510_12633_amd.api import KV_DTYPES, PagedDecodeAttention
from workloads import custom_config, make_workload

pytestmark = pytest.mark.gpu


def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")


@pytest.mark.parametrize("head_dim", [64, 128])
@pytest.mark.parametrize("kv_dtype", ["bf16", "fp8_e4m3fn"])
@pytest.mark.parametrize("which", [0, 1])
@pytest.mark.parametrize("num_tiles", [1, 3, 37 * 3, 5001])
def test_pack_equals_tile_addressing(head_dim, kv_dtype, which, num_tiles):
    """Random bytes (NaN codes included: only bits move) in every tile of a
    pool of 1 .. 5001 tiles, odd counts leaving a workgroup's last pass part
    empty."""
    _need_gpu()
    eb = 2 if kv_dtype == "bf16" else 1
    print(f"[kv-pack] D {head_dim} {kv_dtype} which {which} tiles {num_tiles}",
          flush=True)
    g = torch.Generator().manual_seed(num_tiles * 7 + head_dim + which)
    src = torch.randint(0, 256, (num_tiles, 16 * head_dim * eb), generator=g,
                        dtype=torch.uint8)
    dst = torch.zeros_like(src).cuda()
    N.laminar_kv_pack(src.cuda(), dst, num_tiles, head_dim, KV_DTYPES[kv_dtype],
                      which, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    dt = np.uint16 if eb == 2 else np.uint8
    rows = src.numpy().view(dt).reshape(num_tiles, 16 * head_dim)
    offs = (v_tile_offsets(head_dim) if which else
            k_tile_offsets(head_dim, eb)).reshape(-1)
    want = np.empty_like(rows)
    want[:, offs] = rows
    assert np.array_equal(dst.cpu().numpy().view(dt).reshape(num_tiles, -1), want)


@pytest.mark.parametrize("kv_dtype", ["bf16", "fp8_e4m3fn"])
def test_packed_pools_equal_generated_pools_and_attention(kv_dtype):
    """The generator's logical [P, Hkv, 16, D] pools packed by the library
    equal the pools it lays out itself, and attention over them is the
    same bit for bit."""
    _need_gpu()
    cfg = custom_config([1, 17, 300, 2049, 64], 40 if kv_dtype != "bf16" else 28,
                        8 if kv_dtype != "bf16" else 4, 128, kv_dtype=kv_dtype)
    wl = make_workload(cfg, seed=5, device="cuda", keep_logical=True)
    h = torch.cuda.current_stream().cuda_stream
    c = wl.cfg
    tiles = wl.num_pages * c.num_kv_heads
    kp = torch.empty_like(wl.k_pages)
    vp = torch.empty_like(wl.v_pages)
    N.laminar_kv_pack(wl.k_logical.contiguous(), kp, tiles, c.head_dim,
                      KV_DTYPES[kv_dtype], 0, h)
    N.laminar_kv_pack(wl.v_logical.contiguous(), vp, tiles, c.head_dim,
                      KV_DTYPES[kv_dtype], 1, h)
    torch.cuda.synchronize()
    bits = (lambda t: t.view(torch.int16)) if kv_dtype == "bf16" else (lambda t: t)
    assert torch.equal(bits(kp), bits(wl.k_pages))
    assert torch.equal(bits(vp), bits(wl.v_pages))
    att = PagedDecodeAttention(
        batch=wl.batch, num_q_heads=c.num_q_heads, num_kv_heads=c.num_kv_heads,
        head_dim=c.head_dim, num_pages=wl.num_pages,
        max_blocks_per_seq=wl.block_table.shape[1], seq_lens_host=wl.seq_lens,
        softmax_scale=wl.softmax_scale, kv_dtype=kv_dtype, k_scale=wl.k_scale,
        v_scale=wl.v_scale)
    bt = torch.as_tensor(wl.block_table, device="cuda")
    lens = torch.as_tensor(wl.seq_lens, device="cuda")
    o1, l1 = att(wl.q, wl.k_pages, wl.v_pages, bt, lens)
    o2, l2 = att(wl.q, kp, vp, bt, lens)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(o1).all())
    assert torch.equal(o1, o2) and torch.equal(l1, l2)
    att.close()
