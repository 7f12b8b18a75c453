"""GPU checks of the HBM calibration kernels the bench reports its ceilings
from: the random-tile gather's checksum against the host's sum of the same
words, and the copy kernel's bytes."""
import numpy as np
import pytest
import torch

from paper_2510_12633_amd import _native as N

pytestmark = pytest.mark.gpu


def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")


@pytest.mark.parametrize("tile_bytes,n_tiles,n_idx", [
    (4096, 1024, 5000), (64, 4096, 77777), (16, 64, 3), (4096, 3, 1),
    (1 << 16, 40, 100)])
def test_gather_checksum(tile_bytes, n_tiles, n_idx):
    """Sum mod 2^32 of every 32-bit word of the listed tiles, repeats and
    all, as the host computes it; out-of-range indices read the last tile."""
    _need_gpu()
    print(f"[calib] gather tile {tile_bytes} B x {n_idx}", flush=True)
    g = torch.Generator().manual_seed(tile_bytes + n_idx)
    words = torch.randint(0, 1 << 31, (n_tiles * tile_bytes // 4,), generator=g,
                          dtype=torch.int64).to(torch.int32)
    idx = torch.randint(0, n_tiles, (n_idx,), generator=g, dtype=torch.int32)
    idx[::97] = n_tiles + 5          # clamped to the last tile
    src = words.cuda()
    sink = torch.zeros(max(N.laminar_hbm_gather_sink_words(n_idx, tile_bytes), 1),
                       dtype=torch.int32, device="cuda")
    d_idx = idx.cuda()
    N.laminar_hbm_gather(src, n_tiles * tile_bytes, tile_bytes, d_idx, n_idx,
                         sink, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    got = int(sink.cpu().numpy().view(np.uint32).astype(np.uint64).sum()) & 0xFFFFFFFF
    tiles = words.numpy().view(np.uint32).reshape(n_tiles, -1).astype(np.uint64)
    per_tile = tiles.sum(axis=1)
    want = int(per_tile[np.minimum(idx.numpy(), n_tiles - 1)].sum()) & 0xFFFFFFFF
    assert got == want


def test_copy_and_read():
    _need_gpu()
    n = (3 << 20) + 48
    src = torch.randint(0, 256, (n,), dtype=torch.uint8, device="cuda")
    dst = torch.zeros_like(src)
    h = torch.cuda.current_stream().cuda_stream
    N.laminar_hbm_copy(dst, src, n, h)
    sink = torch.zeros(N.laminar_hbm_read_sink_floats(), dtype=torch.float32,
                       device="cuda")
    N.laminar_hbm_read(src, n, sink, h)
    torch.cuda.synchronize()
    assert torch.equal(dst, src)
    assert bool(torch.isfinite(sink).all())
