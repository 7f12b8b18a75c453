"""CPU checks of the repack host code in the library: the consolidation
planner against the oracle (exact plans), its argument errors, and the
migration page assignment."""
import ctypes

import numpy as np
import pytest

from oracle.repack import best_fit_consolidation
from paper_2510_12633_amd import _native as N


def test_planner_matches_oracle_on_the_hand_example():
    used = [10, 40, 25, 95, 60, 30, 100]
    prev = [12, 50, 30, 99, 55, 35, 120]
    reqs = [3, 8, 5, 20, 10, 6, 4]
    assert N.laminar_repack_plan(used, prev, reqs, 100, 16) == [(0, 1), (2, 1)]


@pytest.mark.parametrize("seed", range(200))
def test_planner_matches_oracle_random(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(0, 40))
    scale = int(rng.choice([5, 100, 10 ** 6]))
    used = [int(x) for x in rng.integers(0, scale, n)]
    # some ties on purpose
    if n > 3:
        used[1] = used[2]
    prev = [u + int(d) for u, d in zip(used, rng.integers(-scale // 5 - 1, scale, n))]
    prev = [max(p, 0) for p in prev]
    reqs = [int(x) for x in rng.integers(0, 40, n)]
    c_max = int(rng.integers(0, 3 * scale))
    b_max = int(rng.integers(0, 64))
    want = best_fit_consolidation(used, prev, reqs, c_max, b_max)
    assert N.laminar_repack_plan(used, prev, reqs, c_max, b_max) == want


def test_planner_argument_errors():
    lib = N.lib()
    k = ctypes.c_int32(7)
    st = (N.LaminarRolloutState * 1)()
    i32 = (ctypes.c_int32 * 1)()
    INV = N.LAMINAR_ERR_INVALID_ARG
    assert lib.laminar_repack_plan(None, 0, 10, 4, None, None, ctypes.byref(k)) == N.LAMINAR_OK
    assert k.value == 0
    assert lib.laminar_repack_plan(None, 1, 10, 4, i32, i32, ctypes.byref(k)) == INV
    assert lib.laminar_repack_plan(st, -1, 10, 4, i32, i32, ctypes.byref(k)) == INV
    assert lib.laminar_repack_plan(st, 1, -1, 4, i32, i32, ctypes.byref(k)) == INV
    assert lib.laminar_repack_plan(st, 1, 10, 4, i32, i32, None) == INV
    st[0].kv_used = -5
    assert lib.laminar_repack_plan(st, 1, 10, 4, i32, i32, ctypes.byref(k)) == INV


def test_migration_pairs_dedups_shared_pages():
    # trajectories 0 and 1 share their first two pages (a prompt prefix)
    src = np.array([[7, 3, 9, -1], [7, 3, 4, 11], [5, -1, -1, -1]], np.int32)
    lens = np.array([40, 60, 16], np.int32)
    free = np.array([100, 101, 102, 103, 104, 105, 106, 107], np.int32)
    table, pairs, used = N.laminar_migration_pairs(src, lens, free, 5)
    assert used == 6
    assert pairs.tolist() == [[7, 100], [3, 101], [9, 102], [4, 103],
                              [11, 104], [5, 105]]
    assert table.tolist() == [[100, 101, 102, -1, -1], [100, 101, 103, 104, -1],
                              [105, -1, -1, -1, -1]]
    # mapping pages through the new table gives the same pages back
    m = dict(pairs.tolist())
    for t in range(3):
        nb = -(-lens[t] // 16)
        assert [m[p] for p in src[t, :nb]] == table[t, :nb].tolist()


def test_migration_pairs_errors():
    src = np.array([[1, 2]], np.int32)
    with pytest.raises(N.LaminarError):                  # too few free pages
        N.laminar_migration_pairs(src, np.array([32], np.int32),
                                  np.array([9], np.int32), 4)
    with pytest.raises(N.LaminarError):                  # too wide
        N.laminar_migration_pairs(src, np.array([40], np.int32),
                                  np.arange(8, dtype=np.int32), 4)
    with pytest.raises(N.LaminarError):                  # hole in the row
        N.laminar_migration_pairs(np.array([[1, -1]], np.int32),
                                  np.array([20], np.int32),
                                  np.arange(8, dtype=np.int32), 4)
    t, p, u = N.laminar_migration_pairs(np.zeros((1, 2), np.int32),
                                        np.array([0], np.int32),
                                        np.arange(2, dtype=np.int32), 2)
    assert p.shape == (0, 2) and u == 0 and t.tolist() == [[-1, -1]]


def test_migrate_pages_errors_before_any_launch():
    lib = N.lib()
    INV = N.LAMINAR_ERR_INVALID_ARG
    assert lib.laminar_migrate_pages(16, 4, 32, 4, 16, 64, 0, None) == N.LAMINAR_OK
    assert lib.laminar_migrate_pages(None, 4, 32, 4, 16, 64, 1, None) == INV
    assert lib.laminar_migrate_pages(16, 4, 32, 4, 0, 64, 1, None) == INV
    assert lib.laminar_migrate_pages(16, 4, 32, 4, 6, 64, 1, None) == INV
    assert lib.laminar_migrate_pages(16, 4, 40, 4, 16, 64, 1, None) == INV  # align
    assert lib.laminar_migrate_pages(16, 4, 32, 4, 16, 68, 1, None) == INV  # pairs
    assert lib.laminar_migrate_pages(16, -1, 32, 4, 16, 64, 1, None) == INV


def _shape(m):
    return N.LaminarModelShape(
        layers=m.layers, hidden=m.hidden, q_heads=m.q_heads,
        kv_heads=m.kv_heads, head_dim=m.head_dim, intermediate=m.intermediate,
        vocab=m.vocab, weight_bytes=m.weight_bytes, act_bytes=m.act_bytes,
        kv_bytes=m.kv_bytes)


def test_roofline_bound_matches_oracle():
    from oracle.roofline import QWEN25_7B, QWEN25_32B, ModelShape, batch_bound
    peaks = [(2_500_000_000_000_000, 8_000_000_000_000),
             (5_000_000_000_000_000, 8_000_000_000_000),
             (989_000_000_000_000, 3_350_000_000_000), (10 ** 12, 10 ** 12)]
    shapes = [QWEN25_7B, QWEN25_32B, ModelShape(2, 64, 4, 2, 16, 128, 100),
              ModelShape(1, 2, 1, 1, 2, 2, 2, 2, 64, 2),
              ModelShape(28, 3584, 28, 4, 128, 18944, 152064, 1, 2, 1)]
    for m in shapes:
        for f, bw in peaks:
            want = batch_bound(m, f, bw)
            got = N.laminar_roofline_batch_bound(_shape(m), f, bw)
            assert got == (0 if want is None else want), (m, f, bw)


def test_roofline_step_time_matches_oracle():
    from oracle.roofline import QWEN25_7B, QWEN25_32B, step_time
    f, bw = 2_500_000_000_000_000, 8_000_000_000_000
    for m in (QWEN25_7B, QWEN25_32B):
        for batch in (1, 7, 64, 350, 1024):
            for c in (0, 1, 2048, 98304):
                want = float(step_time(m, batch, c, f, bw))
                got = N.laminar_roofline_step_seconds(_shape(m), batch, c, f, bw)
                assert abs(got - want) <= 1e-12 * want


def test_roofline_argument_errors():
    from oracle.roofline import QWEN25_7B
    s = _shape(QWEN25_7B)
    with pytest.raises(N.LaminarError):
        N.laminar_roofline_batch_bound(s, 0, 10)
    s.layers = 0
    with pytest.raises(N.LaminarError):
        N.laminar_roofline_batch_bound(s, 10, 10)
    with pytest.raises(N.LaminarError):
        N.laminar_roofline_step_seconds(_shape(QWEN25_7B), -1, 0, 10, 10)
