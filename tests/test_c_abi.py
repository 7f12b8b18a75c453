"""CPU checks of the C ABI: exported symbols, the host planner, and the
argument errors returned before any HIP call. No GPU is touched."""
import ctypes
import os
import re
import shutil
import subprocess

import numpy as np
import pytest

from paper_2510_12633_amd import _native as N

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
INCLUDE = os.path.join(ROOT, "include")


def declared_functions():
    names = set()
    for h in sorted(os.listdir(INCLUDE)):
        if h.endswith(".h"):
            text = open(os.path.join(INCLUDE, h)).read()
            text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
            names |= set(re.findall(r"\b(laminar_\w+)\s*\(", text))
    return sorted(names)


def desc(batch=4, hq=28, hkv=4, d=128, pages=10**6, max_blocks=8192,
         kv=N.LAMINAR_KV_BF16, scale=0.1, ppi=0, waves=0, k_scale=None,
         v_scale=None, page_size=16, stride=0):
    return N.LaminarAttnDesc(batch=batch, num_q_heads=hq, num_kv_heads=hkv,
                             head_dim=d, page_size=page_size, num_pages=pages,
                             max_blocks_per_seq=max_blocks, kv_dtype=kv,
                             softmax_scale=scale, k_scale=k_scale,
                             v_scale=v_scale, pages_per_item=ppi,
                             waves_per_item=waves, input_row_stride=stride)


def plan_tables(d, lens, cus=256):
    p = N.laminar_plan_create(d, np.asarray(lens, np.int32), cus)
    try:
        return (N.laminar_plan_items_copy(p), N.laminar_plan_merges_copy(p),
                N.laminar_plan_pages_per_item(p), N.laminar_plan_waves_per_item(p),
                N.laminar_plan_workspace_bytes(p))
    finally:
        N.laminar_plan_destroy(p)


def test_library_exports_every_declared_symbol():
    lib = N.lib()
    names = declared_functions()
    assert len(names) >= 18 and "laminar_kv_append" in names
    for name in names:
        assert hasattr(lib, name), name
    nm = shutil.which("nm")
    if nm:
        out = subprocess.run([nm, "-D", "--defined-only", N.library_path()],
                             capture_output=True, text=True).stdout
        exported = set(re.findall(r"\bT (laminar_\w+)", out))
        assert set(names) <= exported, set(names) - exported


def test_status_strings():
    for st in range(5):
        assert N.laminar_status_string(st) not in ("", "unknown status")
    assert N.laminar_status_string(99) == "unknown status"


def check_xcd_rounds(items, hkv):
    """Items of one (trajectory or cascade chunk, first page) over the
    kv-heads: in every full round of 8 x hkv items, the kv-heads of a group
    sit at indices congruent mod 8 (workgroup k runs on XCD k % 8)."""
    if hkv <= 1:
        return
    key = lambda it: ((int(it[0]) < 0), (-int(it[0]) - 1 if it[0] < 0
                                         else int(it[0])) // hkv, int(it[1]))
    full = len(items) // (8 * hkv) * 8 * hkv
    pos = {}
    for i, it in enumerate(items[:full]):
        pos.setdefault(key(it), []).append(i)
    for k, idx in pos.items():
        assert len(idx) == hkv and len({i % 8 for i in idx}) == 1, (k, idx)


def check_plan(lens, hkv, items, merges, ppi):
    """Coverage, size, ordering and slot invariants of a plan."""
    pages = -(-np.asarray(lens, np.int64) // 16)
    covered = {}
    by_unit = {}
    for unit, p0, p1, slot in items:
        b, h = divmod(int(unit), hkv)
        assert 0 <= p0 <= p1 <= pages[b]
        assert p1 - p0 <= ppi
        by_unit.setdefault(int(unit), []).append((int(p0), int(p1), int(slot)))
        for p in range(p0, p1):
            key = (int(unit), p)
            assert key not in covered
            covered[key] = True
    # every (trajectory, kv-head, page) exactly once; empty units once
    assert len(covered) == int(pages.sum()) * hkv
    assert set(by_unit) == set(range(len(lens) * hkv))
    sizes = [int(p1 - p0) for _, p0, p1, _ in items]
    # longest first for every kv-head; groups of a page range over the
    # kv-heads laid out eight at a time, kv-head-major (one XCD per group)
    for h in range(hkv):
        sub = [sz for (u, _, _, _), sz in zip(items, sizes) if u % hkv == h]
        assert sub == sorted(sub, reverse=True)
    check_xcd_rounds(items, hkv)
    merged = {int(m[0]): (int(m[1]), int(m[2])) for m in merges}
    assert len(merged) == len(merges)
    all_slots = []
    for unit, chunks in by_unit.items():
        sz = [p1 - p0 for p0, p1, _ in sorted(chunks)]   # page order
        if max(sz) - min(sz) > 1:
            # halves: the first ceil(n/2) pieces twice as long as the rest,
            # each half near-equal (batches mixing short and long units)
            k = (len(sz) + 1) // 2
            lng, sht = sz[:k], sz[k:]
            assert max(lng) - min(lng) <= 1 and max(sht) - min(sht) <= 1, sz
            assert 2 * min(sht) - 2 <= min(lng) and max(lng) <= 2 * max(sht) + 2, sz
        if len(chunks) == 1:
            assert chunks[0][2] == -1 and unit not in merged
        else:
            slot0, n = merged[unit]
            assert n == len(chunks)
            got = sorted(s for _, _, s in chunks)
            assert got == list(range(slot0, slot0 + n))
            # slots follow page order inside the unit
            assert [s for _, _, s in sorted(chunks)] == got
            all_slots += got
    assert len(all_slots) == len(set(all_slots))


@pytest.mark.parametrize("seed", range(6))
def test_planner_invariants_random(seed):
    rng = np.random.default_rng(seed)
    b = int(rng.integers(1, 300))
    lens = np.minimum(np.exp(rng.normal(7, 1.5, b)).astype(np.int64), 70000)
    lens[rng.random(b) < 0.05] = 0
    hkv = int(rng.choice([1, 2, 4, 8]))
    for ppi, waves in ((0, 0), (1, 1), (3, 2), (64, 4), (1 << 20, 0)):
        d = desc(batch=b, hq=hkv * int(rng.integers(1, 9)), hkv=hkv, ppi=ppi,
                 waves=waves)
        items, merges, chosen, w, ws = plan_tables(d, lens)
        if ppi:
            assert chosen == ppi
        assert w == (waves or 4)
        check_plan(lens, hkv, items, merges, chosen)
        assert ws % 256 == 0 and ws >= 16 * (len(items) + len(merges))


def test_planner_auto_split_fills_the_gpu():
    """Eight 64k-token trajectories x 4 kv-heads (32 units) still give
    about 1.5 items per resident 4-wave workgroup (512 on 256 CUs)."""
    lens = [65536] * 8
    items, merges, chosen, waves, _ = plan_tables(desc(batch=8), lens)
    assert len(items) >= 700 and len(merges) == 32
    assert chosen % (2 * waves) == 0
    check_plan(lens, 4, items, merges, chosen)


def test_dynamic_tail_is_the_small_end_of_the_list():
    """Items at most half the largest, together at most half the work, are
    handed out dynamically; equal-sized items and cascade plans keep every
    item bound to its workgroup index."""
    rng = np.random.default_rng(3)
    lens = np.minimum(np.exp(rng.normal(np.log(2048), 1.0, 256)).astype(np.int64),
                      32768)
    d = desc(batch=256)
    p = N.laminar_plan_create(d, lens.astype(np.int32), 256)
    try:
        items = N.laminar_plan_items_copy(p)
        dyn = int(N.lib().laminar_plan_num_dynamic_items(p))
    finally:
        N.laminar_plan_destroy(p)
    sizes = items[:, 2] - items[:, 1]
    assert 0 < dyn < len(items)
    tail = sizes[len(items) - dyn:]
    assert tail.max() <= sizes[0] // 2 and 2 * tail.sum() <= sizes.sum()
    # the next larger item would break one of the two limits
    nxt = sizes[len(items) - dyn - 1]
    assert nxt > sizes[0] // 2 or 2 * (tail.sum() + nxt) > sizes.sum()
    # equal pieces: nothing to rebalance
    p = N.laminar_plan_create(desc(batch=8), np.full(8, 40000, np.int32), 256)
    try:
        assert N.lib().laminar_plan_num_dynamic_items(p) == 0
    finally:
        N.laminar_plan_destroy(p)
    # cascade plans keep every item bound
    p = N.laminar_plan_create_cascade(d, lens.astype(np.int32),
                                      np.arange(256, dtype=np.int32) // 8,
                                      np.full(32, 8, np.int32), 256)
    try:
        assert N.lib().laminar_plan_num_dynamic_items(p) == 0
    finally:
        N.laminar_plan_destroy(p)


def test_plan_input_row_stride_checked():
    lens = np.array([5, 17, 300, 0], np.int32)
    for stride, ok in ((0, True), (28 * 128, True), (36 * 128, True),
                       (28 * 128 - 8, False), (36 * 128 + 4, False)):
        try:
            N.laminar_plan_destroy(N.laminar_plan_create(desc(stride=stride),
                                                         lens, 256))
            st = N.LAMINAR_OK
        except N.LaminarError as e:
            st = e.status
        assert st == (N.LAMINAR_OK if ok else N.LAMINAR_ERR_INVALID_ARG), stride


def test_planner_edge_lengths():
    for lens in ([0], [1], [16], [17], [0, 0, 0], [98304], [1, 98304, 0, 15]):
        d = desc(batch=len(lens), hq=64, hkv=8)
        items, merges, chosen, _, _ = plan_tables(d, lens)
        check_plan(lens, 8, items, merges, chosen)
    items, merges, _, _, _ = plan_tables(desc(batch=0), [])
    assert len(items) == 0 and len(merges) == 0


def test_planner_deterministic():
    rng = np.random.default_rng(3)
    lens = rng.integers(0, 40000, 200)
    a = plan_tables(desc(batch=200), lens)
    b = plan_tables(desc(batch=200), lens)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def _status(d, lens, cus=256):
    out = ctypes.c_void_p()
    arr = None if lens is None else np.asarray(lens, np.int32)
    ptr = None if arr is None else arr.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    st = N.lib().laminar_plan_create(None if d is None else ctypes.byref(d),
                                     ptr, cus, ctypes.byref(out))
    if out.value:
        N.laminar_plan_destroy(out.value)
    return st


def test_planner_argument_errors():
    INV, UNS = N.LAMINAR_ERR_INVALID_ARG, N.LAMINAR_ERR_UNSUPPORTED
    assert _status(None, [1]) == INV
    assert _status(desc(batch=1), None) == INV
    assert _status(desc(batch=1), [1], cus=0) == INV
    assert _status(desc(batch=1), [-1]) == INV
    assert _status(desc(batch=1, max_blocks=2), [33]) == INV
    assert _status(desc(batch=1, max_blocks=3), [33]) == N.LAMINAR_OK
    assert _status(desc(batch=1, hq=30, hkv=4), [5]) == INV
    assert _status(desc(batch=1, kv=N.LAMINAR_KV_FP8_E4M3FN), [5]) == INV
    assert _status(desc(batch=1, kv=7), [5]) == INV
    assert _status(desc(batch=1, scale=0.0), [5]) == INV
    assert _status(desc(batch=1, waves=3), [5]) == INV
    assert _status(desc(batch=1, waves=4), [5]) == N.LAMINAR_OK
    assert _status(desc(batch=1, ppi=-1), [5]) == INV
    assert _status(desc(batch=1, pages=0), [5]) == INV
    assert _status(desc(batch=1, page_size=32), [5]) == UNS
    assert _status(desc(batch=1, d=96), [5]) == UNS
    assert _status(desc(batch=1, hq=34, hkv=2), [5]) == UNS
    st = N.lib().laminar_plan_create(ctypes.byref(desc(batch=1)),
                                     np.asarray([5], np.int32).ctypes.data_as(
                                         ctypes.POINTER(ctypes.c_int32)), 256,
                                     None)
    assert st == INV


def test_call_errors_before_any_launch():
    lib = N.lib()
    assert lib.laminar_decode_attn(None, *([None] * 7), None) == \
        N.LAMINAR_ERR_INVALID_ARG
    assert lib.laminar_decode_attn_merge(None, None, None, None) == \
        N.LAMINAR_ERR_INVALID_ARG
    assert lib.laminar_plan_bind_workspace(None, None, 0, None) == \
        N.LAMINAR_ERR_INVALID_ARG
    p = N.laminar_plan_create(desc(batch=2), np.array([40, 9], np.int32), 256)
    try:
        # unbound plan
        assert lib.laminar_decode_attn(p, 16, 16, 16, 16, 16, 16, 16, None) == \
            N.LAMINAR_ERR_WORKSPACE
        assert lib.laminar_decode_attn_partial(p, 16, 16, 16, 16, 16, 16, 16,
                                               None) == N.LAMINAR_ERR_WORKSPACE
        # too small / misaligned workspace
        need = N.laminar_plan_workspace_bytes(p)
        assert lib.laminar_plan_bind_workspace(p, 256, need - 1, None) == \
            N.LAMINAR_ERR_WORKSPACE
        assert lib.laminar_plan_bind_workspace(p, 257, need, None) == \
            N.LAMINAR_ERR_WORKSPACE
        assert lib.laminar_plan_bind_workspace(p, None, need, None) == \
            N.LAMINAR_ERR_WORKSPACE
    finally:
        N.laminar_plan_destroy(p)
    assert lib.laminar_hbm_read(None, 16, None, None) == N.LAMINAR_ERR_INVALID_ARG
    assert lib.laminar_hbm_read(16, 17, 16, None) == N.LAMINAR_ERR_INVALID_ARG
    assert lib.laminar_hbm_copy(16, 16, 8, None) == N.LAMINAR_ERR_INVALID_ARG
    gather = lib.laminar_hbm_gather
    assert gather(None, 4096, 4096, 16, 1, 16, None) == N.LAMINAR_ERR_INVALID_ARG
    assert gather(8, 4096, 4096, 16, 1, 16, None) == N.LAMINAR_ERR_INVALID_ARG
    assert gather(16, 4096, 48, 16, 1, 16, None) == N.LAMINAR_ERR_INVALID_ARG
    assert gather(16, 4096, 8, 16, 1, 16, None) == N.LAMINAR_ERR_INVALID_ARG
    assert gather(16, 2048, 4096, 16, 1, 16, None) == N.LAMINAR_ERR_INVALID_ARG
    assert gather(16, 4096, 4096, None, 1, 16, None) == N.LAMINAR_ERR_INVALID_ARG
    assert gather(16, 4096, 4096, 18, 1, 16, None) == N.LAMINAR_ERR_INVALID_ARG
    assert gather(16, 4096, 4096, 16, -1, 16, None) == N.LAMINAR_ERR_INVALID_ARG
    assert gather(16, 4096, 4096, None, 0, None, None) == N.LAMINAR_OK
    assert lib.laminar_hbm_gather_sink_words(0, 4096) == 0
    assert lib.laminar_hbm_gather_sink_words(1, 4096) == 1
    assert lib.laminar_hbm_gather_sink_words(1 << 20, 4096) == \
        N.laminar_hbm_read_sink_floats()
    assert lib.laminar_plan_num_items(None) == -1
    assert lib.laminar_plan_workspace_bytes(None) == 0


def cascade_tables(d, lens, group_of, group_pages, cus=256):
    p = N.laminar_plan_create_cascade(d, np.asarray(lens, np.int32),
                                      np.asarray(group_of, np.int32),
                                      np.asarray(group_pages, np.int32), cus)
    try:
        return (N.laminar_plan_items_copy(p), N.laminar_plan_merges_copy(p),
                N.laminar_plan_cascade_units_copy(p),
                N.laminar_plan_cascade_members_copy(p),
                N.laminar_plan_waves_per_item(p))
    finally:
        N.laminar_plan_destroy(p)


def check_cascade_plan(lens, hkv, g, group_of, group_pages, items, merges,
                       cunits, cmembers, waves):
    """Every (trajectory, kv-head, page) exactly once, by its own item or by
    a cascade item of a chunk it belongs to; chunk and slot structure."""
    lens = np.asarray(lens, np.int64)
    pages = -(-lens // 16)
    cap = waves * (16 // g)
    covered = {}
    slot_of = {}                     # (unit) -> list of (first page, slot)
    members_of = []
    for cu, (row, cnt, moff, kvh) in enumerate(cunits):
        mem = cmembers[moff:moff + cnt]
        bs = [int(b) for b in mem[:, 0]]
        assert 2 <= cnt <= cap and bs == sorted(bs)
        grp = {int(group_of[b]) for b in bs}
        assert len(grp) == 1 and -1 not in grp
        # the row read is the member with the most tokens (not just pages)
        assert int(row) in bs and lens[row] == max(lens[b] for b in bs)
        members_of.append((bs, mem[:, 1], int(kvh)))
    cost = []
    for unit, p0, p1, slot in items:
        if unit >= 0:
            b, h = divmod(int(unit), hkv)
            assert 0 <= p0 <= p1 <= pages[b]
            for pg in range(p0, p1):
                assert (b, h, pg) not in covered
                covered[(b, h, pg)] = True
            slot_of.setdefault(int(unit), []).append((int(p0), int(slot)))
            cost.append(int(p1 - p0))
        else:
            bs, slot0s, h = members_of[-unit - 1]
            for b, s0 in zip(bs, slot0s):
                for pg in range(p0, min(p1, pages[b])):
                    assert (b, h, pg) not in covered
                    covered[(b, h, pg)] = True
                slot_of.setdefault(b * hkv + h, []).append((-1, int(s0 + slot)))
            cost.append(waves * int(p1 - p0))
    assert len(covered) == int(pages.sum()) * hkv
    for h in range(hkv):
        sub = [c for it, c in zip(items, cost)
               if (int(it[0]) if it[0] >= 0 else -int(it[0]) - 1) % hkv == h]
        assert sub == sorted(sub, reverse=True)
    check_xcd_rounds(items, hkv)
    merged = {int(m[0]): (int(m[1]), int(m[2])) for m in merges}
    all_slots = []
    for unit, lst in slot_of.items():
        if unit in merged:
            s0, n = merged[unit]
            assert n == len(lst)
            # cascade pieces first, then own pieces in page order
            got = [s for _, s in sorted(lst, key=lambda x: (x[0], x[1]))]
            assert got == list(range(s0, s0 + n)), (unit, lst, s0, n)
            all_slots += got
        else:
            assert len(lst) == 1 and lst[0][1] == -1
    assert len(all_slots) == len(set(all_slots))


@pytest.mark.parametrize("seed", range(6))
def test_cascade_planner_invariants_random(seed):
    rng = np.random.default_rng(100 + seed)
    b = int(rng.integers(1, 200))
    lens = rng.integers(0, 6000, b)
    hkv = int(rng.choice([1, 2, 4, 8]))
    g = int(rng.choice([1, 2, 5, 7, 8, 16]))
    n_groups = int(rng.integers(1, 30))
    group_of = rng.integers(-1, n_groups, b)
    group_pages = rng.integers(0, 100, n_groups)
    for ppi, waves in ((0, 0), (1, 1), (6, 2), (64, 4)):
        d = desc(batch=b, hq=hkv * g, hkv=hkv, ppi=ppi, waves=waves)
        items, merges, cunits, cmem, w = cascade_tables(d, lens, group_of,
                                                        group_pages)
        check_cascade_plan(lens, hkv, g, group_of, group_pages, items, merges,
                           cunits, cmem, w)


def test_cascade_plan_of_the_agentic_shape():
    """Groups of 8 sharing 64 pages, g = 8, 4 wavefronts: one cascade unit
    per (group, kv-head) with all 8 members, and no trajectory's own items
    start before page 64 unless it is shorter than the prefix."""
    rng = np.random.default_rng(1)
    b = 64
    lens = np.where(rng.random(b) < 0.1, rng.integers(32768, 98305, b),
                    rng.integers(256, 4097, b))
    group_of = np.arange(b) // 8
    d = desc(batch=b, hq=64, hkv=8, max_blocks=8192)
    items, merges, cunits, cmem, w = cascade_tables(d, lens, group_of,
                                                    np.full(8, 64))
    assert len(cunits) == 8 * 8 and all(cunits[:, 1] == 8)
    check_cascade_plan(lens, 8, 8, group_of, np.full(8, 64), items, merges,
                       cunits, cmem, w)
    own = items[items[:, 0] >= 0]
    b_of = own[:, 0] // 8
    assert np.all(own[:, 1] >= np.minimum(64, -(-lens[b_of] // 16)))
    # no cascade without sharing, or for lone members
    items2, _, cu2, _, _ = cascade_tables(d, lens, group_of, np.zeros(8))
    assert len(cu2) == 0 and np.all(items2[:, 0] >= 0)
    items3, _, cu3, _, _ = cascade_tables(d, lens, np.arange(b), np.full(b, 64))
    assert len(cu3) == 0


def test_cascade_planner_argument_errors():
    d = desc(batch=3)
    lens = np.array([10, 20, 30], np.int32)
    lib = N.lib()
    out = ctypes.c_void_p()
    P = ctypes.POINTER(ctypes.c_int32)

    def st(group_of, n, pages):
        g = np.asarray(group_of, np.int32)
        pg = np.asarray(pages, np.int32)
        return lib.laminar_plan_create_cascade(
            ctypes.byref(d), lens.ctypes.data_as(P), g.ctypes.data_as(P), n,
            pg.ctypes.data_as(P), 256, ctypes.byref(out))

    INV = N.LAMINAR_ERR_INVALID_ARG
    assert st([0, 0, -1], 1, [2]) == N.LAMINAR_OK
    N.laminar_plan_destroy(out.value)
    assert st([0, 0, -1], -1, [2]) == INV
    assert st([0, 2, -1], 2, [2, 2]) == INV          # group out of range
    assert st([0, -2, -1], 1, [2]) == INV
    assert st([0, 0, 0], 1, [-1]) == INV
    assert lib.laminar_plan_create_cascade(ctypes.byref(d), lens.ctypes.data_as(P),
                                           None, 1, None, 256,
                                           ctypes.byref(out)) == INV


def test_kv_append_errors_before_any_launch():
    lib = N.lib()
    INV, UNS = N.LAMINAR_ERR_INVALID_ARG, N.LAMINAR_ERR_UNSUPPORTED

    def call(d, k_new=16, v_new=16, bt=16, lens=16, kp=16, vp=16, ks=16,
             vs=16):
        return lib.laminar_kv_append(
            None if d is None else ctypes.byref(d), k_new, v_new, bt, lens, kp,
            vp, ks, vs, None)

    assert call(None) == INV
    assert call(desc(batch=0)) == N.LAMINAR_OK          # nothing to append
    assert call(desc(batch=-1)) == INV
    assert call(desc(hkv=0)) == INV
    assert call(desc(pages=0)) == INV
    assert call(desc(max_blocks=-1)) == INV
    assert call(desc(kv=7)) == INV
    assert call(desc(stride=4 * 128 - 8)) == INV          # below Hkv x D
    assert call(desc(stride=4 * 128 + 4)) == INV          # not 16-byte rows
    assert call(desc(page_size=32)) == UNS
    assert call(desc(d=96)) == UNS
    assert call(desc(), k_new=None) == INV
    assert call(desc(), lens=None) == INV
    assert call(desc(), vp=None) == INV
    assert call(desc(), k_new=24) == INV                # misaligned
    assert call(desc(), kp=24) == INV
    assert call(desc(), bt=18) == INV                   # 4-byte words
    assert call(desc(), lens=17) == INV
    fp8 = desc(kv=N.LAMINAR_KV_FP8_E4M3FN)
    assert call(fp8, ks=None) == INV
    assert call(fp8, vs=None) == INV
    assert call(fp8, ks=18) == INV
    assert call(fp8, vs=17) == INV


def test_linear_errors_before_any_launch():
    lib = N.lib()
    INV, UNS = N.LAMINAR_ERR_INVALID_ARG, N.LAMINAR_ERR_UNSUPPORTED
    assert lib.laminar_linear(None, 16, 16, 1, 16, 128, None, 0, None) == INV
    assert lib.laminar_linear(16, 24, 16, 1, 16, 128, None, 0, None) == INV
    assert lib.laminar_linear(16, 16, 16, 0, 16, 128, None, 0, None) == UNS
    assert lib.laminar_linear(16, 16, 16, 129, 16, 128, None, 0, None) == UNS
    assert lib.laminar_linear(16, 16, 16, 1, 24, 128, None, 0, None) == UNS
    assert lib.laminar_linear(16, 16, 16, 1, 16, 100, None, 0, None) == UNS
    assert lib.laminar_linear(16, 16, 16, 1, 16, (1 << 24) + 128, None, 0,
                              None) == UNS
    # bf16 output: NULL output, misaligned residual, shapes
    assert lib.laminar_linear_bf16(16, 16, None, None, 1, 16, 128, None, 0,
                                   None) == INV
    assert lib.laminar_linear_bf16(16, 16, 16, 24, 1, 16, 128, None, 0,
                                   None) == INV
    assert lib.laminar_linear_bf16(16, 16, 16, None, 129, 16, 128, None, 0,
                                   None) == UNS
    # fused x kinds: unknown kind, misaligned x, x offsets past 31 bits
    ex = lib.laminar_linear_bf16_ex
    assert ex(16, 3, 16, 16, None, 1, 16, 128, None, 0, None) == INV
    assert ex(16, -1, 16, 16, None, 1, 16, 128, None, 0, None) == INV
    assert ex(24, N.LAMINAR_X_F32, 16, 16, None, 1, 16, 128, None, 0, None) == INV
    assert ex(16, N.LAMINAR_X_SILU_MUL, 16, None, None, 1, 16, 128, None, 0,
              None) == INV
    assert ex(16, N.LAMINAR_X_F32, 16, 16, None, 128, 16, 1 << 22, None, 0,
              None) == UNS                      # 128 rows x 16 MiB of fp32
    assert ex(16, N.LAMINAR_X_SILU_MUL, 16, 16, None, 65, 16, 1 << 22, None,
              0, None) == UNS                   # 128 padded rows x 16 MiB of gate+up
    assert lib.laminar_linear(16, 16, 16, 128, 16, 1 << 23, None, 0,
                              None) == UNS      # 128 rows x 16 MiB of bf16
    assert ex(16, 3, 16, 16, None, 1, 16, 128, None, 0, None) == INV
    # the fused norm: weight, eps, at most 4 rows
    f = ctypes.c_float
    nm = lib.laminar_linear_bf16_rmsnorm
    assert nm(16, None, f(1e-6), 16, 16, None, 1, 16, 128, None, 0, None) == INV
    assert nm(16, 24, f(1e-6), 16, 16, None, 1, 16, 128, None, 0, None) == INV
    assert nm(16, 16, f(-1.0), 16, 16, None, 1, 16, 128, None, 0, None) == INV
    assert nm(16, 16, f(float("inf")), 16, 16, None, 1, 16, 128, None, 0,
              None) == INV
    assert nm(16, 16, f(1e-6), 16, None, None, 1, 16, 128, None, 0, None) == INV
    assert nm(16, 16, f(1e-6), 16, 16, None, 9, 16, 128, None, 0, None) == UNS
    # the product with the next step: NULL or misaligned outputs, the norm's
    # eps, the RMS-norm kind of x (it has its own call)
    f = N.ctypes.c_float
    nrm = lib.laminar_linear_bf16_norm
    assert nrm(16, 0, 16, 16, None, 16, f(1e-6), None, 1, 16, 128, None, 0,
               None) == INV
    assert nrm(16, 0, 16, 16, None, 16, f(1e-6), 24, 1, 16, 128, None, 0,
               None) == INV
    assert nrm(16, 0, 16, 16, None, 40, f(1e-6), 32, 1, 16, 128, None, 0,
               None) == INV
    assert nrm(16, 0, 16, 16, None, 16, f(-1.0), 32, 1, 16, 128, None, 0,
               None) == INV
    assert nrm(16, 0, 16, 16, None, 16, f(float("nan")), 32, 1, 16, 128, None,
               0, None) == INV
    assert nrm(16, 3, 16, 16, None, 16, f(1e-6), 32, 1, 16, 128, None, 0,
               None) == INV
    assert nrm(16, 0, 16, None, None, 16, f(1e-6), 32, 1, 16, 128, None, 0,
               None) == INV
    assert nrm(16, 0, 16, 16, None, 16, f(1e-6), 32, 129, 16, 128, None, 0,
               None) == UNS
    sw = lib.laminar_linear_bf16_swiglu
    assert sw(16, 0, 16, 16, None, 1, 32, 128, None, 0, None) == INV
    assert sw(16, 0, 16, 16, 24, 1, 32, 128, None, 0, None) == INV
    assert sw(16, 3, 16, 16, 32, 1, 32, 128, None, 0, None) == INV
    assert sw(16, 0, 16, None, 32, 1, 32, 128, None, 0, None) == INV
    assert sw(16, 0, 16, 16, 32, 1, 24, 128, None, 0, None) == UNS
    # packing: NULL, in place, misaligned, shapes
    assert lib.laminar_linear_pack(None, 16, 16, 128, None) == INV
    assert lib.laminar_linear_pack(16, 16, 16, 128, None) == INV
    assert lib.laminar_linear_pack(16, 40, 16, 128, None) == INV
    assert lib.laminar_linear_pack(16, 32, 24, 128, None) == UNS
    assert lib.laminar_linear_pack(16, 32, 16, 100, None) == UNS
    # a K split needs a workspace
    assert N.laminar_linear_splits(64, 3584, 18944) > 1
    need = N.laminar_linear_workspace_bytes(64, 3584, 18944)
    assert need >= 64 * 3584 * 4 * 2
    assert lib.laminar_linear(16, 16, 16, 64, 3584, 18944, None, 0, None) == INV
    assert lib.laminar_linear(16, 16, 16, 64, 3584, 18944, 256, need - 1,
                              None) == INV
    assert N.laminar_linear_splits(1, 152064, 3584) == 1
    assert N.laminar_linear_workspace_bytes(1, 152064, 3584) == 0
    # up to 4 rows and 160 steps of K the split stays inside a workgroup
    for m, n, k in ((1, 3584, 3584), (4, 3584, 18944), (3, 48, 640)):
        assert N.laminar_linear_splits(m, n, k) == 1
        assert N.laminar_linear_workspace_bytes(m, n, k) == 0
    assert N.laminar_linear_splits(5, 3584, 3584) > 1
    assert N.laminar_linear_splits(1, 5120, 27648) > 1     # 216 steps
    assert N.laminar_linear_splits(0, 16, 128) == 0
    # the balanced split (from 17 rows, uneven group grids): gate and up of
    # 7B is 296 groups, one full round and 40 left over, cut into pieces of
    # 4 or 5 steps of K (at most 7 per group) with two partial slots per
    # workgroup, after the 256 group counters every shape keeps at the start
    # of the workspace (so calls of any M can share one)
    ctrl = 256 * 4
    assert N.laminar_linear_splits(64, 37888, 3584) == 7
    assert (N.laminar_linear_workspace_bytes(64, 37888, 3584)
            == ctrl + 2 * 256 * 64 * 128 * 4)
    # the group split: the counters, then its ranges of partial sums: QKV
    # of 7B at 64 rows is 36 groups of 8 tiles in 7 ranges
    assert N.laminar_linear_splits(64, 4608, 3584) == 7
    assert (N.laminar_linear_workspace_bytes(64, 4608, 3584)
            == ctrl + 7 * 64 * 4608 * 4)
    # an even grid keeps the group split up to 64 rows: the LM head (1188
    # groups, 5 rounds); from 65 rows any grid past 256 workgroups is
    # balanced (1188 = 4 full rounds and 164 left over)
    assert N.laminar_linear_splits(64, 152064, 3584) == 1
    assert N.laminar_linear_workspace_bytes(64, 152064, 3584) == 0
    assert N.laminar_linear_splits(128, 152064, 3584) > 1
    # one row tile keeps the group split
    assert N.laminar_linear_workspace_bytes(16, 37888, 3584) == 0


def test_planner_under_address_and_ub_sanitizers(tmp_path):
    gxx = shutil.which("g++")
    if not gxx:
        pytest.skip("g++ not available")
    exe = tmp_path / "plan_check"
    src = os.path.join(ROOT, "tests", "plan_check.cpp")
    plan = os.path.join(ROOT, "paper_2510_12633_amd", "csrc", "plan.cpp")
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-I", os.path.join(ROOT, "include"),
           "-I", os.path.dirname(plan), src, plan, "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    env = dict(os.environ,
               ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env,
                       timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "plan_check OK" in r.stdout


def test_repack_host_code_under_address_and_ub_sanitizers(tmp_path):
    """Algorithm 1, the page assignment of a migration and the roofline
    bound over random and edge-case inputs, built with g++ under ASan and
    UBSan; every returned index and count is checked."""
    gxx = shutil.which("g++")
    if not gxx:
        pytest.skip("g++ not available")
    exe = tmp_path / "repack_check"
    src = os.path.join(ROOT, "tests", "repack_check.cpp")
    repack = os.path.join(ROOT, "paper_2510_12633_amd", "csrc", "repack.cpp")
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-I", os.path.join(ROOT, "include"),
           src, repack, "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    env = dict(os.environ,
               ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env,
                       timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "repack_check OK" in r.stdout


def test_attention_kernels_do_not_spill_in_the_page_loop():
    """The page-pair double buffer fills most of the register file. A spill
    inside the page loop costs ~15% of bandwidth, so no attention kernel
    instantiation may use scratch at all (the loop check below names the
    offending lines if one ever does), and every instantiation keeps two
    wavefronts per SIMD."""
    from paper_2510_12633_amd import build as B
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    src = os.path.join(B.CSRC, "decode_attn.hip")
    base = [hipcc, "--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang",
            "-target-feature", "-Xclang", "-packed-fp32-ops", "-I", B.INCLUDE,
            "-I", B.CSRC]
    r = subprocess.run(base + ["-c", src, "-o", os.devnull,
                               "-Rpass-analysis=kernel-resource-usage"],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    names = re.findall(r"Function Name: (\S+)", r.stderr)
    scratch = [int(x) for x in
               re.findall(r"ScratchSize \[bytes/lane\]: (\d+)", r.stderr)]
    occ = [int(x) for x in re.findall(r"Occupancy \[waves/SIMD\]: (\d+)",
                                      r.stderr)]
    assert len(names) == len(scratch) == len(occ) and names
    kernels = [(n, sc, o) for n, sc, o in zip(names, scratch, occ)
               if "decode_items" in n]
    assert len(kernels) == 24   # 2 head dims x 2 dtypes x 3 waves x cascade
    assert all(sc == 0 and o >= 2 for _, sc, o in kernels), kernels
    r = subprocess.run(base + ["--cuda-device-only", "-S", src, "-o", "-"],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    in_loop, fn, bad = False, None, []
    for line in r.stdout.splitlines():
        m = re.match(r"^(\w+):", line)
        if m and "decode_items" in m.group(1):
            fn, in_loop = m.group(1), False
        if line.startswith(".LBB") or line.startswith("; %bb."):
            in_loop = "Loop" in line
        if fn and in_loop and "scratch_" in line:
            bad.append((fn, line.strip()))
        if line.strip() == "s_endpgm":
            fn = None
    assert not bad, bad[:4]


def test_decode_step_errors_before_any_launch():
    lib = N.lib()
    INV = N.LAMINAR_ERR_INVALID_ARG
    f = ctypes.c_float
    assert lib.laminar_rmsnorm(None, None, 16, 1, 64, f(1e-6), None) == INV
    assert lib.laminar_rmsnorm(16, None, 24, 1, 64, f(1e-6), None) == INV
    assert lib.laminar_rmsnorm(16, 8, 32, 1, 64, f(1e-6), None) == INV
    assert lib.laminar_rmsnorm(16, None, 32, 1, 60, f(1e-6), None) == INV
    assert lib.laminar_rmsnorm(16, None, 32, 0, 64, f(1e-6), None) == INV
    assert lib.laminar_rmsnorm(16, None, 32, 1, 64, f(-1.0), None) == INV
    assert lib.laminar_rmsnorm(16, None, 32, 1, 64, f(float("nan")), None) == INV
    assert lib.laminar_silu_mul(None, 16, 1, 64, None) == INV
    assert lib.laminar_silu_mul(16, 40, 1, 64, None) == INV
    assert lib.laminar_silu_mul(16, 32, 1, 12, None) == INV
    assert lib.laminar_silu_mul(16, 32, 0, 64, None) == INV


def test_linear_kernels_use_no_scratch():
    """The projection kernels keep every pipeline buffer in registers: no
    scratch at all, and at least two wavefronts per SIMD."""
    from paper_2510_12633_amd import build as B
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    src = os.path.join(B.CSRC, "linear.hip")
    r = subprocess.run([hipcc, "--offload-arch=gfx950", "-O3", "-std=c++17",
                        "-Xclang", "-target-feature", "-Xclang",
                        "-packed-fp32-ops", "-I", B.INCLUDE, "-I", B.CSRC,
                        "-c", src, "-o", os.devnull,
                        "-Rpass-analysis=kernel-resource-usage"],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    names = re.findall(r"Function Name: (\S+)", r.stderr)
    scratch = [int(x) for x in
               re.findall(r"ScratchSize \[bytes/lane\]: (\d+)", r.stderr)]
    occ = [int(x) for x in re.findall(r"Occupancy \[waves/SIMD\]: (\d+)",
                                      r.stderr)]
    kernels = [(n, sc, o) for n, sc, o in zip(names, scratch, occ)
               if "linear_kernel" in n or "linear_wave_split" in n]
    # 16, 32, 64 and 128 batch rows and the split over wavefronts for bf16,
    # fp32 and gate-and-up x; one tile and the split over wavefronts for the
    # fused norm
    assert len(kernels) == 17, kernels
    assert all(sc == 0 for _, sc, o in kernels), kernels
    # two wavefronts per SIMD for the workgroup split up to 64 rows (the
    # 128-row kernels hold two tiles' accumulators for 128 rows and run one
    # per SIMD, which measured faster than one tile at two); the split over
    # wavefronts, which runs up to 1024 tiles in one grid, keeps them all
    # resident with four per SIMD (three with the fused norm's prologue,
    # which only delays a second round of workgroups past 768 tiles)
    for n, _, o in kernels:
        if "wave_split" in n:
            assert o >= (3 if "ILi3E" in n else 4), (n, o)
        elif "linear_kernelILi8E" not in n:
            assert o >= 2, (n, o)
    # the balanced split: 32, 64 and 128 rows for bf16, fp32 and gate-and-up
    # x, eight wavefronts (two per SIMD) in the one workgroup per CU
    balanced = [(n, sc, o) for n, sc, o in zip(names, scratch, occ)
                if "linear_balanced_kernel" in n]
    assert len(balanced) == 9, balanced
    assert all(sc == 0 and o >= 2 for _, sc, o in balanced), balanced


def test_attention_pointer_alignment_checked_before_any_launch():
    """q, k_pages, v_pages and out are read or written in 16-byte vectors,
    block_table, seq_lens and lse in 4-byte words: a pointer off that
    alignment (a sliced tensor) is refused before the workspace is even
    looked at, so an unbound plan still reports INVALID_ARG for it."""
    lib = N.lib()
    p = N.laminar_plan_create(desc(batch=2), np.array([40, 9], np.int32), 256)
    try:
        good = [4096] * 7           # q, k, v, table, lens, out, lse
        for fn in (lib.laminar_decode_attn, lib.laminar_decode_attn_partial):
            assert fn(p, *good, None) == N.LAMINAR_ERR_WORKSPACE
            for i, need in enumerate((16, 16, 16, 4, 4, 16, 4)):
                for off in {need // 2, 2} - {0}:
                    if off % need == 0:
                        continue
                    bad = list(good)
                    bad[i] += off
                    assert fn(p, *bad, None) == N.LAMINAR_ERR_INVALID_ARG, (i, off)
                bad = list(good)
                bad[i] = None
                assert fn(p, *bad, None) == N.LAMINAR_ERR_INVALID_ARG, i
        merge = lib.laminar_decode_attn_merge
        assert merge(p, 4096, 4096, None) == N.LAMINAR_ERR_WORKSPACE
        assert merge(p, 4096 + 8, 4096, None) == N.LAMINAR_ERR_INVALID_ARG
        assert merge(p, 4096, 4096 + 2, None) == N.LAMINAR_ERR_INVALID_ARG
        assert merge(p, None, 4096, None) == N.LAMINAR_ERR_INVALID_ARG
    finally:
        N.laminar_plan_destroy(p)
    # fp8 scales are read as 4-byte words
    with pytest.raises(N.LaminarError) as e:
        N.laminar_plan_create(desc(kv=N.LAMINAR_KV_FP8_E4M3FN, k_scale=4098,
                                   v_scale=4096), np.array([40, 9, 1, 1], np.int32), 256)
    assert e.value.status == N.LAMINAR_ERR_INVALID_ARG


def test_kv_pack_errors_before_any_launch():
    pack = N.lib().laminar_kv_pack
    bf, f8 = N.LAMINAR_KV_BF16, N.LAMINAR_KV_FP8_E4M3FN
    big = 1 << 40
    assert pack(None, None, 0, 128, bf, 0, None) == N.LAMINAR_OK
    assert pack(None, big, 1, 128, bf, 0, None) == N.LAMINAR_ERR_INVALID_ARG
    assert pack(big, None, 1, 128, bf, 1, None) == N.LAMINAR_ERR_INVALID_ARG
    assert pack(big + 8, 2 * big, 1, 128, bf, 0, None) == N.LAMINAR_ERR_INVALID_ARG
    assert pack(big, 2 * big + 4, 1, 128, f8, 0, None) == N.LAMINAR_ERR_INVALID_ARG
    # overlapping buffers (one tile is 4 KiB in bf16 at head_dim 128)
    assert pack(big, big + 4096 - 16, 1, 128, bf, 0, None) == N.LAMINAR_ERR_INVALID_ARG
    assert pack(big + 4096 - 16, big, 1, 128, bf, 0, None) == N.LAMINAR_ERR_INVALID_ARG
    assert pack(big, 2 * big, -1, 128, bf, 0, None) == N.LAMINAR_ERR_INVALID_ARG
    assert pack(big, 2 * big, 1, 128, bf, 2, None) == N.LAMINAR_ERR_INVALID_ARG
    assert pack(big, 2 * big, 1, 128, 7, 0, None) == N.LAMINAR_ERR_INVALID_ARG
    assert pack(big, 2 * big, 1, 96, bf, 0, None) == N.LAMINAR_ERR_UNSUPPORTED


def test_linear_kv_append_errors_before_any_launch():
    """laminar_linear_bf16_kv_append refuses, before any launch, what
    laminar_kv_append refuses and a description or K / V columns that do
    not fit the product: NULL kv_desc, batch != M, columns not a multiple of
    8, past N or overlapping."""
    from paper_2510_12633_amd.api import kv_append_desc
    lib = N.lib()
    INV = N.LAMINAR_ERR_INVALID_ARG
    m, n, k = 64, 4608, 3584
    ws = N.laminar_linear_workspace_bytes(m, n, k)
    good = dict(x=4096, kind=0, w=4096, y=4096, m=m, n=n, k=k, ws=4096,
                wsb=ws, desc=kv_append_desc(m, 4, 128, 1024, 8), kc=3584,
                vc=4096, table=4096, lens=4096, kp=4096, vp=4096)

    def call(**over):
        a = dict(good, **over)
        d = a["desc"]
        return lib.laminar_linear_bf16_kv_append(
            a["x"], a["kind"], a["w"], a["y"], a["m"], a["n"], a["k"], a["ws"],
            a["wsb"], ctypes.byref(d) if d is not None else None, a["kc"],
            a["vc"], a["table"], a["lens"], a["kp"], a["vp"], None, None, None)

    assert call(desc=None) == INV
    assert call(desc=kv_append_desc(m - 1, 4, 128, 1024, 8)) == INV
    assert call(kc=3588) == INV                 # not a multiple of 8
    assert call(vc=4608 - 256) == INV           # V past N
    assert call(kc=3584, vc=3584 + 256) == INV  # overlapping
    assert call(kc=-8) == INV
    assert call(table=4098) == INV              # as laminar_kv_append
    assert call(kp=4104) == INV
    assert call(lens=None) == INV
    assert call(desc=kv_append_desc(m, 4, 96, 1024, 8)) == N.LAMINAR_ERR_UNSUPPORTED
    assert call(desc=kv_append_desc(m, 4, 128, 1024, 8, "fp8_e4m3fn")) == INV
