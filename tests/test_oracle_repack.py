"""Pins of the repack oracle: a hand-worked example, a closed form for
identical rollouts, brute-force feasibility and optimality bounds on small
instances, and the page migration's invariance of attention."""
import itertools
import os

import numpy as np
import pytest

from oracle import decode_attention_from_host
from oracle.repack import best_fit_consolidation, candidates, migrate_pages
from workloads import custom_config, host_arrays, make_workload

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def load_example():
    used, prev, reqs, pairs = [], [], [], []
    c_max = b_max = None
    for line in open(os.path.join(GOLDEN, "repack_example.txt")):
        f = line.split()
        if not f or f[0].startswith("#"):
            continue
        if f[0] == "c_max":
            c_max = int(f[1])
        elif f[0] == "b_max":
            b_max = int(f[1])
        elif f[0] == "rollout":
            assert int(f[1]) == len(used)
            used.append(int(f[2])); prev.append(int(f[3])); reqs.append(int(f[4]))
        elif f[0] == "pair":
            pairs.append((int(f[1]), int(f[2])))
    return used, prev, reqs, c_max, b_max, pairs


def test_hand_worked_example():
    used, prev, reqs, c_max, b_max, want = load_example()
    assert candidates(used, prev, reqs, c_max, b_max) == [0, 1, 2, 5]
    assert best_fit_consolidation(used, prev, reqs, c_max, b_max) == want


@pytest.mark.parametrize("n,k", [(1, 3), (2, 2), (7, 3), (12, 4), (9, 1), (10, 5)])
def test_identical_rollouts_fill_destinations_to_the_limit(n, k):
    """n rollouts of u pages each, limit k*u: destinations take k-1 sources
    each, so n - ceil(n/k) rollouts are released."""
    u = 10
    plan = best_fit_consolidation([u] * n, [u + 1] * n, [1] * n, k * u, 10 ** 6)
    assert len(plan) == n - -(-n // k)


def feasible(plan, used, reqs, c_max, b_max, cands):
    srcs = [s for s, _ in plan]
    dsts = {d for _, d in plan}
    if len(set(srcs)) != len(srcs) or dsts & set(srcs):
        return False
    if not all(s in cands and d in cands for s, d in plan):
        return False
    for d in dsts:
        c = used[d] + sum(used[s] for s, dd in plan if dd == d)
        n = reqs[d] + sum(reqs[s] for s, dd in plan if dd == d)
        if c > c_max or n > b_max:
            return False
    return True


def brute_force_max_released(used, reqs, c_max, b_max, cands):
    best = 0
    for assign in itertools.product([None] + list(cands), repeat=len(cands)):
        plan = [(s, d) for s, d in zip(cands, assign) if d is not None and d != s]
        if len(plan) <= best:
            continue
        if feasible(plan, used, reqs, c_max, b_max, cands):
            best = len(plan)
    return best


@pytest.mark.parametrize("seed", range(40))
def test_brute_force_feasible_and_bounded(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 8))
    used = [int(x) for x in rng.integers(0, 60, n)]
    prev = [u + int(d) for u, d in zip(used, rng.integers(-5, 20, n))]
    reqs = [int(x) for x in rng.integers(0, 12, n)]
    c_max, b_max = int(rng.integers(20, 120)), int(rng.integers(4, 24))
    cands = candidates(used, prev, reqs, c_max, b_max)
    plan = best_fit_consolidation(used, prev, reqs, c_max, b_max)
    assert feasible(plan, used, reqs, c_max, b_max, cands)
    opt = brute_force_max_released(used, reqs, c_max, b_max, cands)
    assert len(plan) <= opt
    assert (opt >= 1) == (len(plan) >= 1)


def test_candidate_filter_edges():
    # falling and under both limits -> candidate; equal to prev, at c_max or
    # at b_max -> not
    used, prev, reqs = [5, 5, 10, 5, 5], [6, 5, 11, 6, 6], [1, 1, 1, 4, 3]
    assert candidates(used, prev, reqs, c_max=10, b_max=4) == [0, 4]


def test_migration_preserves_attention():
    """Pages copied to other physical pages with the block table rewritten:
    the attention oracle gives bitwise the same result."""
    cfg = custom_config([40, 17, 300], 8, 2, 64)
    wl = make_workload(cfg, seed=2)
    a = host_arrays(wl)
    out0, lse0 = decode_attention_from_host(a)
    rng = np.random.default_rng(0)
    n_pages = a["k_pages"].shape[0]
    dst = rng.permutation(2 * n_pages)[:n_pages]           # a bigger pool
    pairs = np.stack([np.arange(n_pages), dst], axis=1)
    big_k = np.zeros((2 * n_pages,) + a["k_pages"].shape[1:], a["k_pages"].dtype)
    big_v = np.zeros_like(big_k)
    a2 = dict(a)
    a2["k_pages"] = migrate_pages(a["k_pages"], big_k, pairs)
    a2["v_pages"] = migrate_pages(a["v_pages"], big_v, pairs)
    bt = a["block_table"]
    a2["block_table"] = np.where(bt >= 0, dst[np.maximum(bt, 0)], -1).astype(np.int32)
    out1, lse1 = decode_attention_from_host(a2)
    assert np.array_equal(out0, out1) and np.array_equal(lse0, lse1)


def _literal_algorithm1(used, prev, reqs, c_max, b_max):
    """Algorithm 1 of §5.2 taken word for word: a visited candidate is
    skipped only when it was emptied; CanFit counts the destination's own
    usage, what is planned into it and the source's own usage."""
    s_list = sorted(candidates(used, prev, reqs, c_max, b_max),
                    key=lambda r: used[r])
    plan, emptied = [], set()
    for s in s_list:
        if s in emptied:
            continue
        into = lambda d: [x for x, dd in plan if dd == d]
        fits = [d for d in s_list if d != s and d not in emptied
                and used[d] + sum(used[x] for x in into(d)) + used[s] <= c_max
                and reqs[d] + sum(reqs[x] for x in into(d)) + reqs[s] <= b_max]
        if not fits:
            continue
        best = max(used[d] + sum(used[x] for x in into(d)) for d in fits)
        plan.append((s, next(d for d in fits
                             if used[d] + sum(used[x] for x in into(d)) == best)))
        emptied.add(s)
    return plan


def _final_loads(plan, used, reqs):
    """Usage and trajectory count of every rollout once the plan has run:
    a moved rollout takes everything it holds, including what was planned
    into it, to its destination."""
    dest = dict(plan)

    def home(r):
        while r in dest:
            r = dest[r]
        return r
    c = [0] * len(used)
    n = [0] * len(used)
    for r in range(len(used)):
        c[home(r)] += used[r]
        n[home(r)] += reqs[r]
    return c, n


def test_literal_loop_breaks_the_limit_on_the_worked_example():
    """Why the oracle keeps a destination in place: on the worked example
    the literal loop also moves rollout 1, which already received 0 and 2,
    into rollout 5, and rollout 5 then ends above C_max (105 > 100 pages)
    and above B (22 > 16 trajectories). The oracle's plan stays within
    both bounds."""
    used, prev, reqs, c_max, b_max, want = load_example()
    literal = _literal_algorithm1(used, prev, reqs, c_max, b_max)
    assert literal == want + [(1, 5)]
    c, n = _final_loads(literal, used, reqs)
    assert c[5] == 105 > c_max and n[5] == 22 > b_max
    c, n = _final_loads(want, used, reqs)
    for _, d in want:
        assert c[d] <= c_max and n[d] <= b_max
