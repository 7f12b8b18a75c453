"""CPU oracle for trajectory repacking: the best-fit consolidation plan and
the page migration that carries it out on one GPU.

TEST INFRASTRUCTURE. Only the tests, the package smoke check and the bench's
CPU-baseline leg may import or call this module. The GPU library never does,
and this module imports nothing from the GPU path.

Consolidation (Algorithm 1, §5.2 "Repacking algorithm"). Each rollout
replica r reports its KV-cache usage r.used, its usage at the previous check
r.prev and its running trajectory count r.reqs. With the usage limit c_max
and the roofline batch bound b_max:

  1. Candidates are the rollouts whose usage is falling and below the limit,
     used < min(c_max, prev), and that run fewer than b_max trajectories.
  2. Candidates are visited in increasing usage (smallest first: they are
     the easiest to place elsewhere).
  3. A visited candidate s that has not been emptied looks for destinations
     d among the other candidates that are not emptied and can take it: the
     usage of d plus everything already planned into d plus s.used stays
     within c_max, and likewise the trajectory counts stay within b_max.
  4. Among those, s goes to the destination that ends up fullest (largest
     d.used plus what is already planned into it); s is recorded as emptied.

Readings where the paper is silent (the library's planner follows them too):
  * A candidate that has already received a source is not itself moved
    later: the feasibility test counts only the source's own usage, so
    moving a destination would strand what was planned into it (the plan
    could exceed c_max).
  * Usage is counted in KV pages (integers), so ties are exact. Equal usage
    keeps the input order in the sort; among equally full destinations the
    first in visiting order wins.

Migration. Moving a trajectory between rollouts that share one GPU copies
each of its pages from the source pool to a free page of the destination
pool and rewrites its block-table row; the page contents are unchanged, so
attention over the moved trajectory gives the same result.
"""
from __future__ import annotations

from typing import List, Sequence, Tuple

import numpy as np


def candidates(used: Sequence[int], prev: Sequence[int], reqs: Sequence[int],
               c_max: int, b_max: int) -> List[int]:
    """Step 1: rollouts in their ramp-down phase with room under b_max."""
    return [r for r in range(len(used))
            if used[r] < min(c_max, prev[r]) and reqs[r] < b_max]


def best_fit_consolidation(used: Sequence[int], prev: Sequence[int],
                           reqs: Sequence[int], c_max: int,
                           b_max: int) -> List[Tuple[int, int]]:
    """The (source, destination) pairs of the consolidation plan, in the
    order they are decided."""
    s_list = candidates(used, prev, reqs, c_max, b_max)
    s_list = sorted(s_list, key=lambda r: used[r])          # stable
    plan: List[Tuple[int, int]] = []
    emptied = set()
    received = set()

    def load(d):
        extra_c = sum(used[s] for s, dd in plan if dd == d)
        extra_n = sum(reqs[s] for s, dd in plan if dd == d)
        return used[d] + extra_c, reqs[d] + extra_n

    def can_fit(d, s):
        c, n = load(d)
        return c + used[s] <= c_max and n + reqs[s] <= b_max

    for s in s_list:
        if s in emptied or s in received:
            continue
        dests = [d for d in s_list
                 if d not in emptied and d != s and can_fit(d, s)]
        if not dests:
            continue
        best = max(load(d)[0] for d in dests)
        d_star = next(d for d in dests if load(d)[0] == best)
        plan.append((s, d_star))
        emptied.add(s)
        received.add(d_star)
    return plan


def migrate_pages(src_pool: np.ndarray, dst_pool: np.ndarray,
                  pairs: np.ndarray) -> np.ndarray:
    """Copy page src_pool[s] to dst_pool[d] for every (s, d) row of pairs;
    returns the updated copy of dst_pool."""
    out = np.array(dst_pool)
    for s, d in np.asarray(pairs).reshape(-1, 2):
        out[d] = src_pool[s]
    return out
