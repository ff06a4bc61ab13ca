"""Caller-given costs placed at the edges of the key types (reading R10).

Costs are M - x with x in [0, 4) drawn from a seed: dense ties (the lowest-index
tie-break), and every sum the recurrence forms close to its bound, so that the
keys the fill compares sit close to the bound that chooses the key type.  The
key type of a plan grows with M, so the largest M of a key type is found by
bisection on the host (no device work)."""
import numpy as np

from workloads import random_costs


def near_costs(seed, K, shapes, M):
    layer, edge = random_costs(seed, K, shapes, hi=4)
    M = np.uint64(M)
    return [M - a for a in layer], [M - e for e in edge]


def plan_key_type(P, pg, seed, K, shapes, M):
    """Key type the library plans for the costs at M (-1: OVERFLOW)."""
    try:
        pg.override_costs(*near_costs(seed, K, shapes, M))
    except P.PaseError as e:
        assert e.status == P.OVERFLOW, e
        return -1
    return pg.vertex_info(0)["key_type"]


def largest_m(P, pg, seed, K, shapes, accept, lo=4, hi=1 << 63):
    """Largest M in [lo, hi) whose planned key type satisfies accept(kt);
    accept(kt at lo) must hold and accept must flip once as M grows."""
    assert accept(plan_key_type(P, pg, seed, K, shapes, lo))
    while hi - lo > 1:
        mid = (lo + hi) // 2
        if accept(plan_key_type(P, pg, seed, K, shapes, mid)):
            lo = mid
        else:
            hi = mid
    return lo


def key_top(pg, K):
    """Largest key bound of the plan: max over vertices of (key_bound + 1) * 2^bits."""
    top = 0
    for v in range(len(K)):
        info = pg.vertex_info(v)
        bits = max(0, (int(K[v]) - 1).bit_length())
        top = max(top, (int(info["key_bound"]) + 1) << bits)
    return top
