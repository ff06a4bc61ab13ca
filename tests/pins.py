"""Independent checks that pin the CPU oracle to the mathematics of the paper.

Nothing here reuses the oracle's code: each function recomputes a quantity
from its definition with a different method (exhaustive enumeration, the
Viterbi min-plus recursion, breadth-first search), using only the oracle's
cost tables as inputs (the cost model itself is pinned by hand-derived
values in the tests).
"""
from __future__ import annotations

import itertools
from collections import deque

import numpy as np


def total_cost(strategy, L, R, src, dst) -> int:
    """F(G, phi) of eq. (1) from cost tables: sum of layer costs plus the
    (already r-weighted) transfer cost of every edge."""
    tot = 0
    for v, c in enumerate(strategy):
        tot += int(L[v][c])
    for e in range(len(src)):
        tot += int(R[e][strategy[src[e]], strategy[dst[e]]])
    return tot


def brute_force(L, R, src, dst, limit: int = 2_000_000):
    """min over all strategies of F (Theorem 1's right-hand side) and the
    boolean array of optimal strategies (axes = vertex ids).  Vectorised with
    broadcasting; the search space must stay below `limit` strategies."""
    n = len(L)
    Ks = [len(x) for x in L]
    if int(np.prod(Ks, dtype=np.float64)) > limit:
        raise ValueError("search space too large for brute force")
    F = np.zeros(Ks, dtype=np.uint64)
    for v in range(n):
        shape = [1] * n
        shape[v] = Ks[v]
        F = F + np.asarray(L[v], np.uint64).reshape(shape)
    for e in range(len(src)):
        u, v = src[e], dst[e]
        M = np.asarray(R[e], np.uint64)
        shape = [1] * n
        shape[u] = Ks[u]
        shape[v] = Ks[v]
        # axes u < v keep M as is; otherwise transpose so that axis order matches
        F = F + (M if u < v else M.T).reshape(shape)
    m = F.min()
    return int(m), F == m


def viterbi_chain(L, R, forward):
    """Min-plus Viterbi on a path graph v0 - v1 - ... in that order.

    forward[k] says whether edge k is stored (v_k -> v_{k+1}) (True) or
    (v_{k+1} -> v_k) (False).  delta_k(c) = L_k[c] + min_c' (delta_{k-1}(c') +
    R_k(c', c)); back-pointers keep the lowest index on ties.  Returns
    (min cost, strategy)."""
    n = len(L)
    delta = np.asarray(L[0], dtype=object)
    back = []
    for k in range(1, n):
        M = np.asarray(R[k - 1], dtype=object)
        if not forward[k - 1]:
            M = M.T
        cand = delta[:, None] + M             # [c_{k-1}, c_k]
        best_prev = [_argmin_first(cand[:, c]) for c in range(cand.shape[1])]
        back.append(best_prev)
        delta = np.array([cand[best_prev[c], c] for c in range(cand.shape[1])], dtype=object) + \
            np.asarray(L[k], dtype=object)
    last = _argmin_first(delta)
    strat = [0] * n
    strat[n - 1] = last
    for k in range(n - 1, 0, -1):
        strat[k - 1] = back[k - 1][strat[k]]
    return int(delta[last]), strat


def _argmin_first(arr) -> int:
    best, arg = None, 0
    for i, x in enumerate(arr):
        if best is None or x < best:
            best, arg = x, i
    return arg


def viterbi_table_strategy(L, R, forward):
    """Same chain, but backtracked the way a table indexed by the *next*
    vertex's configuration is (the order FindBestStrategy uses on a path):
    c_{n-1} = lowest argmin of delta_{n-1}; c_k = lowest argmin over c of
    delta_k(c) + R_k(c, c_{k+1})."""
    n = len(L)
    deltas = [np.asarray(L[0], dtype=object)]
    for k in range(1, n):
        M = np.asarray(R[k - 1], dtype=object)
        if not forward[k - 1]:
            M = M.T
        cand = deltas[-1][:, None] + M
        deltas.append(np.array([min(cand[:, c]) for c in range(cand.shape[1])], dtype=object)
                      + np.asarray(L[k], dtype=object))
    strat = [0] * n
    strat[n - 1] = _argmin_first(deltas[n - 1])
    for k in range(n - 2, -1, -1):
        M = np.asarray(R[k], dtype=object)
        if not forward[k]:
            M = M.T
        strat[k] = _argmin_first(deltas[k] + M[:, strat[k + 1]])
    return int(min(deltas[n - 1])), strat


def neighbours(nv, src, dst):
    nb = [set() for _ in range(nv)]
    for u, v in zip(src, dst):
        nb[u].add(v)
        nb[v].add(u)
    return nb


def connected_set(nb, seq, i):
    """X(i): vertices of positions <= i reachable from seq[i] through such vertices (BFS)."""
    pos = {v: k for k, v in enumerate(seq)}
    start = seq[i]
    seen = {start}
    q = deque([start])
    while q:
        x = q.popleft()
        for y in nb[x]:
            if pos[y] <= i and y not in seen:
                seen.add(y)
                q.append(y)
    return seen


def dependent_set(nb, seq, i):
    """D(i) = N(X(i)) intersected with the vertices after position i."""
    pos = {v: k for k, v in enumerate(seq)}
    X = connected_set(nb, seq, i)
    return sorted({y for x in X for y in nb[x] if pos[y] > i})


def connected_subsets(nb, seq, i):
    """S(i): components of X(i) - {v_i} (as sorted vertex lists)."""
    pos = {v: k for k, v in enumerate(seq)}
    X = connected_set(nb, seq, i) - {seq[i]}
    comps, seen = [], set()
    for s in sorted(X):
        if s in seen:
            continue
        comp, q = {s}, deque([s])
        seen.add(s)
        while q:
            x = q.popleft()
            for y in nb[x]:
                if y in X and y not in seen and pos[y] < i:
                    seen.add(y)
                    comp.add(y)
                    q.append(y)
        comps.append(sorted(comp))
    return comps


def bfs_dependent_set(nb, seq, i):
    """D_B(i) of the breadth-first recurrence (2): N(V_{<=i}) after position i."""
    pos = {v: k for k, v in enumerate(seq)}
    return sorted({y for x in seq[:i + 1] for y in nb[x] if pos[y] > i})


def conditioned_table(L, R, src, dst, seq, i, Ks, limit: int = 2_000_000):
    """Every entry of DP table i by exhaustive search: for each assignment phi
    of D(i), T_i[phi] = min over assignments of X(i) of the sum over v in X(i)
    of the node function (layer cost of v plus transfer cost of every edge
    joining v and a later vertex), and A_i[phi] = the lowest configuration of
    seq[i] attaining it.  Returns (D(i), T, A) in canonical order (D(i)
    ascending, first digit slowest)."""
    nv = len(L)
    nb = neighbours(nv, src, dst)
    pos = {v: k for k, v in enumerate(seq)}
    X = sorted(connected_set(nb, seq, i))
    D = dependent_set(nb, seq, i)
    vi = seq[i]
    # each edge is charged to its earlier endpoint; keep those charged inside X(i)
    later_edges = [e for e in range(len(src))
                   if (src[e] in X and pos[dst[e]] > pos[src[e]])
                   or (dst[e] in X and pos[src[e]] > pos[dst[e]])]
    space = 1
    for v in X + D:
        space *= Ks[v]
    if space > limit:
        raise ValueError("conditioned search too large")
    NT = int(np.prod([Ks[w] for w in D])) if D else 1
    T = [None] * NT
    A = [None] * NT
    for phi_idx, phi in enumerate(itertools.product(*[range(Ks[w]) for w in D])):
        cfg = dict(zip(D, phi))
        best, best_c = None, None
        for xs in itertools.product(*[range(Ks[v]) for v in X]):
            cfg.update(zip(X, xs))
            cost = sum(int(L[v][cfg[v]]) for v in X)
            for e in later_edges:
                cost += int(R[e][cfg[src[e]], cfg[dst[e]]])
            c = cfg[vi]
            if best is None or cost < best or (cost == best and c < best_c):
                best, best_c = cost, c
        T[phi_idx], A[phi_idx] = best, best_c
    return D, T, A


def conditioned_qmax(L, R, src, dst, seq, i, Ks, limit: int = 2_000_000) -> int:
    """The largest value the DP minimises over at position i: max over
    assignments phi of D(i) and configurations c of seq[i] of the min over
    the rest of X(i) of the same sum as in conditioned_table (exhaustive)."""
    nv = len(L)
    nb = neighbours(nv, src, dst)
    pos = {v: k for k, v in enumerate(seq)}
    X = sorted(connected_set(nb, seq, i))
    D = dependent_set(nb, seq, i)
    vi = seq[i]
    later_edges = [e for e in range(len(src))
                   if (src[e] in X and pos[dst[e]] > pos[src[e]])
                   or (dst[e] in X and pos[src[e]] > pos[dst[e]])]
    space = 1
    for v in X + D:
        space *= Ks[v]
    if space > limit:
        raise ValueError("conditioned search too large")
    best = {}
    for phi in itertools.product(*[range(Ks[w]) for w in D]):
        cfg = dict(zip(D, phi))
        for xs in itertools.product(*[range(Ks[v]) for v in X]):
            cfg.update(zip(X, xs))
            cost = sum(int(L[v][cfg[v]]) for v in X)
            for e in later_edges:
                cost += int(R[e][cfg[src[e]], cfg[dst[e]]])
            key = (phi, cfg[vi])
            if key not in best or cost < best[key]:
                best[key] = cost
    return max(best.values())


def volume_transfer_elements(m, src_dim, dst_dim, s_src, s_dst, r) -> int:
    """r * t_x of the volume model by enumerating tensor elements: tensor
    dims of sizes m (each divisible by the splits that cut it), element index
    i of dim t lies in part i * s // m_t on a side whose loop dim (mapped by
    src_dim / dst_dim, -1 = unmapped, s = 1) is split s ways; device d of a
    configuration is the mixed-radix grid point spelled by d (loop dim 0
    slowest), devices past the product take no part.  Forward = the largest
    count of elements a consumer device needs but does not hold, backward the
    same with the roles swapped; r * (forward + backward)."""
    def coords(d, splits):
        out = [0] * len(splits)
        for k in range(len(splits) - 1, -1, -1):
            out[k] = d % splits[k]
            d //= splits[k]
        return out

    Pu, Pv = int(np.prod(s_src)), int(np.prod(s_dst))
    elems = list(itertools.product(*[range(x) for x in m]))

    def part(side_dims, splits, xs):
        keep = set()
        for el in elems:
            ok = True
            for t, i in enumerate(el):
                k = side_dims[t]
                s = splits[k] if k >= 0 else 1
                x = xs[k] if k >= 0 else 0
                if i * s // m[t] != x:
                    ok = False
                    break
            if ok:
                keep.add(el)
        return keep

    fwd = bwd = 0
    for d in range(max(Pu, Pv)):
        A_u = part(src_dim, s_src, coords(d, s_src)) if d < Pu else set()
        A_v = part(dst_dim, s_dst, coords(d, s_dst)) if d < Pv else set()
        fwd = max(fwd, len(A_v - A_u))
        bwd = max(bwd, len(A_u - A_v))
    return r * (fwd + bwd)


def assigned_transfer_elements(m, src_dim, dst_dim, s_src, s_dst, part_src, part_dst, r):
    """Locality and r * t_x of one edge under explicit device maps, by
    enumerating tensor elements (dims of sizes m, each divisible by the splits
    that cut it): part_src[d] / part_dst[d] is the part (mixed-radix grid
    point, loop dim 0 slowest) each end holds on device d, -1 for none.
    Locality = sum over devices of the elements both ends hold there; forward
    = the largest count a consumer device needs but does not hold, backward
    the same with the roles swapped."""
    def coords(g, splits):
        out = [0] * len(splits)
        for k in range(len(splits) - 1, -1, -1):
            out[k] = g % splits[k]
            g //= splits[k]
        return out

    elems = list(itertools.product(*[range(x) for x in m]))

    def part(side_dims, splits, g):
        if g < 0:
            return set()
        xs = coords(g, splits)
        return {el for el in elems
                if all(i * (splits[side_dims[t]] if side_dims[t] >= 0 else 1) // m[t]
                       == (xs[side_dims[t]] if side_dims[t] >= 0 else 0) for t, i in enumerate(el))}

    loc = fwd = bwd = 0
    for d in range(len(part_src)):
        A_u, A_v = part(src_dim, s_src, part_src[d]), part(dst_dim, s_dst, part_dst[d])
        loc += len(A_u & A_v)
        fwd = max(fwd, len(A_v - A_u))
        bwd = max(bwd, len(A_u - A_v))
    return loc, r * (fwd + bwd)


def splitmix64_mix(z: int) -> int:
    """SplitMix64 output function (Steele, Lea and Flood, 2014)."""
    m = (1 << 64) - 1
    z &= m
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & m
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & m
    return z ^ (z >> 31)


def fingerprint(T, A):
    m = (1 << 64) - 1
    fa = fb = 0
    for idx, (t, a) in enumerate(zip(T, A)):
        h = splitmix64_mix(idx)
        fa = (fa + splitmix64_mix(h ^ int(t))) & m
        fb = (fb + splitmix64_mix(h ^ int(a))) & m
    return fa, fb
