"""Pins of the CPU oracle (no GPU).

The oracle is the reference every GPU result is compared with, so it is first
checked against things it does not compute itself: hand-derived values of the
integer cost model, closed forms (binomial configuration counts, the FC-chain
optimum), exhaustive search over all strategies (Theorem 1), exhaustive search
of every DP table entry, the Viterbi recursion on path graphs, the definition
of the dependent set (Theorem 2), and order independence of the minimum.
"""
import itertools
import math

import numpy as np
import pytest

import pins
from workloads import chain_graph, fc_chain, random_costs, random_graph, workload

pytestmark = pytest.mark.usefixtures("oracle_lib")


def _solve(g, p=None, rule=0, costs=None, order=None, lib=None):
    from oracle.oracle import Oracle
    o = Oracle(g, lib)
    K = o.configs(p or g["p"])
    if costs is not None:
        o.set_costs(*costs)
    o.solve(rule=rule, order=order)
    return o, K


def _tables(o, g):
    L = [o.layer_costs(v) for v in range(len(g["vertices"]))]
    R = [o.edge_costs(e) for e in range(len(g["edges"]))]
    src = [e["src"] for e in g["edges"]]
    dst = [e["dst"] for e in g["edges"]]
    return L, R, src, dst


# ------------------------------------------------------------------ configurations
@pytest.mark.parametrize("d", [1, 2, 3, 4, 5])
@pytest.mark.parametrize("p", [1, 2, 4, 8, 16, 64])
def test_config_count_and_order(d, p):
    """|C(v)| = C(L+d, d) for power-of-two splits with product <= p = 2^L
    (stars and bars); order is lexicographic in the exponent tuple, dim 0
    slowest; every tuple has product <= p and all are distinct."""
    from oracle.oracle import Oracle
    g = {"name": "one", "p": p, "comm_weight": 8,
         "vertices": [{"name": "v", "dims": [7] * d, "dim_names": ["x"] * d, "reduce": [],
                       "flops_per_point": 1}], "edges": []}
    o = Oracle(g)
    K = o.configs(p)
    L = int(math.log2(p))
    assert int(K[0]) == math.comb(L + d, d)
    ex = [tuple(int(x) for x in row) for row in o.exponents(0)]
    assert ex == sorted(ex)
    assert len(set(ex)) == len(ex)
    assert all(sum(t) <= L for t in ex)
    # every admissible tuple is present
    assert set(ex) == {t for t in itertools.product(range(L + 1), repeat=d) if sum(t) <= L}


def test_workload_config_counts():
    """10 (W0, p=4, 3 dims), 56 (W1, p=8, 5 dims), 126/70/35 (W2, p=16),
    56 (W3, p=32, 3 dims), 462/210/84 (W4, p=64)."""
    from oracle.oracle import Oracle
    expect = {"w0_fc_chain": {10}, "w1_residual_cnn": {56}, "w2_inception": {126, 70, 35},
              "w3_lstm_grid": {56}, "w4_transformer": {462, 210, 84}}
    for name, ks in expect.items():
        g = workload(name)
        o = Oracle(g)
        assert set(int(k) for k in o.configs(g["p"])) == ks


def test_p_must_be_power_of_two():
    from oracle.oracle import Oracle, OracleError
    o = Oracle(fc_chain())
    with pytest.raises(OracleError):
        o.configs(6)



# ------------------------------------------------------------------ all-integer configurations
def _one_vertex(d, p, size=7):
    return {"name": "one", "p": p, "comm_weight": 8,
            "vertices": [{"name": "v", "dims": [size] * d, "dim_names": ["x"] * d, "reduce": [],
                          "flops_per_point": 1}], "edges": []}


def _divisor_power_count(p, d):
    """Number of d-tuples of positive integers with product <= p, by the
    recurrence N_d(p) = sum_{s=1..p} N_{d-1}(floor(p/s)), N_0 = 1 (the first
    factor s leaves floor(p/s) for the product of the others)."""
    if d == 0:
        return 1
    return sum(_divisor_power_count(p // s, d - 1) for s in range(1, p + 1))


@pytest.mark.parametrize("d", [1, 2, 3, 4])
@pytest.mark.parametrize("p", [1, 2, 3, 5, 6, 12])
def test_all_integer_config_count_and_order(d, p):
    """C(v) with every positive-integer split: exactly the tuples with product
    <= p (exhaustive over [1, p]^d), each once, lexicographic with dim 0
    slowest; the count agrees with the divisor-sum recurrence (p = 12, d = 2:
    sum of the divisor counts of 1..12 = 35)."""
    from oracle.oracle import Oracle
    o = Oracle(_one_vertex(d, p))
    K = o.configs(p, all_integers=True)
    sp = [tuple(int(x) for x in row) for row in o.splits(0)]
    brute = [t for t in itertools.product(range(1, p + 1), repeat=d) if math.prod(t) <= p]
    assert sp == brute
    assert int(K[0]) == len(brute) == _divisor_power_count(p, d)
    if (p, d) == (12, 2):
        assert int(K[0]) == 35


def test_all_integer_contains_the_power_of_two_set():
    """At p = 2^L the power-of-two configurations are the all-integer ones whose
    factors are all powers of two, in the same relative order, with the same
    layer costs."""
    from oracle.oracle import Oracle
    g = fc_chain(p=8)
    a, b = Oracle(g), Oracle(g)
    a.configs(8)
    b.configs(8, all_integers=True)
    sa = [tuple(int(x) for x in r) for r in a.splits(0)]
    sb = [tuple(int(x) for x in r) for r in b.splits(0)]
    pw = [t for t in sb if all(x & (x - 1) == 0 for x in t)]
    assert sa == pw
    La, Lb = a.layer_costs(0), b.layer_costs(0)
    for i, t in enumerate(sa):
        assert int(La[i]) == int(Lb[sb.index(t)])


def test_all_integer_p_limits():
    """p = 1 leaves the single unsplit configuration; p < 1 is rejected; a
    configuration count above the uint16 argmin range is rejected."""
    from oracle.oracle import Oracle, OracleError
    o = Oracle(_one_vertex(3, 1))
    assert o.configs(1, all_integers=True).tolist() == [1]
    assert o.splits(0).tolist() == [[1, 1, 1]]
    with pytest.raises(OracleError):
        o.configs(0, all_integers=True)
    with pytest.raises(OracleError):
        Oracle(_one_vertex(4, 1)).configs(1000, all_integers=True)   # N_4(1000) > 65535


def test_layer_cost_non_power_of_two_hand_values():
    """FC (64, 256, 256) = 8 388 608 FLOPs, contraction over `in`, r = 8, p = 6:
    (3,1,1): ceil(8388608/3) = 2 796 203;  (1,1,3): 2 796 203 + 8*2*16384 = 3 058 347;
    (2,3,1): ceil(8388608/6) = 1 398 102;  (1,2,3): 1 398 102 + 8*2*8192 = 1 529 174;
    (1,5,1): ceil(8388608/5) = 1 677 722.
    Ragged dims (3, 5), contraction over dim 1, 45 FLOPs, p = 6:
    (3,2): 8 + 8*1*1 = 16;  (1,5): 9 + 8*4*3 = 105;  (5,1): 9;  (2,3): 8 + 8*2*2 = 40."""
    from oracle.oracle import Oracle
    o = Oracle(fc_chain(p=6))
    o.configs(6, all_integers=True)
    sp = [tuple(int(x) for x in r) for r in o.splits(0)]
    L = o.layer_costs(0)
    want = {(3, 1, 1): 2_796_203, (1, 1, 3): 3_058_347, (2, 3, 1): 1_398_102,
            (1, 2, 3): 1_529_174, (1, 5, 1): 1_677_722}
    for t, v in want.items():
        assert int(L[sp.index(t)]) == v, t
    g = {"name": "r", "p": 6, "comm_weight": 8,
         "vertices": [{"name": "v", "dims": [3, 5], "dim_names": ["a", "b"], "reduce": [1],
                       "flops_per_point": 3}], "edges": []}
    o = Oracle(g)
    o.configs(6, all_integers=True)
    sp = [tuple(int(x) for x in r) for r in o.splits(0)]
    L = o.layer_costs(0)
    for t, v in {(3, 2): 16, (1, 5): 105, (5, 1): 9, (2, 3): 40}.items():
        assert int(L[sp.index(t)]) == v, t


def test_transfer_cost_non_power_of_two_hand_values():
    """Edge fc0 -> fc1 of the FC chain, (b, feat) = 64 x 256 = 16 384 words, r = 8, p = 6:
    (3,1,1) vs (1,1,3): b 3 != 1 -> 8 * ceil(16384/3) = 43 696;
    (1,1,1) vs (5,1,1): 8 * ceil(16384/5) = 26 216;
    (2,3,1) vs (2,1,3): b 2 = 2 and feat out 3 = in 3 -> 0."""
    from oracle.oracle import Oracle
    o = Oracle(fc_chain(p=6))
    o.configs(6, all_integers=True)
    sp = [tuple(int(x) for x in r) for r in o.splits(0)]
    R = o.edge_costs(0)
    i = sp.index
    assert int(R[i((3, 1, 1)), i((1, 1, 3))]) == 43_696
    assert int(R[i((1, 1, 1)), i((5, 1, 1))]) == 26_216
    assert int(R[i((2, 3, 1)), i((2, 1, 3))]) == 0


@pytest.mark.parametrize("seed", range(8))
def test_theorem1_all_integer_configs(seed):
    """Theorem 1 with every positive-integer split (p = 3, 5, 6)."""
    p = (3, 5, 6)[seed % 3]
    g = random_graph(seed + 40, n=3 + seed % 3, p=p, max_dims=2, extra_edges=seed % 3)
    from oracle.oracle import Oracle
    o = Oracle(g)
    K = o.configs(p, all_integers=True)
    o.solve()
    L, R, src, dst = _tables(o, g)
    mc, strat = o.result()
    bf_min, optimal = pins.brute_force(L, R, src, dst)
    assert mc == bf_min
    assert pins.total_cost(strat, L, R, src, dst) == mc and bool(optimal[tuple(strat)])
    seq = o.sequence()
    for i in range(len(seq)):
        D, T, A = pins.conditioned_table(L, R, src, dst, seq, i, [int(k) for k in K])
        To, Ao = o.table(i)
        assert To.tolist() == T and Ao.tolist() == A, (i, seq)


@pytest.mark.parametrize("seed", range(4))
def test_viterbi_all_integer_configs(seed):
    """Path graphs with every positive-integer split at p = 6 or 12: the DP is
    the Viterbi recursion (same minimum, same lowest-index strategy)."""
    p = 6 if seed % 2 else 12
    g = chain_graph(seed + 30, n=4 + seed, p=p, max_dims=2)
    from oracle.oracle import Oracle
    o = Oracle(g)
    o.configs(p, all_integers=True)
    o.solve()
    assert o.sequence() == list(range(len(g["vertices"])))
    L, R, src, dst = _tables(o, g)
    forward = [e["src"] < e["dst"] for e in g["edges"]]
    mc, strat = o.result()
    vmin, _ = pins.viterbi_chain(L, R, forward)
    tmin, tstrat = pins.viterbi_table_strategy(L, R, forward)
    assert mc == vmin == tmin
    assert strat == tstrat

# ------------------------------------------------------------------ cost model (hand values)
def test_layer_cost_fc_hand_values():
    """FC (64, 256, 256), contraction over `in`, r = 8, p = 4.
    (4,1,1): 2*64*256*256/4 = 2 097 152 FLOPs, no partial sums.
    (1,1,4): same compute + 8 * (4-1) * 64*256 = 2 097 152 + 393 216.
    (1,1,1): 8 388 608.  (2,2,1): 2 097 152.  (1,2,2): 2 097 152 + 8*(2-1)*64*128."""
    from oracle.oracle import Oracle
    o = Oracle(fc_chain())
    o.configs(4)
    ex = [tuple(int(x) for x in r) for r in o.exponents(0)]
    L = o.layer_costs(0)
    want = {(2, 0, 0): 2_097_152, (0, 0, 2): 2_490_368, (0, 0, 0): 8_388_608,
            (1, 1, 0): 2_097_152, (0, 1, 1): 2_097_152 + 8 * 64 * 128}
    for t, v in want.items():
        assert int(L[ex.index(t)]) == v, t
    assert ex.index((2, 0, 0)) == 9


def test_layer_cost_ragged_hand_values():
    """dims (3, 5), contraction over dim 1, 3 FLOPs per point (45 total), r = 8, p = 4:
    (2,2): ceil(45/4)=12 + 8*(2-1)*ceil(3/2)=16 -> 28;  (1,4): 12 + 8*3*3 = 84;
    (4,1): 12;  (1,1): 45;  (2,1): ceil(45/2)=23;  (1,2): 23 + 8*1*3 = 47."""
    from oracle.oracle import Oracle
    g = {"name": "r", "p": 4, "comm_weight": 8,
         "vertices": [{"name": "v", "dims": [3, 5], "dim_names": ["a", "b"], "reduce": [1],
                       "flops_per_point": 3}], "edges": []}
    o = Oracle(g)
    o.configs(4)
    ex = [tuple(int(x) for x in r) for r in o.exponents(0)]
    L = o.layer_costs(0)
    want = {(1, 1): 28, (0, 2): 84, (2, 0): 12, (0, 0): 45, (1, 0): 23, (0, 1): 47}
    for t, v in want.items():
        assert int(L[ex.index(t)]) == v, t


def test_transfer_cost_hand_values():
    """Edge fc0 -> fc1 carries (b, feat) from (b, out) of fc0 to (b, in) of fc1.
    Equal splits on both tensor dims -> 0; otherwise 8 * ceil(16384 / max(P_u, P_v))."""
    from oracle.oracle import Oracle
    o = Oracle(fc_chain())
    o.configs(4)
    ex = [tuple(int(x) for x in r) for r in o.exponents(0)]
    R = o.edge_costs(0)
    i = ex.index
    assert int(R[i((2, 0, 0)), i((2, 0, 0))]) == 0
    assert int(R[i((2, 0, 0)), i((0, 0, 2))]) == 8 * 4096
    assert int(R[i((0, 0, 0)), i((0, 0, 0))]) == 0
    assert int(R[i((1, 1, 0)), i((1, 0, 1))]) == 0          # b:2=2, feat: out 2 = in 2
    assert int(R[i((1, 1, 0)), i((1, 1, 0))]) == 8 * 4096   # feat: out 2 vs in 1
    assert int(R[i((0, 0, 0)), i((1, 0, 0))]) == 8 * 8192   # max(P) = 2
    # the unsplit `out` dim of fc1 plays no role: (2,1,1) vs (2,2,1) on fc1 side
    assert int(R[i((1, 0, 0)), i((1, 1, 0))]) == 0


def test_transfer_cost_unsplit_tensor_dim():
    """A tensor dim mapped to -1 on one side counts as split factor 1 there."""
    from oracle.oracle import Oracle
    g = {"name": "u", "p": 4, "comm_weight": 2,
         "vertices": [{"name": "a", "dims": [8, 8], "dim_names": ["x", "y"], "reduce": [],
                       "flops_per_point": 1},
                      {"name": "b", "dims": [8], "dim_names": ["x"], "reduce": [],
                       "flops_per_point": 1}],
         "edges": [{"src": 0, "dst": 1, "src_dim": [0, 1], "dst_dim": [0, -1], "elems": 10}]}
    o = Oracle(g)
    o.configs(4)
    exa = [tuple(int(x) for x in r) for r in o.exponents(0)]
    exb = [tuple(int(x) for x in r) for r in o.exponents(1)]
    R = o.edge_costs(0)
    assert int(R[exa.index((1, 0)), exb.index((1,))]) == 0
    assert int(R[exa.index((1, 1)), exb.index((1,))]) == 2 * math.ceil(10 / 4)
    assert int(R[exa.index((0, 0)), exb.index((2,))]) == 2 * math.ceil(10 / 4)


def test_cost_overflow_is_reported():
    from oracle.oracle import Oracle, OracleError
    g = {"name": "big", "p": 2, "comm_weight": 8,
         "vertices": [{"name": "v", "dims": [2**40, 2**30], "dim_names": ["a", "b"], "reduce": [],
                       "flops_per_point": 1}], "edges": []}
    o = Oracle(g)
    with pytest.raises(OracleError):
        o.configs(2)


# ------------------------------------------------------------------ GenerateSeq
def test_generate_seq_fc_chain_both_rules():
    """Hand trace of Fig. 3 on the path 0-1-2-3: excluding self gives [0,1,2,3];
    the printed update (v may count itself) gives [0,3,1,2]."""
    g = fc_chain()
    o, _ = _solve(g, rule=0)
    assert o.sequence() == [0, 1, 2, 3]
    assert [o.dependent_set(i) for i in range(4)] == [[1], [2], [3], []]
    o, _ = _solve(g, rule=1)
    assert o.sequence() == [0, 3, 1, 2]
    assert [o.dependent_set(i) for i in range(4)] == [[1], [2], [2], []]


@pytest.mark.parametrize("seed", range(12))
@pytest.mark.parametrize("rule", [0, 1])
def test_theorem2_dependent_sets(seed, rule):
    """Theorem 2: the d-set GenerateSeq records equals N(X(i)) after position i."""
    g = random_graph(seed, n=5 + seed % 7, extra_edges=seed % 5, p=2)
    o, _ = _solve(g, rule=rule)
    seq = o.sequence()
    nb = pins.neighbours(len(g["vertices"]), [e["src"] for e in g["edges"]],
                         [e["dst"] for e in g["edges"]])
    assert sorted(seq) == list(range(len(seq)))
    for i in range(len(seq)):
        assert o.dependent_set(i) == pins.dependent_set(nb, seq, i)
    assert o.dependent_set(len(seq) - 1) == []


def test_workload_dependent_set_histograms():
    """Structure of the large workloads under the default rule."""
    from oracle.oracle import Oracle
    for name, hist in [("w1_residual_cnn", {0: 1, 1: 8, 2: 7}),
                       ("w4_transformer", {0: 1, 1: 17, 2: 102, 3: 16})]:
        g = workload(name)
        o = Oracle(g)
        o.configs(g["p"])
        o.solve(max_cells=1)
        h = {}
        for i in range(len(g["vertices"])):
            k = len(o.dependent_set(i))
            h[k] = h.get(k, 0) + 1
        assert h == hist


# ------------------------------------------------------------------ dynamic program
def test_fc_chain_closed_form():
    """W0: every 4-way config costs 2 097 152; zero communication needs s_in = 1,
    zero redistribution needs equal batch splits and s_out = 1 upstream, so the
    unique optimum is (4,1,1) everywhere: 4 * 2 097 152 = 8 388 608."""
    o, _ = _solve(fc_chain())
    assert o.result() == (8_388_608, [9, 9, 9, 9])
    assert o.cells() == 310


def _check_against_brute_force(g, costs=None, rule=0):
    o, K = _solve(g, costs=costs, rule=rule)
    L, R, src, dst = _tables(o, g)
    mc, strat = o.result()
    bf_min, optimal = pins.brute_force(L, R, src, dst)
    assert mc == bf_min                                   # Theorem 1
    assert pins.total_cost(strat, L, R, src, dst) == mc   # recovered strategy costs the minimum
    assert bool(optimal[tuple(strat)])
    return o, K, L, R, src, dst


@pytest.mark.parametrize("seed", range(16))
def test_theorem1_model_costs(seed):
    g = random_graph(seed, n=3 + seed % 4, p=4 if seed % 2 else 2, max_dims=2,
                     extra_edges=seed % 3)
    _check_against_brute_force(g)


@pytest.mark.parametrize("seed", range(16))
@pytest.mark.parametrize("rule", [0, 1])
def test_every_table_entry_random_ties(seed, rule):
    """Random integer costs in [0, 4) make ties dense; every entry of every
    table and its argmin (lowest configuration index among the optimal ones)
    must equal an exhaustive search conditioned on D(i)."""
    g = random_graph(seed + 100, n=3 + seed % 4, p=4, max_dims=2, extra_edges=1 + seed % 3)
    from oracle.oracle import Oracle
    o0 = Oracle(g)
    K = o0.configs(4)
    costs = random_costs(seed, K, [(K[e["src"]], K[e["dst"]]) for e in g["edges"]], hi=4)
    o, K, L, R, src, dst = _check_against_brute_force(g, costs=costs, rule=rule)
    seq = o.sequence()
    for i in range(len(seq)):
        D, T, A = pins.conditioned_table(L, R, src, dst, seq, i, [int(k) for k in K])
        assert o.dependent_set(i) == D
        To, Ao = o.table(i)
        assert To.tolist() == T, (i, seq)
        assert Ao.tolist() == A, (i, seq)
        assert o.fingerprint(i) == pins.fingerprint(T, A)


@pytest.mark.parametrize("seed", range(10))
def test_viterbi_on_chains(seed):
    """On a path graph the sequence is the path and the DP is the Viterbi
    recursion: equal minimum and equal (lowest-index) strategy."""
    g = chain_graph(seed, n=4 + seed % 5, p=8, max_dims=3)
    from oracle.oracle import Oracle
    o0 = Oracle(g)
    K = o0.configs(8)
    for costs in (None, random_costs(seed, K, [(K[e["src"]], K[e["dst"]]) for e in g["edges"]], hi=3)):
        o, _ = _solve(g, costs=costs)
        assert o.sequence() == list(range(len(g["vertices"])))
        L, R, src, dst = _tables(o, g)
        forward = [e["src"] < e["dst"] for e in g["edges"]]
        mc, strat = o.result()
        vmin, _ = pins.viterbi_chain(L, R, forward)
        tmin, tstrat = pins.viterbi_table_strategy(L, R, forward)
        assert mc == vmin == tmin
        assert strat == tstrat


@pytest.mark.parametrize("seed", range(8))
def test_order_independence(seed):
    """Theorem 1 holds for any order: GenerateSeq (both rules), breadth-first
    and random orders give the same minimum, and each recovered strategy costs it."""
    g = random_graph(seed + 7, n=6, p=4, max_dims=2, extra_edges=3)
    from oracle.oracle import Oracle
    mins = set()
    nv = len(g["vertices"])
    nb = pins.neighbours(nv, [e["src"] for e in g["edges"]], [e["dst"] for e in g["edges"]])
    bfs = [0]
    for v in bfs:
        for u in sorted(nb[v]):
            if u not in bfs:
                bfs.append(u)
    rng = np.random.default_rng(seed)
    orders = [None, None, bfs, rng.permutation(nv).tolist(), rng.permutation(nv).tolist()]
    for k, order in enumerate(orders):
        o = Oracle(g)
        o.configs(4)
        o.solve(rule=1 if k == 1 else 0, order=order)
        L, R, src, dst = _tables(o, g)
        mc, strat = o.result()
        assert pins.total_cost(strat, L, R, src, dst) == mc
        if order is not None:
            seq = o.sequence()
            for i in range(nv):
                assert o.dependent_set(i) == pins.dependent_set(nb, seq, i)
        mins.add(mc)
    assert len(mins) == 1


def _fig2_graph():
    """A graph built to satisfy the facts stated for the toy example (the
    figure itself is not available): with the identity order v1..v9,
    X(5) = {v1,v2,v3,v5}, S(5) = {{v1,v2},{v3}}, D(5) = {v8}, and the
    breadth-first dependent set of position 5 is {v7,v8,v9}."""
    edges = [(1, 2), (2, 5), (3, 5), (3, 8), (5, 8), (4, 7), (4, 9), (6, 7), (6, 9), (8, 9)]
    vs = [{"name": f"v{k}", "dims": [4, 3], "dim_names": ["a", "b"], "reduce": [1],
           "flops_per_point": k} for k in range(1, 10)]
    es = [{"src": a - 1, "dst": b - 1, "src_dim": [0], "dst_dim": [0], "elems": 6 * a + b}
          for a, b in edges]
    return {"name": "fig2", "p": 2, "comm_weight": 8, "vertices": vs, "edges": es}


def test_fig2_facts():
    g = _fig2_graph()
    order = list(range(9))
    src = [e["src"] for e in g["edges"]]
    dst = [e["dst"] for e in g["edges"]]
    nb = pins.neighbours(9, src, dst)
    i5 = 4  # position of v5 (0-based)
    assert pins.connected_set(nb, order, i5) == {0, 1, 2, 4}
    assert pins.connected_subsets(nb, order, i5) == [[0, 1], [2]]
    assert pins.dependent_set(nb, order, i5) == [7]
    assert pins.bfs_dependent_set(nb, order, i5) == [6, 7, 8]
    from oracle.oracle import Oracle
    o = Oracle(g)
    K = o.configs(2)
    costs = random_costs(5, K, [(K[a], K[b]) for a, b in zip(src, dst)], hi=5)
    o.set_costs(*costs)
    o.solve(order=order)
    assert o.dependent_set(i5) == [7]
    L, R = costs
    D, T, A = pins.conditioned_table(L, R, src, dst, order, i5, [int(k) for k in K])
    To, Ao = o.table(i5)
    assert To.tolist() == T and Ao.tolist() == A
    mc, strat = o.result()
    assert mc == pins.brute_force(L, R, src, dst)[0]


def test_multi_edges_counted_per_edge():
    """Parallel edges each contribute their transfer cost (sum over E in eq. 1)."""
    g = random_graph(3, n=4, p=2, max_dims=2, extra_edges=4, multi_edges=True)
    pairs = [frozenset((e["src"], e["dst"])) for e in g["edges"]]
    assert len(pairs) != len(set(pairs))
    _check_against_brute_force(g)


def test_disconnected_graph_rejected():
    from oracle.oracle import Oracle, OracleError
    g = random_graph(1, n=3, p=2)
    g["vertices"].append({"name": "lonely", "dims": [2], "dim_names": ["a"], "reduce": [],
                          "flops_per_point": 1})
    o = Oracle(g)
    o.configs(2)
    with pytest.raises(OracleError):
        o.solve()




# ------------------------------------------------------------------ volume-intersection transfer cost
def test_volume_transfer_hand_values():
    """FC chain p = 4, edge fc0 -> fc1, tensor (b, feat) = 16 384 words, r = 8.
    (4,1,1) -> (4,1,1): device d holds and needs batch quarter d: 0.
    (1,1,1) -> (4,1,1): forward, devices 1..3 need a quarter the producer's
    single device does not give them (4096); backward, device 0 of the
    producer needs the whole gradient but holds a quarter of it on the consumer
    side (12 288): 8 * 16 384 = 131 072.
    (2,2,1) -> (2,1,2): device b*2+x holds feat half x (out) and needs feat half
    x (in): 0.  (1,2,2) -> (1,1,2): the producer's device d = 2*out + in holds
    feat half d // 2, the consumer's device d needs half d: device 1 misses a
    half forward, devices 1..3 a half backward: 8 * (8192 + 8192) = 131 072,
    where the split-match model charges nothing (both split feat 2 ways)."""
    from oracle.oracle import Oracle
    o = Oracle(fc_chain())
    o.configs(4, volume=True)
    sp = [tuple(int(x) for x in r) for r in o.splits(0)]
    R = o.edge_costs(0)
    i = sp.index
    assert int(R[i((4, 1, 1)), i((4, 1, 1))]) == 0
    assert int(R[i((1, 1, 1)), i((4, 1, 1))]) == 131_072
    assert int(R[i((2, 2, 1)), i((2, 1, 2))]) == 0
    assert int(R[i((1, 2, 2)), i((1, 1, 2))]) == 131_072
    o2 = Oracle(fc_chain())
    o2.configs(4)
    assert int(o2.edge_costs(0)[i((1, 2, 2)), i((1, 1, 2))]) == 0


@pytest.mark.parametrize("seed", range(10))
def test_volume_transfer_against_element_enumeration(seed):
    """Every entry of the volume model's edge matrix on a random two-vertex
    graph equals the count over individual tensor elements (sizes divisible by
    every split, random dim maps with unmapped dims on either side)."""
    from oracle.oracle import Oracle
    rng = np.random.default_rng(seed)
    p = (2, 4, 6)[seed % 3]
    all_int = p == 6
    du, dv = int(rng.integers(1, 4)), int(rng.integers(1, 4))
    rank = 1 if all_int else int(rng.integers(1, 3))
    size = 60 if all_int else 12          # divisible by every split factor <= p
    src_dim = [int(x) for x in rng.permutation(du)[:rank]] + [-1] * max(0, rank - du)
    dst_dim = [int(x) for x in rng.permutation(dv)[:rank]] + [-1] * max(0, rank - dv)
    src_dim, dst_dim = src_dim[:rank], dst_dim[:rank]
    if seed % 4 == 1 and rank > 1:
        src_dim[0] = -1
    m = [size] * rank
    g = {"name": "vol", "p": p, "comm_weight": 3,
         "vertices": [{"name": "u", "dims": [size] * du, "dim_names": ["x"] * du, "reduce": [],
                       "flops_per_point": 1},
                      {"name": "v", "dims": [size] * dv, "dim_names": ["x"] * dv, "reduce": [],
                       "flops_per_point": 1}],
         "edges": [{"src": 0, "dst": 1, "src_dim": src_dim, "dst_dim": dst_dim, "elems": size ** rank}]}
    o = Oracle(g)
    K = o.configs(p, all_integers=all_int, volume=True)
    R = o.edge_costs(0)
    su, sv = o.splits(0), o.splits(1)
    for cu in range(int(K[0])):
        for cv in range(int(K[1])):
            want = pins.volume_transfer_elements(m, src_dim, dst_dim, [int(x) for x in su[cu]],
                                                 [int(x) for x in sv[cv]], 3)
            assert int(R[cu, cv]) == want, (su[cu], sv[cv])


def test_volume_transfer_symmetric_and_bounded():
    """t_x does not depend on the edge's direction (reversing every edge
    transposes every matrix), vanishes on identical unsplit ends, and never
    exceeds twice the tensor (r * 2 * elems)."""
    from oracle.oracle import Oracle
    g = workload("w1_residual_cnn")
    rev = dict(g, edges=[dict(e, src=e["dst"], dst=e["src"], src_dim=e["dst_dim"], dst_dim=e["src_dim"])
                         for e in g["edges"]])
    a, b = Oracle(g), Oracle(rev)
    a.configs(4, volume=True)
    b.configs(4, volume=True)
    for k, e in enumerate(g["edges"]):
        Ra, Rb = a.edge_costs(k), b.edge_costs(k)
        assert np.array_equal(Ra, Rb.T)
        assert int(Ra[0, 0]) == 0
        assert int(Ra.max()) <= 2 * 8 * e["elems"]


@pytest.mark.parametrize("seed", range(6))
def test_theorem1_volume_costs(seed):
    """The DP is unchanged by the transfer model: with volume costs the
    minimum equals exhaustive search and every table entry the conditioned
    exhaustive search."""
    from oracle.oracle import Oracle
    g = random_graph(seed + 580, n=3 + seed % 3, p=4, max_dims=2, extra_edges=seed % 3)
    o = Oracle(g)
    K = [int(k) for k in o.configs(4, volume=True)]
    o.solve()
    L, R, src, dst = _tables(o, g)
    mc, strat = o.result()
    assert mc == pins.brute_force(L, R, src, dst)[0] == pins.total_cost(strat, L, R, src, dst)
    seq = o.sequence()
    for i in range(len(seq)):
        D, T, A = pins.conditioned_table(L, R, src, dst, seq, i, K)
        To, Ao = o.table(i)
        assert To.tolist() == T and Ao.tolist() == A


# ------------------------------------------------------------------ weight-gradient all-reduce
def test_grad_sync_hand_values():
    """FC (64, 256, 256), weights (out, in) = 65 536 words, r = 8, p = 4:
    (4,1,1): 4 replicas of the whole weight, ring all-reduce 2*3/4*65536 = 98 304
    words: 2 097 152 + 786 432 = 2 883 584.  (1,4,1): one replica, no term:
    2 097 152.  (1,1,4): 2 490 368 (partial sums only).  (2,2,1): shards of
    32 768 held twice: 32 768 words, 2 359 296.  (2,1,2): 2 097 152 + 65 536
    (partial sums) + 262 144 = 2 424 832.  p = 6, (3,2,1): 3 replicas of
    32 768-word shards, ceil(2*2/3*32768) = 43 691 words: 1 398 102 + 349 528."""
    from oracle.oracle import Oracle
    o = Oracle(fc_chain())
    o.configs(4, grad_sync=True)
    sp = [tuple(int(x) for x in r) for r in o.splits(0)]
    L = o.layer_costs(0)
    want = {(4, 1, 1): 2_883_584, (1, 4, 1): 2_097_152, (1, 1, 4): 2_490_368, (2, 2, 1): 2_359_296,
            (2, 1, 2): 2_424_832}
    for t, v in want.items():
        assert int(L[sp.index(t)]) == v, t
    o = Oracle(fc_chain(p=6))
    o.configs(6, all_integers=True, grad_sync=True)
    sp = [tuple(int(x) for x in r) for r in o.splits(0)]
    assert int(o.layer_costs(0)[sp.index((3, 2, 1))]) == 1_747_630
    # without the option the costs are the benchmark's model
    o = Oracle(fc_chain())
    o.configs(4)
    sp = [tuple(int(x) for x in r) for r in o.splits(0)]
    assert int(o.layer_costs(0)[sp.index((4, 1, 1))]) == 2_097_152


def test_grad_sync_fc_chain_optimum():
    """With the gradient term W0's optimum is no longer data parallel: every
    layer split 4 ways over `out` (no replicas, no partial sums) costs
    2 097 152, and each of the 3 edges re-distributes 16 384 / 4 words, x 8:
    8 388 608 + 98 304 = 8 486 912, equal to exhaustive search."""
    from oracle.oracle import Oracle
    g = fc_chain()
    o = Oracle(g)
    o.configs(4, grad_sync=True)
    o.solve()
    L, R, src, dst = _tables(o, g)
    mc, strat = o.result()
    assert mc == 8_486_912 == pins.brute_force(L, R, src, dst)[0]
    sp = [tuple(int(x) for x in r) for r in o.splits(0)]
    assert [sp[c] for c in strat] == [(1, 4, 1)] * 4


@pytest.mark.parametrize("seed", range(6))
def test_theorem1_grad_sync(seed):
    """Random graphs with random weight tensors: the DP with the gradient term
    matches exhaustive search, entry by entry."""
    from oracle.oracle import Oracle
    g = random_graph(seed + 620, n=3 + seed % 3, p=4, max_dims=2, extra_edges=seed % 3)
    o = Oracle(g)
    K = [int(k) for k in o.configs(4, grad_sync=True)]
    o.solve()
    L, R, src, dst = _tables(o, g)
    assert o.result()[0] == pins.brute_force(L, R, src, dst)[0]
    seq = o.sequence()
    for i in range(len(seq)):
        D, T, A = pins.conditioned_table(L, R, src, dst, seq, i, K)
        To, Ao = o.table(i)
        assert To.tolist() == T and Ao.tolist() == A

# ------------------------------------------------------------------ breadth-first recurrence (eq. 2)
def _bfs_order(g):
    """Breadth-first traversal from vertex 0, neighbours in ascending id
    (collections.deque; independent of the oracle's traversal)."""
    from collections import deque
    nb = pins.neighbours(len(g["vertices"]), [e["src"] for e in g["edges"]], [e["dst"] for e in g["edges"]])
    order, seen, q = [], {0}, deque([0])
    while q:
        v = q.popleft()
        order.append(v)
        for u in sorted(nb[v]):
            if u not in seen:
                seen.add(u)
                q.append(u)
    return order, nb


@pytest.mark.parametrize("seed", range(12))
def test_bf_recurrence_against_brute_force(seed):
    """Eq. (2): the order is a breadth-first traversal, D_B(i) = N(V<=i) after
    i, B(|V|, empty) is the minimum over all strategies, and every entry of
    every table B_i (with its lowest-index argmin) equals the exhaustive
    conditioned search; model costs and dense random ties; both configuration
    sets."""
    from oracle.oracle import Oracle
    all_int = seed % 4 == 3
    p = 6 if all_int else 4
    g = random_graph(seed + 500, n=3 + seed % 5, p=p, max_dims=2, extra_edges=seed % 4)
    o = Oracle(g)
    K = [int(k) for k in o.configs(p, all_integers=all_int)]
    if seed % 2:
        o.set_costs(*random_costs(seed, K, [(K[e["src"]], K[e["dst"]]) for e in g["edges"]], hi=4))
    o.solve_bf()
    L, R, src, dst = _tables(o, g)
    order, nb = _bfs_order(g)
    assert o.sequence() == order
    mc, strat = o.result()
    bf_min, optimal = pins.brute_force(L, R, src, dst)
    assert mc == bf_min and pins.total_cost(strat, L, R, src, dst) == mc and bool(optimal[tuple(strat)])
    for i in range(len(order)):
        assert o.dependent_set(i) == pins.bfs_dependent_set(nb, order, i)
        D, T, A = pins.conditioned_table(L, R, src, dst, order, i, K)
        assert D == o.dependent_set(i)
        To, Ao = o.table(i)
        assert To.tolist() == T and Ao.tolist() == A, i


@pytest.mark.parametrize("seed", range(6))
def test_bf_recurrence_is_recurrence4_on_a_bf_order(seed):
    """On a breadth-first order V<=i is connected, so X(i) = V<=i, D(i) = D_B(i)
    and S(i) = {V<=i-1}: recurrence (4) over that order gives the same tables,
    entry by entry, as the chain recurrence (2)."""
    from oracle.oracle import Oracle
    g = random_graph(seed + 520, n=6 + seed % 4, p=8, max_dims=3, extra_edges=2 + seed % 3)
    a, b = Oracle(g), Oracle(g)
    a.configs(8)
    b.configs(8)
    a.solve_bf()
    order, _ = _bfs_order(g)
    b.solve(order=order)
    assert a.sequence() == b.sequence() == order
    assert a.result() == b.result()
    for i in range(len(order)):
        assert a.dependent_set(i) == b.dependent_set(i)
        Ta, Aa = a.table(i)
        Tb, Ab = b.table(i)
        assert np.array_equal(Ta, Tb) and np.array_equal(Aa, Ab)


@pytest.mark.parametrize("seed", range(4))
def test_bf_recurrence_viterbi_on_chains(seed):
    """A path numbered from one end: the breadth-first order is the path and
    eq. (2) is the Viterbi recursion."""
    from oracle.oracle import Oracle
    g = chain_graph(seed + 40, n=5 + seed, p=8, max_dims=3)
    o = Oracle(g)
    o.configs(8)
    o.solve_bf()
    assert o.sequence() == list(range(len(g["vertices"])))
    L, R, src, dst = _tables(o, g)
    forward = [e["src"] < e["dst"] for e in g["edges"]]
    mc, strat = o.result()
    vmin, _ = pins.viterbi_chain(L, R, forward)
    tmin, tstrat = pins.viterbi_table_strategy(L, R, forward)
    assert mc == vmin == tmin and strat == tstrat


def test_bf_dependent_sets_blow_up_on_dense_graphs():
    """The contrast of Table I: on the Inception-style and Transformer graphs
    the breadth-first dependent sets reach 8 and 19 vertices (tables past
    2^34 entries, refused), while GenerateSeq keeps them at 2 and 3; on the
    FC chain both orders give the same 310 cells."""
    from oracle.oracle import Oracle, OracleError
    for name, want, ours in (("w2_inception", 8, 2), ("w4_transformer", 19, 3)):
        g = workload(name)
        order, nb = _bfs_order(g)
        assert max(len(pins.bfs_dependent_set(nb, order, i)) for i in range(len(order))) == want
        o = Oracle(g)
        o.configs(g["p"])
        with pytest.raises(OracleError):
            o.solve_bf()
        o.solve(max_cells=1)
        assert max(len(o.dependent_set(i)) for i in range(len(order))) == ours
    o = Oracle(fc_chain())
    o.configs(4)
    o.solve_bf()
    assert o.result() == (8_388_608, [9, 9, 9, 9]) and o.cells() == 310

# ------------------------------------------------------------------ halo exchange of convolutions
def _conv_graph(h, w, k, p):
    return {"name": "conv", "p": p, "comm_weight": 8,
            "vertices": [{"name": "c", "dims": [2, 4, 3, h, w], "dim_names": ["b", "co", "ci", "h", "w"],
                          "reduce": [2], "flops_per_point": 2 * k * k,
                          "halo": [0, 0, 0, k // 2, k // 2], "input_dims": [0, 2, 3, 4]}], "edges": []}


def test_halo_hand_values():
    """A 3x3 convolution (b 2, co 4, ci 3, h 8, w 6), r = 8, p = 4, FLOPs
    18 * 1152 = 20 736.  (1,1,1,2,1): 10 368 + 8 * 2 * 1 * (b ci w = 36) = 10 944.
    (1,1,1,2,2): 5 184 + 8 * (2 * ceil(36 / 2) + 2 * ceil(48 / 2)) = 5 856.
    (2,1,1,2,1): 5 184 + 8 * 2 * ceil(36 / 2) = 5 472.  (1,1,4,1,1): no halo,
    5 184 + 8 * 3 * 384 = 14 400.  Ragged, every integer split, p = 6, h 7,
    w 5, (1,1,1,3,2): ceil(15 120 / 6) = 2 520 + 8 * (2 * ceil(30 / 2) +
    2 * ceil(42 / 3)) = 2 984; with a 5x5 kernel (halo 2, 18 * 25 / 9 the
    FLOPs): 7 000 + 8 * (4 * 15 + 4 * 14) = 7 928."""
    from oracle.oracle import Oracle
    o = Oracle(_conv_graph(8, 6, 3, 4))
    o.configs(4, halo=True)
    sp = [tuple(int(x) for x in r) for r in o.splits(0)]
    L = o.layer_costs(0)
    want = {(1, 1, 1, 2, 1): 10_944, (1, 1, 1, 2, 2): 5_856, (2, 1, 1, 2, 1): 5_472, (1, 1, 4, 1, 1): 14_400,
            (1, 1, 1, 1, 1): 20_736}
    for t, v in want.items():
        assert int(L[sp.index(t)]) == v, t
    o.configs(4)   # the option off: the benchmark's model
    assert int(o.layer_costs(0)[sp.index((1, 1, 1, 2, 1))]) == 10_368
    o = Oracle(_conv_graph(7, 5, 3, 6))
    o.configs(6, all_integers=True, halo=True)
    sp = [tuple(int(x) for x in r) for r in o.splits(0)]
    assert int(o.layer_costs(0)[sp.index((1, 1, 1, 3, 2))]) == 2_984
    o = Oracle(_conv_graph(7, 5, 5, 6))
    o.configs(6, all_integers=True, halo=True)
    assert int(o.layer_costs(0)[sp.index((1, 1, 1, 3, 2))]) == 7_928


def test_halo_invariants():
    """The halo term vanishes for configurations that split no halo dim and
    for 1x1 kernels; it is symmetric in h and w on a square input; it never
    grows when a non-halo input dim is split further."""
    from oracle.oracle import Oracle
    for k in (1, 3, 5):
        g = _conv_graph(8, 8, k, 16)
        a, b = Oracle(g), Oracle(g)
        a.configs(16, halo=True)
        b.configs(16)
        sp = [tuple(int(x) for x in r) for r in a.splits(0)]
        La, Lb = a.layer_costs(0), b.layer_costs(0)
        for c, t in enumerate(sp):
            if k == 1 or (t[3] == 1 and t[4] == 1):
                assert La[c] == Lb[c], t
            else:
                assert La[c] > Lb[c], t
            mirror = (t[0], t[1], t[2], t[4], t[3])
            assert La[c] - Lb[c] == La[sp.index(mirror)] - Lb[sp.index(mirror)], t
            if t[0] * 2 * t[1] * t[2] * t[3] * t[4] <= 16:
                more_b = (2 * t[0],) + t[1:]
                d = sp.index(more_b)
                assert La[d] - Lb[d] <= La[c] - Lb[c], t


def _halo_graph(seed):
    """The first random graph from seed on whose layers carry a halo."""
    while True:
        g = random_graph(seed, n=3 + seed % 3, p=4, max_dims=3, extra_edges=seed % 3)
        if sum(1 for v in g["vertices"] if any(v.get("halo", []))) >= 2:
            return g
        seed += 1000


@pytest.mark.parametrize("seed", range(4))
def test_theorem1_halo(seed):
    """Random graphs with convolution geometry: the DP minimum under the halo
    term equals exhaustive search over every strategy."""
    g = _halo_graph(seed + 1400)
    from oracle.oracle import Oracle
    o = Oracle(g)
    o.configs(4, halo=True)
    o.solve()
    L, R, src, dst = _tables(o, g)
    assert o.result()[0] == pins.brute_force(L, R, src, dst)[0]


# ------------------------------------------------------------------ greedy device assignment
def _pair_graph(m, src_dim, dst_dim, du, dv, p=4, r=2):
    """Two vertices joined by one edge carrying a tensor of dims m."""
    return {"name": "pair", "p": p, "comm_weight": r,
            "vertices": [{"name": "u", "dims": [max(m)] * du, "dim_names": [f"a{k}" for k in range(du)],
                          "reduce": [], "flops_per_point": 1},
                         {"name": "v", "dims": [max(m)] * dv, "dim_names": [f"b{k}" for k in range(dv)],
                          "reduce": [], "flops_per_point": 1}],
            "edges": [{"src": 0, "dst": 1, "src_dim": list(src_dim), "dst_dim": list(dst_dim),
                       "elems": int(np.prod(m))}]}


def test_assign_transposed_splits():
    """u splits (x, y) 2 x 2, v receives the tensor transposed (tensor dim 0
    on its loop dim 1) and splits it 2 x 2 too: the grid numbering puts
    mismatched parts on devices 1 and 2 (the volume model charges 2 * 2 * 4 =
    16), the greedy assignment swaps them -- full locality, no transfer."""
    from oracle.oracle import Oracle
    g = _pair_graph([4, 4], [0, 1], [1, 0], 2, 2)
    o = Oracle(g)
    o.configs(4, volume=True)
    sp = [[tuple(int(x) for x in r) for r in o.splits(v)] for v in range(2)]
    cu, cv = sp[0].index((2, 2)), sp[1].index((2, 2))
    assert int(o.edge_costs(0)[cu, cv]) == 16
    dev, loc, xfer = o.assign_devices([cu, cv])
    assert dev[0].tolist() == [0, 1, 2, 3]
    assert dev[1].tolist() == [0, 2, 1, 3]
    assert loc.tolist() == [16] and xfer.tolist() == [0]
    assert pins.assigned_transfer_elements([4, 4], [0, 1], [1, 0], [2, 2], [2, 2], dev[0].tolist(),
                                           dev[1].tolist(), 2) == (16, 0)


@pytest.mark.parametrize("seed", range(12))
def test_assign_against_enumeration(seed):
    """Random two-vertex edges (tensor dims of 4 or 8 elements, random maps,
    p = 4, every strategy): the oracle's locality and transfer under its
    assignment equal element enumeration with the same device maps; each
    vertex's parts sit on distinct devices; the first keeps the grid
    numbering (and then the transfer equals the volume model's when the
    second does too); the greedy reaches at least half the best locality over
    every injective map of the second vertex's parts (the greedy matching
    bound), and the best itself when that best is the whole tensor."""
    from oracle.oracle import Oracle
    rng = np.random.default_rng(seed + 77)
    rank = int(rng.integers(1, 3))
    m = [int(rng.choice([4, 8])) for _ in range(rank)]
    du, dv = int(rng.integers(1, 3)), int(rng.integers(1, 3))
    sd = [int(rng.integers(-1, du)) for _ in range(rank)]
    dd = [int(rng.integers(-1, dv)) for _ in range(rank)]
    g = _pair_graph(m, sd, dd, du, dv)
    o = Oracle(g)
    K = o.configs(4, volume=True)
    sp = [[[int(x) for x in r] for r in o.splits(v)] for v in range(2)]
    R = o.edge_costs(0)
    for cu in range(int(K[0])):
        for cv in range(int(K[1])):
            dev, loc, xfer = o.assign_devices([cu, cv])
            pu, pv = int(np.prod(sp[0][cu])), int(np.prod(sp[1][cv]))
            assert dev[0].tolist() == list(range(pu)) + [-1] * (4 - pu)
            assert sorted(x for x in dev[1].tolist() if x >= 0) == list(range(pv))
            want = pins.assigned_transfer_elements(m, sd, dd, sp[0][cu], sp[1][cv], dev[0].tolist(),
                                                   dev[1].tolist(), 2)
            assert (int(loc[0]), int(xfer[0])) == want, (cu, cv)
            if dev[1].tolist() == list(range(pv)) + [-1] * (4 - pv):
                assert int(xfer[0]) == int(R[cu, cv])
            best = 0
            for devs in itertools.permutations(range(4), pv):
                part_v = [-1] * 4
                for h, d in enumerate(devs):
                    part_v[d] = h
                best = max(best, pins.assigned_transfer_elements(m, sd, dd, sp[0][cu], sp[1][cv],
                                                                 dev[0].tolist(), part_v, 2)[0])
            assert 2 * int(loc[0]) >= best, (cu, cv)
            if best == int(np.prod(m)) and pu == pv:
                assert int(loc[0]) == best, (cu, cv)


def test_assign_workloads_are_consistent():
    """On W0 and a residual CNN strategy the assignment is a set of injective
    maps, and the locality of each edge never exceeds its tensor."""
    from oracle.oracle import Oracle
    for g in (fc_chain(), workload("w1_residual_cnn")):
        o = Oracle(g)
        o.configs(g["p"], volume=True)
        o.solve()
        dev, loc, xfer = o.assign_devices(o.result()[1])
        for v in range(len(g["vertices"])):
            parts = [x for x in dev[v].tolist() if x >= 0]
            assert len(parts) == len(set(parts))
        for e, ed in enumerate(g["edges"]):
            assert int(loc[e]) <= ed["elems"]


# ------------------------------------------------------------------ planted mistakes
MUTANTS = {
    "tie_break_last": ("if (c == 0 || cand < best) { best = cand; best_c = c; }",
                       "if (c == 0 || cand <= best) { best = cand; best_c = c; }"),
    "transposed_edge": ("uint64_t x = o->Rx[e][(size_t)cfg_of[u] * o->K[v] + cfg_of[v]];",
                        "uint64_t x = o->Rx[e][(size_t)cfg_of[v] * o->K[u] + cfg_of[u]];"),
    "dropped_lookup": ("for (int t = 0; t < nsub; t++) {   /* the subproblems' optima */",
                       "for (int t = 1; t < nsub; t++) {   /* the subproblems' optima */"),
    "earlier_edges": ("if (other >= 0 && o->pos[other] > i) later[nlater++] = e;",
                      "if (other >= 0 && o->pos[other] < i) later[nlater++] = e;"),
    "seq_tie_highest": ("if (best < 0 || sz < best_sz) { best = u; best_sz = sz; }",
                        "if (best < 0 || sz <= best_sz) { best = u; best_sz = sz; }"),
    "comm_off_by_one": ("if (!mul_ok(red_split - 1, ceil_div(keep_n, keep_split), &comm)) return 0;",
                        "if (!mul_ok(red_split, ceil_div(keep_n, keep_split), &comm)) return 0;"),
    "floor_not_ceil": ("static uint64_t ceil_div(uint64_t a, uint64_t b) { return a / b + (a % b != 0); }",
                       "static uint64_t ceil_div(uint64_t a, uint64_t b) { return a / b; }"),
    "no_match_check": ("if (su != sv) match = 0;", "if (su != sv) match = 1;"),
    "budget_difference": ("if (!enum_rec(d, k + 1, budget / s, pow2, cur, out, count, cap)) return 0;",
                          "if (!enum_rec(d, k + 1, budget - s + 1, pow2, cur, out, count, cap)) return 0;"),
    "bf_no_chain_term": ("if (i > 0 && !add_ok(cost, o->T[i - 1][table_index(o, i - 1, cfg_of)], &cost)) {",
                         "if (i > 1 && !add_ok(cost, o->T[i - 1][table_index(o, i - 1, cfg_of)], &cost)) {"),
    "bf_dependent_inclusive": ("for (int k = 0; k < o->deg[w] && !adjacent; k++) adjacent = o->pos[o->nbr[w][k]] <= i;",
                               "for (int k = 0; k < o->deg[w] && !adjacent; k++) adjacent = o->pos[o->nbr[w][k]] < i;"),
    "bf_earlier_edges": ("if ((a == vi && o->pos[b] > i) || (b == vi && o->pos[a] > i)) later[nlater++] = e;",
                         "if ((a == vi && o->pos[b] < i) || (b == vi && o->pos[a] < i)) later[nlater++] = e;"),
    "volume_forward_only": ("unsigned __int128 words = (E * fwd + cells - 1) / cells + (E * bwd + cells - 1) / cells;",
                            "unsigned __int128 words = (E * fwd + cells - 1) / cells;"),
    "volume_dim0_fastest": ("for (int k = o->ndims[u] - 1; k >= 0; k--) { xu_loop[k] = x % su_[k]; x /= su_[k]; }",
                            "for (int k = 0; k < o->ndims[u]; k++) { xu_loop[k] = x % su_[k]; x /= su_[k]; }"),
    "grad_replicas": ("unsigned __int128 words = ((unsigned __int128)2 * (R - 1) * S + (R - 1)) / R;",
                      "unsigned __int128 words = ((unsigned __int128)2 * R * S + (R - 1)) / R;"),
    "pow2_only": ("for (uint64_t s = 1; s <= budget; s = pow2 ? 2 * s : s + 1) {",
                  "for (uint64_t s = 1; s <= budget; s = 2 * s) {"),
    "edge_min_devices": ("uint64_t words = ceil_div(o->elems[e], Pu > Pv ? Pu : Pv);",
                         "uint64_t words = ceil_div(o->elems[e], Pu < Pv ? Pu : Pv);"),
    "compute_over_kept_split": ("uint64_t compute = ceil_div(flops, P);",
                                "uint64_t compute = ceil_div(flops, keep_split);"),
    "comm_over_all_devices": ("if (!mul_ok(red_split - 1, ceil_div(keep_n, keep_split), &comm)) return 0;",
                              "if (!mul_ok(red_split - 1, ceil_div(keep_n, P), &comm)) return 0;"),
    "seq_keeps_self": ("if (rule == 1) {", "if (rule != 2) {"),
    "assign_smallest": ("if (bg < 0 || W[g * p + d] > best) { bg = (int)g; bd = d; best = W[g * p + d]; }",
                        "if (bg < 0 || W[g * p + d] < best) { bg = (int)g; bd = d; best = W[g * p + d]; }"),
    "assign_later_neighbours": ("if (other < 0 || other > v) continue;   /* placed neighbours only */",
                                "if (other < 0 || other < v) continue;   /* placed neighbours only */"),
    "assign_ties_last": ("if (bg < 0 || W[g * p + d] > best) { bg = (int)g; bd = d; best = W[g * p + d]; }",
                         "if (bg < 0 || W[g * p + d] >= best) { bg = (int)g; bd = d; best = W[g * p + d]; }"),
    "assign_forward_only": ("unsigned __int128 moved = (E * fwd + cells - 1) / cells + (E * bwd + cells - 1) / cells;",
                            "unsigned __int128 moved = (E * fwd + cells - 1) / cells;"),
    "halo_one_neighbour": ("if (!mul_ok(2 * w, ceil_div(rest, rest_split), &words)) return 0;",
                           "if (!mul_ok(w, ceil_div(rest, rest_split), &words)) return 0;"),
    "halo_own_split": ("if (j == k || !(o->in_mask[v] >> j & 1u)) continue;",
                       "if (!(o->in_mask[v] >> j & 1u)) continue;"),
    "halo_when_unsplit": ("if (w == 0 || s[k] == 1) continue;", "if (w == 0) continue;"),
    "grad_replicas_from_weight_dims": ("                Pw *= s[k];\n            } else {\n                R *= s[k];",
                                       "                R *= s[k];\n            } else {\n                Pw *= s[k];"),
}


def _pin_suite(lib):
    """A compact run of the pins above against an oracle library; returns the
    list of pins that failed."""
    failed = []
    from oracle.oracle import Oracle, OracleError

    def guard(name, fn):
        try:
            if not fn():
                failed.append(name)
        except (AssertionError, OracleError, ValueError, IndexError):
            failed.append(name)

    def w0():
        o, _ = _solve(fc_chain(), lib=lib)
        return o.result() == (8_388_608, [9, 9, 9, 9]) and o.sequence() == [0, 1, 2, 3]

    def hand_costs():
        o = Oracle({"name": "r", "p": 4, "comm_weight": 8,
                    "vertices": [{"name": "v", "dims": [3, 5], "dim_names": ["a", "b"],
                                  "reduce": [1], "flops_per_point": 3}], "edges": []}, lib)
        o.configs(4)
        ex = [tuple(int(x) for x in r) for r in o.exponents(0)]
        L = o.layer_costs(0)
        return int(L[ex.index((1, 1))]) == 28 and int(L[ex.index((0, 2))]) == 84

    def edge_costs():
        o = Oracle(fc_chain(), lib)
        o.configs(4)
        ex = [tuple(int(x) for x in r) for r in o.exponents(0)]
        R = o.edge_costs(0)
        return (int(R[ex.index((2, 0, 0)), ex.index((0, 0, 2))]) == 8 * 4096
                and int(R[ex.index((1, 1, 0)), ex.index((1, 0, 1))]) == 0
                and int(R[ex.index((0, 0, 0)), ex.index((1, 0, 0))]) == 8 * 8192)   # max(P_u, P_v) = 2

    def tables():
        for seed in range(6):
            g = random_graph(seed + 100, n=3 + seed % 4, p=4, max_dims=2, extra_edges=1 + seed % 3)
            o0 = Oracle(g, lib)
            K = o0.configs(4)
            costs = random_costs(seed, K, [(K[e["src"]], K[e["dst"]]) for e in g["edges"]], hi=4)
            o, K = _solve(g, costs=costs, lib=lib)
            L, R, src, dst = _tables(o, g)
            seq = o.sequence()
            nb = pins.neighbours(len(seq), src, dst)
            for i in range(len(seq)):
                if o.dependent_set(i) != pins.dependent_set(nb, seq, i):
                    return False
                D, T, A = pins.conditioned_table(L, R, src, dst, seq, i, [int(k) for k in K])
                To, Ao = o.table(i)
                if To.tolist() != T or Ao.tolist() != A:
                    return False
            mc, strat = o.result()
            if mc != pins.brute_force(L, R, src, dst)[0]:
                return False
        return True

    def all_integers():
        o = Oracle({"name": "one", "p": 12, "comm_weight": 8,
                    "vertices": [{"name": "v", "dims": [7, 7], "dim_names": ["x", "y"],
                                  "reduce": [], "flops_per_point": 1}], "edges": []}, lib)
        o.configs(12, all_integers=True)
        sp = [tuple(int(x) for x in r) for r in o.splits(0)]
        o = Oracle(fc_chain(p=6), lib)
        o.configs(6, all_integers=True)
        sf = [tuple(int(x) for x in r) for r in o.splits(0)]
        return (sp == [t for t in itertools.product(range(1, 13), repeat=2) if t[0] * t[1] <= 12]
                and int(o.layer_costs(0)[sf.index((1, 2, 3))]) == 1_529_174
                and int(o.edge_costs(0)[sf.index((3, 1, 1)), sf.index((1, 1, 3))]) == 43_696)

    def bf():
        for seed in range(4):
            g = random_graph(seed + 500, n=4 + seed, p=4, max_dims=2, extra_edges=1 + seed % 3)
            o = Oracle(g, lib)
            K = [int(k) for k in o.configs(4)]
            o.set_costs(*random_costs(seed, K, [(K[e["src"]], K[e["dst"]]) for e in g["edges"]], hi=4))
            o.solve_bf()
            L, R, src, dst = _tables(o, g)
            order = o.sequence()
            for i in range(len(order)):
                D, T, A = pins.conditioned_table(L, R, src, dst, order, i, K)
                To, Ao = o.table(i)
                if o.dependent_set(i) != D or To.tolist() != T or Ao.tolist() != A:
                    return False
            if o.result()[0] != pins.brute_force(L, R, src, dst)[0]:
                return False
        return True

    def volume():
        o = Oracle(fc_chain(), lib)
        o.configs(4, volume=True)
        sp = [tuple(int(x) for x in r) for r in o.splits(0)]
        R = o.edge_costs(0)
        if int(R[sp.index((1, 2, 2)), sp.index((1, 1, 2))]) != 131_072:
            return False
        g = {"name": "vol", "p": 4, "comm_weight": 3,
             "vertices": [{"name": "u", "dims": [12, 12], "dim_names": ["x", "y"], "reduce": [],
                           "flops_per_point": 1},
                          {"name": "v", "dims": [12, 12], "dim_names": ["x", "y"], "reduce": [],
                           "flops_per_point": 1}],
             "edges": [{"src": 0, "dst": 1, "src_dim": [1, 0], "dst_dim": [0, -1], "elems": 144}]}
        o = Oracle(g, lib)
        K = o.configs(4, volume=True)
        R = o.edge_costs(0)
        su, sv = o.splits(0), o.splits(1)
        for cu in range(int(K[0])):
            for cv in range(int(K[1])):
                want = pins.volume_transfer_elements([12, 12], [1, 0], [0, -1], [int(x) for x in su[cu]],
                                                     [int(x) for x in sv[cv]], 3)
                if int(R[cu, cv]) != want:
                    return False
        return True

    def grad():
        o = Oracle(fc_chain(), lib)
        o.configs(4, grad_sync=True)
        sp = [tuple(int(x) for x in r) for r in o.splits(0)]
        L = o.layer_costs(0)
        return int(L[sp.index((4, 1, 1))]) == 2_883_584 and int(L[sp.index((2, 2, 1))]) == 2_359_296

    def halo():
        o = Oracle(_conv_graph(8, 6, 3, 4), lib)
        o.configs(4, halo=True)
        sp = [tuple(int(x) for x in r) for r in o.splits(0)]
        L = o.layer_costs(0)
        return (int(L[sp.index((1, 1, 1, 2, 1))]) == 10_944 and int(L[sp.index((1, 1, 1, 2, 2))]) == 5_856
                and int(L[sp.index((1, 1, 1, 1, 1))]) == 20_736)

    def assign():
        g = _pair_graph([4, 4], [0, 1], [1, 0], 2, 2)
        o = Oracle(g, lib)
        o.configs(4, volume=True)
        sp = [[tuple(int(x) for x in r) for r in o.splits(v)] for v in range(2)]
        dev, loc, xfer = o.assign_devices([sp[0].index((2, 2)), sp[1].index((2, 2))])
        if dev[1].tolist() != [0, 2, 1, 3] or loc.tolist() != [16] or xfer.tolist() != [0]:
            return False
        # a 2-part consumer next to a 4-part producer: ties between the parts'
        # equal localities go to the lowest device
        g = _pair_graph([4, 4], [0, 1], [0, -1], 2, 1)
        o = Oracle(g, lib)
        o.configs(4, volume=True)
        sp = [[tuple(int(x) for x in r) for r in o.splits(v)] for v in range(2)]
        dev, loc, xfer = o.assign_devices([sp[0].index((2, 2)), sp[1].index((2,))])
        if dev[1].tolist() != [0, -1, 1, -1] or loc.tolist() != [8]:
            return False
        # both directions of the transfer against element enumeration
        return (int(loc[0]), int(xfer[0])) == pins.assigned_transfer_elements(
            [4, 4], [0, 1], [0, -1], [2, 2], [2], dev[0].tolist(), dev[1].tolist(), 2)

    guard("w0", w0)
    guard("grad", grad)
    guard("halo", halo)
    guard("assign", assign)
    guard("bf", bf)
    guard("volume", volume)
    guard("all_integers", all_integers)
    guard("hand_costs", hand_costs)
    guard("edge_costs", edge_costs)
    guard("tables", tables)
    return failed


def test_pins_pass_on_the_oracle():
    from oracle import oracle
    assert _pin_suite(oracle._LIB) == []


@pytest.mark.parametrize("mutant", sorted(MUTANTS))
def test_pins_catch_planted_mistakes(mutant, tmp_path):
    """Each plausible mistake planted in a copy of the oracle source makes at
    least one pin fail (the mistake is planted on the CPU, never on a GPU)."""
    from oracle import oracle
    old, new = MUTANTS[mutant]
    src = open(oracle._SRC).read()
    assert src.count(old) == 1, mutant
    path = tmp_path / f"mut_{mutant}.c"
    path.write_text(src.replace(old, new))
    lib = oracle.build(force=True, src=str(path), out=str(tmp_path / f"lib_{mutant}.so"))
    assert _pin_suite(lib) != [], mutant
