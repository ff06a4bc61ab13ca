"""Host-side tests of libpase (no GPU): the library loads and exports the C ABI,
input validation and error paths, configuration enumeration, GenerateSeq and
the dependent sets (checked against the oracle and against their definition)."""
import os
import re

import numpy as np
import pytest

import pins
from workloads import fc_chain, random_costs, random_graph, transformer, workload

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def pase():
    from paper_2407_04001_amd import pase as P
    P.load()
    return P


def test_exports_every_declared_symbol(pase):
    header = open(os.path.join(ROOT, "include", "pase.h")).read()
    declared = set(re.findall(r"\b(pase_[a-z_]+)\s*\(", header))
    assert declared, "no declarations found"
    lib = pase.load()
    for name in sorted(declared):
        assert hasattr(lib, name), name
    assert declared == set(pase.EXPORTS)


def _status(fn):
    from paper_2407_04001_amd.pase import PaseError
    try:
        fn()
    except PaseError as e:
        return e.status
    return 0


def test_create_validation(pase):
    g = fc_chain()
    P = pase
    bad = []
    v = [dict(x) for x in g["vertices"]]
    e = [dict(x) for x in g["edges"]]
    bad.append((v, [dict(e[0], dst=e[0]["src"])]))                       # self-loop
    bad.append(([dict(v[0], dims=[])] + v[1:], e))                        # ndims 0
    bad.append(([dict(v[0], dims=[0, 1, 1])] + v[1:], e))                 # size 0
    bad.append((v, [dict(e[0], src_dim=[0, 5])] + e[1:]))                 # map out of range
    bad.append((v, [dict(e[0], elems=0)] + e[1:]))                        # elems 0
    bad.append((v, [dict(e[0], dst=17)] + e[1:]))                         # id out of range
    bad.append(([dict(v[0], reduce=[3])] + v[1:], e))                     # reduce dim out of range
    for vv, ee in bad:
        assert _status(lambda: P.pase_graph_create(vv, ee)) == P.INVALID_ARGUMENT
    # disconnected: drop the middle edge of the chain
    assert _status(lambda: P.pase_graph_create(v, [e[0], e[2]])) == P.NOT_CONNECTED
    assert _status(lambda: P.pase_graph_create(v, e, seq_rule=2)) == P.INVALID_ARGUMENT


def test_call_order_and_p(pase):
    P = pase
    g = P.Graph(fc_chain())
    assert _status(lambda: g.sequence()) == P.BAD_STATE
    assert _status(lambda: P.pase_num_configs(g.h, 0)) == P.BAD_STATE
    assert _status(lambda: P.pase_stats(g.h)) == P.BAD_STATE
    for p in (0, 3, 6, 1 << 17):
        assert _status(lambda: g.enumerate_configs(p)) == P.INVALID_ARGUMENT
    g.enumerate_configs(4)
    assert _status(lambda: g.table_entry(0, [0])) == P.BAD_STATE       # no search yet


def test_overflow_and_too_large(pase):
    P = pase
    big = {"vertices": [{"dims": [2**40, 2**30], "reduce": [], "flops_per_point": 1}], "edges": []}
    g = P.Graph(big)
    assert _status(lambda: g.enumerate_configs(2)) == P.OVERFLOW
    # a 6-clique at p=64: the first dependent set has 5 members of 84 configs -> table > 2^31
    vs = [{"dims": [8, 8, 8], "reduce": [], "flops_per_point": 1} for _ in range(6)]
    es = [{"src": a, "dst": b, "src_dim": [0], "dst_dim": [0], "elems": 8}
          for a in range(6) for b in range(a + 1, 6)]
    g = P.Graph({"vertices": vs, "edges": es})
    assert _status(lambda: g.enumerate_configs(64)) == P.TOO_LARGE
    # the memory budget is enforced before any device work
    g = P.Graph(transformer())
    g.enumerate_configs(64)
    assert _status(lambda: g.set_option(P.OPT_MEMORY_BUDGET, 1 << 20)) == P.TOO_LARGE


def test_lent_workspace_too_small(pase):
    P = pase
    g = P.Graph(fc_chain())
    g.enumerate_configs(4)
    assert g.workspace_size() > 0
    P.pase_set_workspace(g.h, 4096 * 256, 256)
    assert _status(lambda: P.pase_find_best_strategy(g.h, 4)) == P.OUT_OF_MEMORY
    assert _status(lambda: P.pase_set_workspace(g.h, 4096 * 256 + 8, 1 << 20)) == P.INVALID_ARGUMENT


def test_configs_match_oracle(pase):
    from oracle.oracle import Oracle
    for name in ("w0_fc_chain", "w1_residual_cnn", "w4_transformer"):
        g = workload(name)
        pg = pase.Graph(g)
        pg.enumerate_configs(g["p"])
        K = pg.K
        o = Oracle(g)
        assert list(o.configs(g["p"])) == K
        for v in (0, len(K) - 1):
            ex = o.exponents(v)
            for c in range(K[v]):
                assert pg.config_splits(v, c) == [1 << int(x) for x in ex[c]]
    g = fc_chain()
    pg = pase.Graph(g)
    pg.enumerate_configs(4)
    assert pg.config_splits(0, 9) == [4, 1, 1]


@pytest.mark.parametrize("p", [1, 2, 3, 5, 6, 7, 12, 16, 24, 255])
def test_all_integer_configs_match_oracle(pase, p):
    """PASE_OPT_CONFIG_SET = 1: the library's configurations (count, order and
    split factors) are the oracle's every-integer set, for 1 to 8 loop dims."""
    from oracle.oracle import Oracle
    vs = [{"name": f"v{d}", "dims": [5] * d, "dim_names": ["x"] * d, "reduce": [],
           "flops_per_point": 1} for d in range(1, 9)]
    es = [{"src": d, "dst": d + 1, "src_dim": [0], "dst_dim": [0], "elems": 5} for d in range(7)]
    g = {"name": "dims", "p": p, "comm_weight": 8, "vertices": vs, "edges": es}
    o = Oracle(g)
    try:
        Ko = [int(k) for k in o.configs(p, all_integers=True)]
    except Exception:
        Ko = None
    pg = pase.Graph(g)
    if Ko is None:   # more than 65535 configurations for some vertex
        assert _status(lambda: pg.enumerate_configs(p, all_integers=True)) == pase.TOO_LARGE
        return
    pg.enumerate_configs(p, all_integers=True)
    assert pg.K == Ko
    for v in range(len(vs)):
        sp = o.splits(v)
        for c in range(Ko[v]) if Ko[v] < 2000 else range(0, Ko[v], 7):
            assert pg.config_splits(v, c) == [int(x) for x in sp[c]]


def test_config_set_option(pase):
    """The option takes effect at the next enumeration; p outside the set's
    range is rejected; switching back restores the power-of-two set."""
    P = pase
    g = fc_chain()
    pg = P.Graph(g)
    pg.enumerate_configs(4)
    assert pg.K[0] == 10
    pg.enumerate_configs(4, all_integers=True)
    assert pg.K[0] == 13          # 10 + (3,1,1), (1,3,1), (1,1,3)
    assert pg.config_splits(0, 12) == [4, 1, 1]
    assert _status(lambda: pg.enumerate_configs(256)) == P.INVALID_ARGUMENT
    assert _status(lambda: pg.enumerate_configs(0)) == P.INVALID_ARGUMENT
    pg.enumerate_configs(6)
    assert pg.K[0] == 25          # N_3(6) = N_2(6) + N_2(3) + N_2(2) + 3 N_2(1) = 14 + 5 + 3 + 3
    pg.enumerate_configs(4, all_integers=False)
    assert pg.K[0] == 10
    assert _status(lambda: pg.enumerate_configs(6)) == P.INVALID_ARGUMENT
    assert _status(lambda: P.pase_set_option(pg.h, P.OPT_CONFIG_SET, 2)) == P.INVALID_ARGUMENT


@pytest.mark.parametrize("seed", range(16))
def test_key_bounds_hold(pase, seed):
    """The per-position bounds that size the keys hold on the oracle's tables:
    key_bound >= the largest value minimised over at that position (exhaustive
    search) and table_bound >= every table entry; model costs with both
    configuration sets, with the gradient term, the halo term, volume transfer
    costs, and caller-given costs."""
    from oracle.oracle import Oracle
    all_int = seed % 3 == 1
    p = (4, 6, 8)[seed % 3]
    grad, volume, halo = seed % 4 == 3, seed % 5 == 4, seed % 2 == 1
    g = random_graph(seed + 900, n=3 + seed % 4, p=p, max_dims=2, extra_edges=seed % 3, max_size=200)
    o = Oracle(g)
    K = [int(k) for k in o.configs(p, all_integers=all_int, grad_sync=grad, volume=volume, halo=halo)]
    costs = None
    if seed % 3 == 2:
        costs = random_costs(seed, K, [(K[e["src"]], K[e["dst"]]) for e in g["edges"]], hi=1000)
        o.set_costs(*costs)
    o.solve()
    pg = pase.Graph(g)
    pg.set_option(pase.OPT_GRAD_SYNC, int(grad))
    pg.set_option(pase.OPT_TRANSFER, int(volume))
    pg.set_option(pase.OPT_HALO, int(halo))
    pg.enumerate_configs(p, all_integers=all_int)
    if costs is not None:
        pg.override_costs(*costs)
    L = [o.layer_costs(v) for v in range(len(K))]
    R = [o.edge_costs(e) for e in range(len(g["edges"]))]
    src = [e["src"] for e in g["edges"]]
    dst = [e["dst"] for e in g["edges"]]
    seq = o.sequence()
    for i, v in enumerate(seq):
        info = pg.vertex_info(v)
        T, _ = o.table(i)
        assert info["table_bound"] >= int(max(T)), (i, v)
        assert info["key_bound"] >= pins.conditioned_qmax(L, R, src, dst, seq, i, K), (i, v)


@pytest.mark.parametrize("name,p,all_int", [("w4_transformer", 64, False),
                                            ("w4_transformer", 24, True),
                                            ("w3_lstm_grid", 32, False)])
def test_workload_keys_fit_fp64(pase, name, p, all_int):
    """The recurrence bounds keep exact fp64 keys ((key_bound + 1) * 2^bits
    <= 2^53) on the full-size workloads, including the Transformer at p = 24
    with every integer split (7.2e11 cells)."""
    pg = pase.Graph(workload(name))
    pg.enumerate_configs(p, all_integers=all_int)
    for v in range(len(pg.K)):
        info = pg.vertex_info(v)
        bits = max(0, (pg.K[v] - 1).bit_length())
        assert (info["key_bound"] + 1) << bits <= 1 << 53, v


@pytest.mark.parametrize("seed", range(12))
def test_bf_order_sequence_and_dependent_sets(pase, seed):
    """PASE_OPT_ORDER = 1: the library's sequence is the oracle's breadth-first
    order and its dependent sets are D_B(i) (eq. 2), for both seq rules."""
    from oracle.oracle import Oracle
    g = random_graph(seed + 40, n=4 + seed % 9, extra_edges=seed % 6, p=4)
    o = Oracle(g)
    o.configs(4)
    o.solve_bf(max_cells=1)
    seq = o.sequence()
    nb = pins.neighbours(len(seq), [e["src"] for e in g["edges"]], [e["dst"] for e in g["edges"]])
    for rule in (0, 1):
        pg = pase.Graph(g, seq_rule=rule)
        pg.set_option(pase.OPT_ORDER, 1)
        pg.enumerate_configs(4)
        assert pg.sequence() == seq
        for i, v in enumerate(seq):
            assert pg.dependent_set(v) == o.dependent_set(i) == pins.bfs_dependent_set(nb, seq, i)


def test_bf_order_option(pase):
    """The order option re-plans an enumerated graph; the dense workloads are
    refused under the breadth-first order (dependent sets of 8 and 19), and
    switching back to GenerateSeq plans them again."""
    P = pase
    pg = P.Graph(workload("w1_residual_cnn"))
    pg.enumerate_configs(8)
    pg.set_option(P.OPT_ORDER, 1)
    assert pg.sequence()[0] == 0
    assert sum(pg.vertex_info(v)["cells"] for v in range(len(pg.K))) == 1_254_456
    for name in ("w2_inception", "w4_transformer"):
        g = workload(name)
        pg = P.Graph(g)
        pg.set_option(P.OPT_ORDER, 1)
        assert _status(lambda: pg.enumerate_configs(g["p"])) == P.TOO_LARGE
        pg.set_option(P.OPT_ORDER, 0)
        pg.enumerate_configs(g["p"])
        assert _status(lambda: pg.set_option(P.OPT_ORDER, 1)) == P.TOO_LARGE
        assert _status(lambda: pg.sequence()) == P.BAD_STATE
    assert _status(lambda: P.pase_set_option(pg.h, P.OPT_ORDER, 2)) == P.INVALID_ARGUMENT


def test_grad_sync_option(pase):
    """PASE_OPT_GRAD_SYNC takes 0 or 1; a weight mask past ndims is refused at
    graph creation; the option raises the layer-cost bound by 2 r W (W0: the
    weight tensors are 65 536 words, so the key bound grows)."""
    P = pase
    pg = P.Graph(fc_chain())
    pg.enumerate_configs(4)
    b0 = pg.vertex_info(3)["key_bound"]
    pg.set_option(P.OPT_GRAD_SYNC, 1)
    pg.enumerate_configs(4)
    assert pg.vertex_info(3)["key_bound"] > b0
    assert _status(lambda: P.pase_set_option(pg.h, P.OPT_GRAD_SYNC, 2)) == P.INVALID_ARGUMENT
    bad = fc_chain()
    bad["vertices"][0]["weight_dims"] = [3]
    with pytest.raises(P.PaseError):
        P.Graph(bad)


def test_transfer_model_option(pase):
    """PASE_OPT_TRANSFER = 1 takes effect at the next enumeration, adds the
    edge matrices (8 bytes per entry) to the workspace, accepts tensor dims
    mapped to one loop dim at small p and refuses them when p^(mapped dims)
    passes 2^32."""
    P = pase
    g = workload("w2_inception")
    pg = P.Graph(g)
    pg.enumerate_configs(16)
    ws0 = pg.workspace_size()
    pg.set_option(P.OPT_TRANSFER, 1)
    assert pg.workspace_size() == ws0
    pg.enumerate_configs(16)
    entries = sum(pg.K[e["src"]] * pg.K[e["dst"]] for e in g["edges"])
    assert pg.workspace_size() >= ws0 + 8 * entries
    assert _status(lambda: P.pase_set_option(pg.h, P.OPT_TRANSFER, 2)) == P.INVALID_ARGUMENT
    dup = {"name": "dup", "p": 4, "comm_weight": 8,
           "vertices": [{"name": "a", "dims": [8, 8], "dim_names": ["x", "y"], "reduce": [],
                         "flops_per_point": 1}] * 2,
           "edges": [{"src": 0, "dst": 1, "src_dim": [0, 0], "dst_dim": [0, 1], "elems": 64}]}
    pg = P.Graph(dup)
    pg.enumerate_configs(4)
    pg.set_option(P.OPT_TRANSFER, 1)
    pg.enumerate_configs(4)                                           # 4^4 <= 2^32
    assert _status(lambda: pg.enumerate_configs(512)) == P.INVALID_ARGUMENT   # 512^4 > 2^32


@pytest.mark.parametrize("seed", range(20))
@pytest.mark.parametrize("rule", [0, 1])
def test_sequence_and_dependent_sets(pase, seed, rule):
    from oracle.oracle import Oracle
    g = random_graph(seed, n=4 + seed % 9, extra_edges=seed % 6, p=4)
    pg = pase.Graph(g, seq_rule=rule)
    pg.enumerate_configs(4)
    o = Oracle(g)
    o.configs(4)
    o.solve(rule=rule, max_cells=1)
    seq = pg.sequence()
    assert seq == o.sequence()
    nb = pins.neighbours(len(seq), [e["src"] for e in g["edges"]], [e["dst"] for e in g["edges"]])
    for i, v in enumerate(seq):
        D = pg.dependent_set(v)
        assert D == o.dependent_set(i) == pins.dependent_set(nb, seq, i)


def test_workload_sequences_match_oracle(pase):
    from oracle.oracle import Oracle
    for name in ("w2_inception", "w3_lstm_grid", "w4_transformer"):
        g = workload(name)
        pg = pase.Graph(g)
        pg.enumerate_configs(g["p"])
        o = Oracle(g)
        o.configs(g["p"])
        o.solve(max_cells=1)
        assert pg.sequence() == o.sequence()
        for i, v in enumerate(o.sequence()):
            assert pg.dependent_set(v) == o.dependent_set(i)


def test_options_validate(pase):
    P = pase
    g = P.Graph(fc_chain())
    g.enumerate_configs(4)
    assert _status(lambda: g.set_option(P.OPT_KERNEL, 2)) == P.INVALID_ARGUMENT
    assert _status(lambda: g.set_option(P.OPT_KEY_TYPE, 3)) == P.INVALID_ARGUMENT
    assert _status(lambda: g.set_option(99, 1)) == P.INVALID_ARGUMENT
    g.set_option(P.OPT_KEEP_TABLES, 1)
    g.set_option(P.OPT_KERNEL, 1)
    assert g.sequence() == [0, 1, 2, 3]
    costs = [np.zeros(10, np.uint64)] * 4
    assert _status(lambda: P.pase_override_costs(g.h, costs, [np.zeros((10, 10), np.uint64)] * 3)) == 0


def test_bulk_lane_plan(pase):
    """Schedule 4 on the Transformer graph: the large fills (>= 8e9 cells) and
    every vertex at a level after them that reads only large fills' chain run
    on the bulk stream (lane 1), all others on the caller's stream (lane 0); a
    threshold above every planned time leaves the bulk stream empty; the
    threshold and the schedule values validate."""
    g = transformer()
    pg = pase.Graph(g)
    pg.set_option(pase.OPT_SCHEDULE, 4)
    pg.enumerate_configs(g["p"])
    info = [pg.vertex_info(v) for v in range(len(g["vertices"]))]
    lanes = [x["lane"] for x in info]
    assert set(lanes) == {0, 1}
    for x in info:
        if x["kernel"] == 1 and x["cells"] >= 8e9:
            assert x["lane"] == 1
    # the Transformer's encoder (the sequence's first vertices) never reads a large fill
    seq = pg.sequence()
    assert all(lanes[v] == 0 for v in seq[:20])
    pg.set_option(pase.OPT_BULK_US, 10 ** 9)
    assert {pg.vertex_info(v)["lane"] for v in range(len(g["vertices"]))} == {0}
    assert _status(lambda: pg.set_option(pase.OPT_BULK_US, 10 ** 9 + 1)) == pase.INVALID_ARGUMENT
    for bad in (2, 3, 6):
        assert _status(lambda: pg.set_option(pase.OPT_SCHEDULE, bad)) == pase.INVALID_ARGUMENT


def test_split_chains_plan(pase):
    """Schedule 5 (the default) on the Transformer graph: level 0 is batched
    on lane 1; after it the large fills (>= 8e9 cells) and their readers run
    on lane 1, the encoder's chain of small vertices on lane 0; level 0's
    small row vertices share the tile shape of its largest fill; a hoisted
    prep (the cross-attention block that reads only a level-1 table) is built
    right after that level on the lane of the table it reads; a threshold
    above every planned time leaves only level 0 on lane 1."""
    g = transformer()
    pg = pase.Graph(g)
    pg.enumerate_configs(g["p"])
    assert pg.plan_check() > 0
    info = [pg.vertex_info(v) for v in range(len(g["vertices"]))]
    lanes = [x["lane"] for x in info]
    assert set(lanes) == {0, 1}
    for x in info:
        if x["level"] == 0 or (x["kernel"] == 1 and x["cells"] >= 8e9):
            assert x["lane"] == 1
    seq = pg.sequence()
    chain = [v for v in seq[:50] if info[v]["level"] >= 1]
    assert len(chain) >= 30 and all(lanes[v] == 0 for v in chain)
    rows0 = [x for x in info if x["level"] == 0 and x["kernel"] == 1 and x["column"] >= 0]
    big = max(rows0, key=lambda x: x["cells"])
    assert {(x["tile_cols"], x["tile_rows"]) for x in rows0} == {(big["tile_cols"], big["tile_rows"])}
    hoisted = [x for x in info if x["prep_after"] >= -1]
    assert len(hoisted) == 1 and hoisted[0]["prep_after"] == 1 and hoisted[0]["level"] > 10
    pg.set_option(pase.OPT_BULK_US, 10 ** 9)
    assert pg.plan_check() > 0
    assert {v for v in range(len(g["vertices"])) if pg.vertex_info(v)["lane"] == 1} == \
        {v for v in range(len(g["vertices"])) if pg.vertex_info(v)["level"] == 0}


# random graphs whose lane plans hoist a prep onto the other lane than its
# vertex's: (seed, n, p, max_dims, extra_edges, max_size, schedule, bulk_us)
CROSS_LANE_PREPS = [(2021, 14, 32, 3, 5, 512, 5, 0), (2021, 14, 32, 3, 5, 512, 4, 0),
                    (2060, 9, 32, 4, 4, 64, 5, 10)]


def cross_lane_graph(pase, case):
    seed, n, p, dims, extra, size, sched, bulk = case
    g = random_graph(seed, n=n, p=p, max_dims=dims, extra_edges=extra, max_size=size)
    pg = pase.Graph(g)
    pg.set_option(pase.OPT_SCHEDULE, sched)
    pg.set_option(pase.OPT_BULK_US, bulk)
    pg.set_option(pase.OPT_HOIST_ELEMS, 1)
    pg.enumerate_configs(p)
    return g, pg


@pytest.mark.parametrize("case", CROSS_LANE_PREPS)
def test_hoisted_prep_on_the_other_lane_plan(pase, case):
    """With lanes, a hoisted prep runs on the lane of the tables its blocks
    read, after their slot: these plans hold such a prep on the other lane than
    its vertex's (both directions over the cases), and the launch plan check
    accepts them (the prep after those fills, the vertex's group waiting for
    that lane at that slot or later)."""
    g, pg = cross_lane_graph(pase, case)
    info = [pg.vertex_info(v) for v in range(len(g["vertices"]))]
    other = [x for x in info if x["prep_after"] >= 0 and x["prep_lane"] != x["lane"]]
    assert other
    for x in other:
        assert x["prep_after"] + 2 <= x["level"]
    assert pg.plan_check() > 0
    pg.close()


def test_level_launch_unification(pase):
    """Level schedule: a level's small column-form row vertices take the tile
    shape of its largest one (so they share its launch) when their fill stays
    small; the sequential schedule plans every vertex on its own."""
    g = transformer()
    shapes = {}
    for sched in (0, 1):
        pg = pase.Graph(g)
        pg.set_option(pase.OPT_SCHEDULE, sched)
        pg.enumerate_configs(g["p"])
        info = [pg.vertex_info(v) for v in range(len(g["vertices"]))]
        rows = [x for x in info if x["kernel"] == 1 and x["column"] >= 0]
        shapes[sched] = rows
        if sched == 0:
            by_level = {}
            for x in rows:
                by_level.setdefault(x["level"], []).append(x)
            # level 0 holds the four largest fills and the small leaves of the
            # encoder and decoder layers: one tile shape for all of them
            lvl0 = by_level[0]
            big = max(lvl0, key=lambda x: x["cells"])
            assert {(x["tile_cols"], x["tile_rows"]) for x in lvl0} == {(big["tile_cols"], big["tile_rows"])}
    distinct0 = {(x["tile_cols"], x["tile_rows"]) for x in shapes[0] if x["level"] == 0}
    distinct1 = {(x["tile_cols"], x["tile_rows"]) for x in shapes[1] if x["level"] == 0}
    assert len(distinct0) < len(distinct1)


@pytest.mark.parametrize("seed", range(4))
def test_key_type_windows(pase, seed):
    """Reading R10 on caller-given costs near a magnitude M: fp64 keys exactly
    while the largest key bound (key_bound + 1) * 2^bits stays within 2^53,
    uint64 keys within 2^64, 128-bit keys beyond while every cost bound fits
    64 bits, and OVERFLOW from pase_override_costs once one does not -- with
    the earlier costs' plan still in force.  128-bit plans run every vertex on
    the generic kernel; key type 2 forces them."""
    import keyedge
    g = random_graph(seed + 1200, n=5 + seed % 3, p=8, max_dims=3, extra_edges=2 + seed % 3)
    pg = pase.Graph(g)
    pg.enumerate_configs(8)
    K = pg.K
    shapes = [(K[e["src"]], K[e["dst"]]) for e in g["edges"]]
    m53 = keyedge.largest_m(pase, pg, seed, K, shapes, lambda kt: kt == 0)
    keyedge.plan_key_type(pase, pg, seed, K, shapes, m53)
    assert keyedge.key_top(pg, K) <= 1 << 53
    assert keyedge.plan_key_type(pase, pg, seed, K, shapes, m53 + 1) == 1
    assert keyedge.key_top(pg, K) > 1 << 53
    m64 = keyedge.largest_m(pase, pg, seed, K, shapes, lambda kt: kt in (0, 1), lo=m53)
    keyedge.plan_key_type(pase, pg, seed, K, shapes, m64)
    assert keyedge.key_top(pg, K) <= 1 << 64
    assert keyedge.plan_key_type(pase, pg, seed, K, shapes, m64 + 1) == 2
    assert all(pg.vertex_info(v)["kernel"] == 0 for v in range(len(K)))
    mov = keyedge.largest_m(pase, pg, seed, K, shapes, lambda kt: kt >= 0, lo=m64)
    assert keyedge.plan_key_type(pase, pg, seed, K, shapes, mov) == 2
    assert all(pg.vertex_info(v)["key_bound"] < (1 << 64) - 1 for v in range(len(K)))
    # one past: OVERFLOW, and the plan of the costs at mov stays
    assert keyedge.plan_key_type(pase, pg, seed, K, shapes, mov + 1) == -1
    assert pg.vertex_info(0)["key_type"] == 2
    assert pg.workspace_size() > 0
    # back to small costs: fp64 keys and the row / direct kernels again
    assert keyedge.plan_key_type(pase, pg, seed, K, shapes, 1000) == 0
    # forced 128-bit keys re-plan on the generic kernel
    pg.set_option(pase.OPT_KEY_TYPE, 2)
    assert pg.vertex_info(0)["key_type"] == 2
    assert all(pg.vertex_info(v)["kernel"] == 0 for v in range(len(K)))
    pg.set_option(pase.OPT_KEY_TYPE, 0)
    assert pg.vertex_info(0)["key_type"] == 0


PLAN_WORKLOADS = ["w0_fc_chain", "w1_residual_cnn", "w2_inception", "w3_lstm_grid", "w4_transformer"]


@pytest.mark.parametrize("name", PLAN_WORKLOADS)
def test_plan_check_workloads(pase, name):
    """The launch descriptors, batches and constant-region image of every
    workload, for each schedule and key type, with and without the direct
    fill and the kept tables: every region write in bounds and every vertex
    filled by one launch (checked on the host, no device work)."""
    g = workload(name)
    pg = pase.Graph(g)
    pg.enumerate_configs(g["p"])
    for sched in (0, 1, 4, 5):
        for key in (0, 1, 2):
            for direct, keep in ((None, 0), (0, 1)):
                if name == "w4_transformer" and (key == 2 or direct == 0):
                    continue   # the generic-only plan of 7e10 cells: covered by the smaller graphs
                pg.set_option(pase.OPT_SCHEDULE, sched)
                pg.set_option(pase.OPT_KEY_TYPE, key)
                if direct is not None:
                    pg.set_option(pase.OPT_DIRECT_CELLS, direct)
                pg.set_option(pase.OPT_KEEP_TABLES, keep)
                assert pg.plan_check() > 0
                assert pg.vertex_info(0)["key_type"] == (key if key else pg.vertex_info(0)["key_type"])


@pytest.mark.parametrize("seed", range(8))
def test_plan_check_random_graphs(pase, seed):
    """Seeded random graphs (2-5 loop dims, sizes up to 4096, p up to 64) and
    caller-given costs: the launch image of every schedule and key type."""
    rng = np.random.default_rng(seed + 40)
    for k in range(6):
        n = int(rng.integers(3, 12))
        p = int(rng.choice([4, 8, 16, 32, 64]))
        g = random_graph(seed * 100 + k + 7000, n=n, p=p, max_dims=int(rng.integers(2, 6)),
                         extra_edges=int(rng.integers(0, 6)), max_size=int(rng.choice([8, 64, 512, 4096])))
        pg = pase.Graph(g)
        pg.enumerate_configs(p)
        for sched in (0, 1, 4, 5):
            pg.set_option(pase.OPT_SCHEDULE, sched)
            for key in (0, 2):
                pg.set_option(pase.OPT_KEY_TYPE, key)
                assert pg.plan_check() > 0
        K = pg.K
        costs = random_costs(seed + k, K, [(K[e["src"]], K[e["dst"]]) for e in g["edges"]], hi=1 << 20)
        pg.override_costs(*costs)
        assert pg.plan_check() > 0


def test_halo_option_and_geometry(pase):
    """PASE_OPT_HALO validates; a halo on a dim that is not an input dim, or an
    input dim out of range, is refused at creation; the option changes the
    key bounds (the layer costs) only for graphs with a halo."""
    P = pase
    g = fc_chain()
    pg = P.Graph(g)
    assert _status(lambda: pg.set_option(P.OPT_HALO, 2)) == P.INVALID_ARGUMENT
    bad = dict(g["vertices"][0], halo=[0, 1, 0], input_dims=[0, 2])
    assert _status(lambda: P.pase_graph_create([bad] + g["vertices"][1:], g["edges"])) == P.INVALID_ARGUMENT
    bad = dict(g["vertices"][0], halo=[0, 0, 0], input_dims=[3])
    assert _status(lambda: P.pase_graph_create([bad] + g["vertices"][1:], g["edges"])) == P.INVALID_ARGUMENT
    for name, changes in (("w0_fc_chain", False), ("w1_residual_cnn", True)):
        w = workload(name)
        bounds = []
        for halo in (0, 1):
            pg = P.Graph(w)
            pg.set_option(P.OPT_HALO, halo)
            pg.enumerate_configs(w["p"])
            bounds.append([pg.vertex_info(v)["key_bound"] for v in range(len(w["vertices"]))])
        assert (bounds[0] != bounds[1]) == changes, name


def _oracle_for(g, p, all_int=False):
    from oracle.oracle import Oracle
    o = Oracle(g)
    o.configs(p, all_integers=all_int)   # the assignment needs the configurations only
    return o


@pytest.mark.parametrize("seed", range(16))
def test_assign_devices_match_oracle(pase, seed):
    """Device assignment of random strategies on random graphs (several tensor
    dims on one loop dim, unsplit dims, parallel edges; p = 4, 8, 16 with
    power-of-two splits, p = 6 with every integer split): devices, edge
    localities and transfers equal the oracle's, entry by entry."""
    P = pase
    rng = np.random.default_rng(seed + 500)
    all_int = seed % 4 == 3
    p = 6 if all_int else [4, 8, 16][seed % 3]
    g = random_graph(seed + 40, int(rng.integers(2, 9)), p=p, extra_edges=int(rng.integers(0, 4)))
    o = _oracle_for(g, p, all_int)
    pg = P.Graph(g)
    pg.enumerate_configs(p, all_integers=all_int)
    assert pg.K == [int(k) for k in o.K]
    for trial in range(4):
        strat = [int(rng.integers(0, k)) for k in pg.K]
        dev, loc, xfer = pg.assign_devices(strat)
        odev, oloc, oxfer = o.assign_devices(strat)
        assert np.array_equal(dev, odev), (trial, strat)
        assert np.array_equal(loc, oloc) and np.array_equal(xfer, oxfer), (trial, strat)


@pytest.mark.parametrize("name", ["w0_fc_chain", "w1_residual_cnn", "w2_inception", "w4_transformer"])
def test_assign_devices_workload_strategies(pase, name):
    """The assignment of each workload's optimal strategy (the stored expected
    strategy) equals the oracle's; an edge's locality never exceeds its tensor,
    and on the FC chain (every vertex data parallel) the assignment is the
    identity with zero transfer."""
    import json
    P = pase
    g = workload(name)
    gold = json.load(open(os.path.join(ROOT, "tests", "golden", f"{name}_seed0.json")))
    strat = gold["strategy"]
    o = _oracle_for(g, g["p"])
    pg = P.Graph(g)
    pg.enumerate_configs(g["p"])
    dev, loc, xfer = pg.assign_devices(strat)
    odev, oloc, oxfer = o.assign_devices(strat)
    assert np.array_equal(dev, odev) and np.array_equal(loc, oloc) and np.array_equal(xfer, oxfer)
    assert all(int(loc[e]) <= ed["elems"] for e, ed in enumerate(g["edges"]))
    if name == "w0_fc_chain":
        assert (dev == np.arange(g["p"])).all() and not xfer.any()


def test_assign_devices_errors(pase):
    """Call order, bad strategies and the p bound of the assignment."""
    P = pase
    g = fc_chain()
    pg = P.Graph(g)
    assert _status(lambda: P.pase_assign_devices(pg.h, [0] * pg.nv, pg.nv, pg.ne, 4)) == P.BAD_STATE
    pg.enumerate_configs(4)
    assert _status(lambda: pg.assign_devices([pg.K[0]] + [0] * (pg.nv - 1))) == P.INVALID_ARGUMENT
    assert P.load().pase_assign_devices(pg.h, None, None, None, None) == P.INVALID_ARGUMENT
    pg.enumerate_configs(2048)
    assert _status(lambda: pg.assign_devices([0] * pg.nv)) == P.TOO_LARGE


def test_fused_minimum_plan(pase):
    """PASE_OPT_FUSED_MIN: on the measured Transformer the plan fuses the
    minimum of the last cross-attention key/value projection into its
    predecessor's fill (producer flagged 1, reader 2, adjacent in the order,
    the producer's column digit being the reader); the option validates,
    turns it off and on, and the launch plan checks in every schedule."""
    P = pase
    g = workload("w4_transformer")
    pg = P.Graph(g)
    assert _status(lambda: pg.set_option(P.OPT_FUSED_MIN, 2)) == P.INVALID_ARGUMENT
    pg.enumerate_configs(g["p"])
    info = {v: pg.vertex_info(v) for v in range(pg.nv)}
    prod = [v for v in info if info[v]["fused"] == 1]
    read = [v for v in info if info[v]["fused"] == 2]
    assert len(prod) == 1 and len(read) == 1
    a, b = info[prod[0]], info[read[0]]
    assert b["position"] == a["position"] + 1 and a["column"] == read[0] and b["column"] == -1
    assert a["splits"] == 1 and b["splits"] == 1 and a["outer"] == 1 and a["rows"] == b["rows"]
    for sched in (0, 1, 4, 5):
        for keep in (0, 1):
            pg.set_option(P.OPT_SCHEDULE, sched)
            pg.set_option(P.OPT_KEEP_TABLES, keep)
            assert pg.plan_check() > 0
    pg.set_option(P.OPT_FUSED_MIN, 0)
    assert not any(pg.vertex_info(v)["fused"] for v in range(pg.nv))
    assert pg.plan_check() > 0
    pg.set_option(P.OPT_FUSED_MIN, 1)
    assert sum(pg.vertex_info(v)["fused"] for v in range(pg.nv)) == 3


def test_hoisted_prep_plan(pase):
    """PASE_OPT_HOIST_ELEMS: on the measured Transformer the one large prep
    whose blocks read only an early table (the fourth decoder layer's
    cross-attention key/value projection, level 43, reading level-1 tables)
    is hoisted to start after a slot in [1, 41] (the one before the longest
    planned fill of that window); 0 hoists nothing; the sequential schedule
    never hoists; the launch plan checks either way."""
    P = pase
    g = workload("w4_transformer")
    pg = P.Graph(g)
    pg.enumerate_configs(g["p"])
    h = {v: pg.vertex_info(v) for v in range(pg.nv) if pg.vertex_info(v)["prep_after"] >= -1}
    assert len(h) == 1
    (v, info), = h.items()
    assert g["vertices"][v]["name"] == "dec4_xkv" and 1 <= info["prep_after"] <= 41 and info["level"] == 43
    assert pg.plan_check() > 0
    pg.set_option(P.OPT_HOIST_ELEMS, 0)
    assert all(pg.vertex_info(v)["prep_after"] == -2 for v in range(pg.nv))
    pg.set_option(P.OPT_HOIST_ELEMS, 1)
    assert sum(pg.vertex_info(v)["prep_after"] >= -1 for v in range(pg.nv)) >= 1
    assert pg.plan_check() > 0
    pg.set_option(P.OPT_SCHEDULE, 1)
    assert all(pg.vertex_info(v)["prep_after"] == -2 for v in range(pg.nv))
    assert pg.plan_check() > 0
