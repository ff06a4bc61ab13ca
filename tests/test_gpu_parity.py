"""GPU parity: the HIP search against the CPU oracle, bit for bit.

Costs are integers and ties break to the lowest configuration index, so every
compared quantity must be identical: minimum cost, strategy, vertex order,
dependent sets, every table entry (small graphs, element by element), table
fingerprints and sampled entries (full-size workloads, against the oracle's
committed golden files), and the device cost tables.
"""
import json
import os

import numpy as np
import pytest

from workloads import chain_graph, random_costs, random_graph, workload

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


@pytest.fixture(scope="module")
def P():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2407_04001_amd import pase
    pase.load()
    return pase


def say(*a):
    print(*a, flush=True)


def _oracle(g, p=None, costs=None, rule=0, all_integers=False, bf=False, volume=False, grad=False, halo=False):
    from oracle.oracle import Oracle
    o = Oracle(g)
    o.configs(p or g["p"], all_integers=all_integers, volume=volume, grad_sync=grad, halo=halo)
    if costs is not None:
        o.set_costs(*costs)
    if bf:
        o.solve_bf(threads=os.cpu_count() or 1)
    else:
        o.solve(rule=rule, threads=os.cpu_count() or 1)
    return o


def _compare_all_entries(pg, o, g, max_entries=2048):
    """Every entry of every table element by element (tables up to
    `max_entries` entries; larger ones on a seeded sample of that many), plus
    the fingerprints of every table."""
    K = pg.K
    rng = np.random.default_rng(7)
    for i, v in enumerate(o.sequence()):
        D = o.dependent_set(i)
        assert pg.dependent_set(v) == D
        T, A = o.table(i)
        idxs = range(len(T)) if len(T) <= max_entries else rng.integers(0, len(T), max_entries)
        for idx in idxs:
            idx = int(idx)
            cfg, x = [], idx
            for w in reversed(D):
                cfg.append(x % K[w])
                x //= K[w]
            cfg.reverse()
            got = pg.table_entry(v, cfg)
            assert got == (int(T[idx]), int(A[idx])), (v, cfg)
        assert pg.fingerprint(v) == o.fingerprint(i)


def _run(P, g, p=None, keep=True, kernel=0, key=0, costs=None, rule=0, schedule=0, tile=(0, 0),
         parts=0, splits=0, all_integers=False, bf=False, volume=False, grad=False,
         direct=0, bulk_us=None, halo=False, fuse=None):
    """direct: PASE_OPT_DIRECT_CELLS (0 = off, so the tests aimed at the row and
    generic kernels keep them; None = the library's default)."""
    pg = P.Graph(g, seq_rule=rule)
    if direct is not None:
        pg.set_option(P.OPT_DIRECT_CELLS, direct)
    pg.set_option(P.OPT_ORDER, int(bf))
    pg.set_option(P.OPT_TRANSFER, int(volume))
    pg.set_option(P.OPT_GRAD_SYNC, int(grad))
    pg.set_option(P.OPT_HALO, int(halo))
    pg.enumerate_configs(p or g["p"], all_integers=all_integers)
    pg.set_option(P.OPT_KEEP_TABLES, int(keep))
    pg.set_option(P.OPT_KERNEL, kernel)
    pg.set_option(P.OPT_KEY_TYPE, key)
    pg.set_option(P.OPT_SCHEDULE, schedule)
    pg.set_option(P.OPT_TILE_COLS, tile[0])
    pg.set_option(P.OPT_TILE_ROWS, tile[1])
    pg.set_option(P.OPT_TILE_PARTS, parts)
    pg.set_option(P.OPT_C_SPLITS, splits)
    if bulk_us is not None:
        pg.set_option(P.OPT_BULK_US, bulk_us)
    if fuse is not None:
        pg.set_option(P.OPT_FUSED_MIN, int(fuse))
    if costs is not None:
        pg.override_costs(*costs)
    mc, strat = pg.find_best_strategy()
    return pg, mc, strat


# ------------------------------------------------------------------ small graphs, every entry
@pytest.mark.parametrize("kernel,key", [(0, 0), (1, 0), (0, 1), (1, 1)])
def test_fc_chain_closed_form(P, kernel, key):
    say(f"fc_chain kernel={kernel} key={key}")
    g = workload("w0_fc_chain")
    pg, mc, strat = _run(P, g, kernel=kernel, key=key)
    assert (mc, strat) == (8_388_608, [9, 9, 9, 9])
    _compare_all_entries(pg, _oracle(g), g)


@pytest.mark.parametrize("seed", range(10))
@pytest.mark.parametrize("key", [0, 1])
def test_random_graphs_random_costs(P, seed, key):
    """Dense ties (costs in [0,4)) exercise the lowest-index tie-break."""
    g = random_graph(seed + 200, n=4 + seed % 6, p=8, max_dims=3, extra_edges=1 + seed % 4)
    say(f"random graph seed={seed + 200} key={key}")
    o0 = _oracle(g)
    K = [int(k) for k in o0.K]
    costs = random_costs(seed, K, [(K[e["src"]], K[e["dst"]]) for e in g["edges"]], hi=4)
    o = _oracle(g, costs=costs)
    pg, mc, strat = _run(P, g, key=key, costs=costs)
    assert (mc, strat) == o.result()
    _compare_all_entries(pg, o, g)


@pytest.mark.parametrize("seed", range(8))
def test_random_graphs_model_costs(P, seed):
    g = random_graph(seed + 300, n=5 + seed % 5, p=16, max_dims=3, extra_edges=seed % 5,
                     max_size=512)
    say(f"random graph model costs seed={seed + 300}")
    o = _oracle(g)
    pg, mc, strat = _run(P, g)
    assert (mc, strat) == o.result()
    _compare_all_entries(pg, o, g)
    for v in range(len(g["vertices"])):
        assert np.array_equal(pg.layer_costs(v), o.layer_costs(v))
    for e in range(len(g["edges"])):
        assert np.array_equal(pg.edge_costs(e), o.edge_costs(e))


@pytest.mark.parametrize("seed", range(6))
def test_random_graphs_bulk_lane_schedule(P, seed):
    """Bulk lane schedule on small random graphs, every row-kernel vertex on
    the bulk stream (threshold 0): every table entry against the oracle."""
    g = random_graph(seed + 300, n=5 + seed % 5, p=16, max_dims=3, extra_edges=seed % 5,
                     max_size=512)
    say(f"random graph bulk lane seed={seed + 300}")
    o = _oracle(g)
    pg, mc, strat = _run(P, g, schedule=4, bulk_us=0)
    assert pg.stats()["schedule"] == 4
    assert (mc, strat) == o.result()
    _compare_all_entries(pg, o, g)


# every form of the row kernel: columns x rows per lane, fp64 and uint64 keys
TILES = [(8, 1), (8, 2), (12, 1), (12, 2), (14, 1), (14, 2), (16, 1), (16, 2), (24, 1), (24, 2),
         (28, 1), (28, 2)]


# (seed, n, extra edges, max dims): together these give row-kernel vertices
# with 1, 2, 3 and 4 row terms, with and without a column digit
TILE_GRAPHS = [(600, 8, 6, 3), (600, 10, 10, 2), (600, 9, 8, 3), (601, 8, 6, 3), (601, 9, 8, 3),
               (661, 10, 10, 2)]


@pytest.mark.parametrize("tile", TILES, ids=[f"{a}x{b}" for a, b in TILES])
def test_forced_row_tiles(P, tile):
    """Each tile form on graphs whose vertices take the row kernel with one to
    four row terms, split and unsplit c ranges, and on ties (random costs)."""
    used = 0
    for seed, n, extra, dims in TILE_GRAPHS:
        g = random_graph(seed, n=n, p=16, max_dims=dims, extra_edges=extra, max_size=256)
        o = _oracle(g)
        for key in (0, 1):
            say(f"tile {tile} random graph seed={seed} n={n} key={key}")
            pg, mc, strat = _run(P, g, key=key, tile=tile)
            assert (mc, strat) == o.result()
            _compare_all_entries(pg, o, g, max_entries=256)
            used += pg.stats()["rows_vertices"]
        K = [int(k) for k in o.K]
        costs = random_costs(seed, K, [(K[e["src"]], K[e["dst"]]) for e in g["edges"]], hi=4)
        ot = _oracle(g, costs=costs)
        say(f"tile {tile} random graph seed={seed} n={n} tied costs")
        pg, mc, strat = _run(P, g, costs=costs, tile=tile)
        assert (mc, strat) == ot.result()
        _compare_all_entries(pg, ot, g, max_entries=256)
    assert used > 0


@pytest.mark.parametrize("parts,splits", [(1, 2), (2, 1), (2, 3), (4, 1), (4, 5), (4, 64)],
                         ids=["p1s2", "p2s1", "p2s3", "p4s1", "p4s5", "p4s64"])
def test_forced_parts_and_splits(P, parts, splits):
    """c ranges shared by the waves of a workgroup (merged through LDS) and by
    workgroups (partial keys and a reduction launch), including empty parts
    (more parts or splits than values of c)."""
    for tile in [(16, 1), (14, 2), (28, 1)]:
        for seed, n, extra, dims in TILE_GRAPHS:
            g = random_graph(seed, n=n, p=16, max_dims=dims, extra_edges=extra, max_size=256)
            o = _oracle(g)
            for key in (0, 1):
                say(f"parts {parts} splits {splits} tile {tile} graph seed={seed} n={n} key={key}")
                pg, mc, strat = _run(P, g, key=key, tile=tile, parts=parts, splits=splits)
                assert (mc, strat) == o.result()
                _compare_all_entries(pg, o, g, max_entries=128)


@pytest.mark.parametrize("tile", [(8, 1), (16, 1), (16, 2), (28, 1), (28, 2)],
                         ids=["8x1", "16x1", "16x2", "28x1", "28x2"])
def test_forced_row_tiles_against_golden(P, tile):
    for name in ("w2_inception", "w4_transformer"):
        _check_golden(P, name, 0, tile=tile)


@pytest.mark.parametrize("seed", range(4))
def test_chains(P, seed):
    g = chain_graph(seed, n=6 + seed, p=32, max_dims=3)
    say(f"chain seed={seed}")
    o = _oracle(g)
    pg, mc, strat = _run(P, g)
    assert (mc, strat) == o.result()
    _compare_all_entries(pg, o, g)


def test_long_chain_back_substitution(P):
    """More positions than the level-parallel back-substitution's one
    workgroup takes (1024): the search falls back to the sequential walk."""
    for n in (1024, 1100):
        g = chain_graph(5, n=n, p=4, max_dims=2)
        say(f"long chain n={n}")
        o = _oracle(g)
        pg, mc, strat = _run(P, g, keep=False)
        assert (mc, strat) == o.result()


def test_edge_cases(P):
    # one vertex, no edges: the minimum layer cost
    g = {"name": "one", "p": 8, "comm_weight": 8, "edges": [],
         "vertices": [{"name": "v", "dims": [5, 7, 3], "dim_names": list("abc"), "reduce": [1],
                       "flops_per_point": 3}]}
    say("edge case: single vertex")
    o = _oracle(g)
    pg, mc, strat = _run(P, g)
    assert (mc, strat) == o.result()
    # p = 1: a single configuration everywhere
    g = random_graph(11, n=6, p=1, extra_edges=3)
    say("edge case: p=1")
    o = _oracle(g, p=1)
    pg, mc, strat = _run(P, g, p=1)
    assert (mc, strat) == o.result() and set(strat) == {0}
    # parallel edges and the printed GenerateSeq rule
    g = random_graph(3, n=5, p=4, extra_edges=6, multi_edges=True)
    for rule in (0, 1):
        say(f"edge case: multigraph rule={rule}")
        o = _oracle(g, rule=rule)
        pg, mc, strat = _run(P, g, rule=rule)
        assert pg.sequence() == o.sequence()
        assert (mc, strat) == o.result()
        _compare_all_entries(pg, o, g)


def test_repeat_and_reenumerate(P):
    g = workload("w1_residual_cnn")
    say("repeat + re-enumerate")
    pg = P.Graph(g)
    results = []
    for p in (8, 4, 8):
        pg.enumerate_configs(p)
        results.append(pg.find_best_strategy())
        results.append(pg.find_best_strategy())
        assert results[-1] == results[-2]
    assert results[0] == results[4]
    assert results[2] == _oracle(g, p=4).result()


@pytest.mark.parametrize("name", ["w1_residual_cnn", "w2_inception"])
def test_model_costs_after_override(P, name):
    # model costs -> caller-given costs (the model's doubled) -> model costs
    # again on one graph and workspace.  The model's cost tables are computed
    # on the device; the two workloads put them below (W1, 27 KiB) and above
    # (W2, 353 KiB) the size from which the search leaves them out of its
    # host-to-device upload.  Doubling every cost keeps every argmin, so the
    # strategy is unchanged and the minimum doubles.
    g = workload(name)
    say(f"model / override / model costs: {name}")
    pg = P.Graph(g)
    pg.enumerate_configs(g["p"])
    mc0, s0 = pg.find_best_strategy()
    layer = [pg.layer_costs(v) for v in range(len(g["vertices"]))]
    edge = [pg.edge_costs(e) for e in range(len(g["edges"]))]
    pg.override_costs([2 * np.asarray(a, np.uint64) for a in layer], [2 * np.asarray(a, np.uint64) for a in edge])
    mc1, s1 = pg.find_best_strategy()
    assert mc1 == 2 * mc0 and s1 == s0
    assert np.array_equal(pg.layer_costs(0), 2 * np.asarray(layer[0], np.uint64))
    pg.enumerate_configs(g["p"])
    assert pg.find_best_strategy() == (mc0, s0)
    for v in range(len(g["vertices"])):
        assert np.array_equal(pg.layer_costs(v), layer[v])


def test_library_owned_workspace(P):
    g = workload("w1_residual_cnn", 1)
    say("library-owned workspace")
    pg = P.Graph(g)
    pg.enumerate_configs(g["p"])
    mc, strat = pg.find_best_strategy(torch_workspace=False)
    assert (mc, strat) == _oracle(g).result()
    assert pg.stats()["slots"] < len(g["vertices"])


# ------------------------------------------------------------------ full-size workloads
def _golden(name, seed, p=None, all_integers=False, bf=False, volume=False, grad=False, halo=False):
    if halo:
        fn = f"{name}_seed{seed}_{'grad_' if grad else ''}halo.json"
    elif bf:
        fn = f"{name}_seed{seed}_p{p}_bf.json"
    elif volume:
        fn = f"{name}_seed{seed}_volume.json"
    elif grad:
        fn = f"{name}_seed{seed}_grad.json"
    else:
        fn = f"{name}_seed{seed}_p{p}_all.json" if all_integers else f"{name}_seed{seed}.json"
    with open(os.path.join(GOLDEN, fn)) as f:
        return json.load(f)


def _check_golden(P, name, seed, kernel=0, key=0, keep=True, samples=True, schedule=0, tile=(0, 0),
                  p=None, all_integers=False, bf=False, volume=False, grad=False, direct=None,
                  bulk_us=None, halo=False):
    gold = _golden(name, seed, p, all_integers, bf, volume, grad, halo)
    g = workload(name, seed)
    say(f"{name} seed={seed} kernel={kernel} key={key} keep={keep} schedule={schedule} tile={tile} "
        f"p={p} all_integers={all_integers} bf={bf} volume={volume} grad={grad} direct={direct}")
    pg, mc, strat = _run(P, g, p=p, keep=keep, kernel=kernel, key=key, schedule=schedule, tile=tile,
                         all_integers=all_integers, bf=bf, volume=volume, grad=grad,
                         direct=direct, bulk_us=bulk_us, halo=halo)
    st = pg.stats()
    say(f"   cells {st['cells']:.3e}  wall {st['wall_ms']:.1f} ms  key_type {st['key_type']} "
        f"rows_vertices {st['rows_vertices']} slots {st['slots']} launches {st['launches']} "
        f"schedule {st['schedule']}")
    assert pg.K == gold["num_configs"]
    assert pg.sequence() == gold["sequence"]
    assert st["cells"] == gold["cells"]
    assert mc == int(gold["min_cost"])
    assert strat == gold["strategy"]
    if not keep:
        return
    K = gold["num_configs"]
    for tb in gold["tables"]:
        v = tb["vertex"]
        assert pg.dependent_set(v) == tb["dep"]
        assert pg.fingerprint(v) == (int(tb["fp_cost"]), int(tb["fp_arg"])), v
        if samples:
            for idx, t, a in tb["samples"]:
                cfg, x = [], idx
                for w in reversed(tb["dep"]):
                    cfg.append(x % K[w])
                    x //= K[w]
                cfg.reverse()
                assert pg.table_entry(v, cfg) == (int(t), a), (v, idx)


@pytest.mark.parametrize("name,seed", [("w0_fc_chain", 0), ("w1_residual_cnn", 0),
                                       ("w1_residual_cnn", 1), ("w1_residual_cnn", 2),
                                       ("w2_inception", 0), ("w2_inception", 1),
                                       ("w2_inception", 2), ("w3_lstm_grid", 0)])
def test_workloads_against_golden(P, name, seed):
    """Default plan (small vertices on the direct fill), then without it."""
    _check_golden(P, name, seed)
    _check_golden(P, name, seed, direct=0)


@pytest.mark.parametrize("name", ["w2_inception", "w3_lstm_grid"])
def test_generic_and_u64_paths_against_golden(P, name):
    _check_golden(P, name, 0, kernel=1)
    _check_golden(P, name, 0, key=1)


@pytest.mark.parametrize("name", ["w1_residual_cnn", "w2_inception", "w3_lstm_grid", "w4_transformer"])
def test_sequential_schedule_against_golden(P, name):
    """One vertex per launch slot, in sequence order, gives the same answer."""
    _check_golden(P, name, 0, keep=False, schedule=1)


@pytest.mark.parametrize("name", ["w1_residual_cnn", "w2_inception", "w3_lstm_grid", "w4_transformer"])
def test_bulk_lane_schedule_against_golden(P, name):
    """Large fills on a stream of their own, every other vertex level by
    level on a second one: the same answer as the level schedule, with the
    default threshold and with every row-kernel vertex on the bulk stream."""
    _check_golden(P, name, 0, keep=False, schedule=4)
    _check_golden(P, name, 0, keep=True, samples=False, schedule=4)
    _check_golden(P, name, 0, keep=True, samples=False, schedule=4, bulk_us=0)


@pytest.mark.parametrize("name", ["w1_residual_cnn", "w2_inception", "w3_lstm_grid", "w4_transformer"])
def test_split_chains_schedule_against_golden(P, name):
    """Level 0 batched, then the small vertices' chain on one stream and the
    large fills with their readers on another: the same answer as the level
    schedule, with the default threshold and with every row-kernel vertex
    large (then only the generic and direct fills form the chain)."""
    _check_golden(P, name, 0, keep=False, schedule=5)
    _check_golden(P, name, 0, keep=True, samples=False, schedule=5)
    _check_golden(P, name, 0, keep=True, samples=False, schedule=5, bulk_us=0)


@pytest.mark.parametrize("case", [(2021, 14, 32, 3, 5, 512, 5, 0), (2021, 14, 32, 3, 5, 512, 4, 0),
                                  (2060, 9, 32, 4, 4, 64, 5, 10)])
def test_hoisted_prep_on_the_other_lane(P, case):
    """A hoisted prep that runs on the lane of the tables it reads, not on its
    vertex's (each direction over the cases): the minimum, the strategy and
    every table entry match the oracle."""
    seed, n, p, dims, extra, size, sched, bulk = case
    g = random_graph(seed, n=n, p=p, max_dims=dims, extra_edges=extra, max_size=size)
    say(f"cross-lane hoisted prep seed={seed} schedule={sched} bulk_us={bulk}")
    o = _oracle(g)
    pg = P.Graph(g)
    pg.set_option(P.OPT_SCHEDULE, sched)
    pg.set_option(P.OPT_BULK_US, bulk)
    pg.set_option(P.OPT_HOIST_ELEMS, 1)
    pg.set_option(P.OPT_KEEP_TABLES, 1)
    pg.enumerate_configs(p)
    info = [pg.vertex_info(v) for v in range(len(g["vertices"]))]
    assert any(x["prep_after"] >= 0 and x["prep_lane"] != x["lane"] for x in info)
    mc, strat = pg.find_best_strategy()
    assert pg.stats()["schedule"] == sched
    assert (mc, strat) == o.result()
    _compare_all_entries(pg, o, g, max_entries=2048)


def test_bulk_lane_assignment(P):
    """The Transformer's large fills and every vertex reading their tables run
    on the bulk stream; no vertex of the other stream reads a bulk table."""
    g = workload("w4_transformer")
    pg, _, _ = _run(P, g, keep=False, schedule=4)
    assert pg.stats()["schedule"] == 4
    info = {v: pg.vertex_info(v) for v in range(len(g["vertices"]))}
    bulk = {v for v, x in info.items() if x["lane"] == 1}
    assert bulk and len(bulk) < len(info)
    assert all(x["lane"] in (0, 1) for x in info.values())
    for v, x in info.items():
        if x["kernel"] == 1 and x["cells"] >= 8e9:
            assert v in bulk, v


def test_workloads_run_the_requested_schedule(P):
    """The workloads fit the resident layout: every schedule runs as requested,
    and the bulk lane puts the Transformer's large fills on the bulk stream."""
    for name in ("w1_residual_cnn", "w2_inception", "w3_lstm_grid", "w4_transformer"):
        g = workload(name)
        for sched in (0, 1, 4, 5):
            pg, _, _ = _run(P, g, keep=False, schedule=sched)
            assert pg.stats()["schedule"] == sched, (name, sched)
    lanes = [pg.vertex_info(v)["lane"] for v in range(len(g["vertices"]))]
    assert 0 < sum(1 for x in lanes if x) < len(lanes)


@pytest.mark.skip(reason="captured HIP-graph replay of the search was removed: its first GPU run "
                         "ended in a host segmentation fault inside pase_find_best_strategy (W2, first "
                         "capture) whose cause was not found; the search now uses direct launches")
@pytest.mark.parametrize("name", ["w2_inception", "w4_transformer"])
def test_graph_replays_match_direct_launches(P, name):
    """The captured HIP graph is replayed several times, with unrelated eager
    GPU work and synchronisations in between; every replay must equal the
    result of direct launches (and the oracle's)."""
    import torch
    gold = _golden(name, 0)
    g = workload(name)
    say(f"graph replays {name}")
    _, mc0, st0 = _run(P, g, keep=False)
    assert (mc0, st0) == (int(gold["min_cost"]), gold["strategy"])
    pg = P.Graph(g)
    for rep in range(4):
        pg.enumerate_configs(g["p"])
        mc, st = pg.find_best_strategy()
        x = torch.randn(512, 512, device="cuda")
        (x @ x).sum().item()
        torch.cuda.synchronize()
        assert (mc, st) == (mc0, st0), rep
    # a different plan (other p) forces a new capture; going back replays again
    pg.enumerate_configs(g["p"] // 2)
    pg.find_best_strategy()
    pg.enumerate_configs(g["p"])
    assert pg.find_best_strategy() == (mc0, st0)


def test_transformer_p64_against_golden(P):
    """The measured workload at full size, in the configuration the benchmark
    times (default kernels and memory plan), then with every table kept and
    fingerprinted, and without the direct fill."""
    _check_golden(P, "w4_transformer", 0, keep=False)
    _check_golden(P, "w4_transformer", 0, keep=True)
    _check_golden(P, "w4_transformer", 0, keep=True, samples=False, direct=0)


def test_cost_tables_against_oracle(P):
    for name in ("w0_fc_chain", "w1_residual_cnn", "w2_inception"):
        g = workload(name)
        say(f"cost tables {name}")
        from oracle.oracle import Oracle
        o = Oracle(g)
        o.configs(g["p"])
        pg, _, _ = _run(P, g, keep=False)
        for v in range(len(g["vertices"])):
            assert np.array_equal(pg.layer_costs(v), o.layer_costs(v)), v
        for e in range(len(g["edges"])):
            assert np.array_equal(pg.edge_costs(e), o.edge_costs(e)), e


# ------------------------------------------------------------------ every integer split
@pytest.mark.parametrize("seed", range(8))
@pytest.mark.parametrize("key", [0, 1])
def test_all_integer_random_graphs(P, seed, key):
    """Sec. II's full configuration set (factors 3, 5, 6, 7 ... ): the result,
    every table entry and the device cost tables equal the oracle's."""
    p = (3, 5, 6, 7, 12, 12, 24, 10)[seed]
    g = random_graph(seed + 700, n=4 + seed % 5, p=p, max_dims=3, extra_edges=1 + seed % 4,
                     max_size=300)
    say(f"every-integer random graph seed={seed + 700} p={p} key={key}")
    o = _oracle(g, p=p, all_integers=True)
    pg, mc, strat = _run(P, g, p=p, key=key, all_integers=True)
    assert pg.K == [int(k) for k in o.K]
    assert (mc, strat) == o.result()
    _compare_all_entries(pg, o, g, max_entries=1024)
    for v in range(len(g["vertices"])):
        assert np.array_equal(pg.layer_costs(v), o.layer_costs(v)), v
    for e in range(len(g["edges"])):
        assert np.array_equal(pg.edge_costs(e), o.edge_costs(e)), e


@pytest.mark.parametrize("seed", range(4))
def test_all_integer_tied_costs_and_kernels(P, seed):
    """Dense ties with every integer split, on the row kernel at two tile
    forms and on the generic kernel."""
    g = random_graph(seed + 720, n=5 + seed, p=12, max_dims=3, extra_edges=2 + seed)
    o0 = _oracle(g, p=12, all_integers=True)
    K = [int(k) for k in o0.K]
    costs = random_costs(seed, K, [(K[e["src"]], K[e["dst"]]) for e in g["edges"]], hi=4)
    o = _oracle(g, p=12, costs=costs, all_integers=True)
    for kernel, tile in ((0, (0, 0)), (0, (8, 2)), (0, (28, 1)), (1, (0, 0))):
        say(f"every-integer tied costs seed={seed + 720} kernel={kernel} tile={tile}")
        pg, mc, strat = _run(P, g, p=12, costs=costs, kernel=kernel, tile=tile, all_integers=True)
        assert (mc, strat) == o.result()
        _compare_all_entries(pg, o, g, max_entries=512)


def test_all_integer_edge_cases(P):
    """p = 1 (one configuration), a prime p, and the largest p (255) with
    one- and two-dim vertices."""
    for p, seed, dims in ((1, 730, 3), (7, 731, 3), (255, 732, 1), (255, 733, 2)):
        g = random_graph(seed, n=4, p=p, max_dims=dims, extra_edges=1, max_size=1000)
        say(f"every-integer edge case p={p} seed={seed} dims<={dims}")
        o = _oracle(g, p=p, all_integers=True)
        pg, mc, strat = _run(P, g, p=p, all_integers=True)
        assert (mc, strat) == o.result()
        if p == 1:
            assert set(strat) == {0}
        for e in range(len(g["edges"])):
            assert np.array_equal(pg.edge_costs(e), o.edge_costs(e)), e


@pytest.mark.parametrize("name", ["w0_fc_chain", "w2_inception"])
def test_all_integer_workloads_against_golden(P, name):
    """Full-size workloads at p = 12 with every integer split, against the
    oracle's stored results: default plan, generic kernel, uint64 keys, and
    the sequential and bulk lane schedules."""
    _check_golden(P, name, 0, p=12, all_integers=True)
    if name == "w2_inception":
        _check_golden(P, name, 0, p=12, all_integers=True, kernel=1)
        _check_golden(P, name, 0, p=12, all_integers=True, key=1)
        for sched in (1, 4, 5):
            _check_golden(P, name, 0, p=12, all_integers=True, keep=False, schedule=sched)


def test_all_integer_transformer_p12_against_golden(P):
    _check_golden(P, "w4_transformer", 0, p=12, all_integers=True, keep=False)
    _check_golden(P, "w4_transformer", 0, p=12, all_integers=True, keep=True)


def test_all_integer_transformer_p24_properties(P):
    """Beyond the oracle's reach in a test (7.2e11 cells): the returned
    strategy costs the returned minimum under the oracle's cost tables, the
    level and sequential schedules and both key types agree, and the minimum
    is at most the p = 12 optimum (every p = 12 configuration is a p = 24 one)."""
    from oracle.oracle import Oracle
    g = workload("w4_transformer", 0)
    say("every-integer transformer p=24 level schedule")
    pg, mc, strat = _run(P, g, p=24, keep=False, all_integers=True)
    say(f"   cells {pg.stats()['cells']:.3e} wall {pg.stats()['wall_ms']:.1f} ms")
    say("every-integer transformer p=24 sequential schedule, uint64 keys")
    _, mc1, strat1 = _run(P, g, p=24, keep=False, schedule=1, key=1, all_integers=True)
    assert (mc1, strat1) == (mc, strat)
    assert mc <= int(_golden("w4_transformer", 0, 12, True)["min_cost"])
    o = Oracle(g)
    o.configs(24, all_integers=True)
    L = [o.layer_costs(v) for v in range(len(g["vertices"]))]
    src = [e["src"] for e in g["edges"]]
    dst = [e["dst"] for e in g["edges"]]
    tot = sum(int(L[v][c]) for v, c in enumerate(strat))
    for e in range(len(src)):
        tot += int(o.edge_costs(e)[strat[src[e]], strat[dst[e]]])
    assert tot == mc


# ------------------------------------------------------------------ breadth-first recurrence (eq. 2)
@pytest.mark.parametrize("seed", range(8))
@pytest.mark.parametrize("key", [0, 1])
def test_bf_order_random_graphs(P, seed, key):
    """PASE_OPT_ORDER = 1 against the oracle's literal eq. (2): sequence,
    D_B sets, every table entry, minimum and strategy; model costs, and dense
    ties on odd seeds."""
    g = random_graph(seed + 540, n=4 + seed % 5, p=8, max_dims=3, extra_edges=1 + seed % 3)
    costs = None
    if seed % 2:
        o0 = _oracle(g)
        K = [int(k) for k in o0.K]
        costs = random_costs(seed, K, [(K[e["src"]], K[e["dst"]]) for e in g["edges"]], hi=4)
    say(f"breadth-first random graph seed={seed + 540} key={key} ties={costs is not None}")
    o = _oracle(g, costs=costs, bf=True)
    pg, mc, strat = _run(P, g, key=key, costs=costs, bf=True)
    assert pg.sequence() == o.sequence()
    assert (mc, strat) == o.result()
    _compare_all_entries(pg, o, g, max_entries=1024)


def test_bf_order_kernels_and_schedules(P):
    """The breadth-first chain of tables on the generic kernel, uint64 keys
    and the sequential and bulk lane schedules: the same answer."""
    g = random_graph(560, n=9, p=16, max_dims=3, extra_edges=3, max_size=256)
    o = _oracle(g, bf=True)
    for kw in ({}, {"kernel": 1}, {"key": 1}, {"schedule": 1}, {"schedule": 4, "bulk_us": 0}, {"schedule": 5},
               {"schedule": 5, "bulk_us": 0}):
        say(f"breadth-first seed=560 {kw}")
        pg, mc, strat = _run(P, g, bf=True, **kw)
        assert (mc, strat) == o.result()
        _compare_all_entries(pg, o, g, max_entries=256)


def test_bf_order_workloads(P):
    """W0 and the residual CNN (three seeds) under the breadth-first order
    against the oracle's eq. (2), every table fingerprinted; the residual CNN
    at p = 64 (6.9e8 cells) against the stored golden."""
    for name, seed in (("w0_fc_chain", 0), ("w1_residual_cnn", 0), ("w1_residual_cnn", 1),
                       ("w1_residual_cnn", 2)):
        g = workload(name, seed)
        say(f"breadth-first {name} seed={seed}")
        o = _oracle(g, bf=True)
        pg, mc, strat = _run(P, g, bf=True)
        assert pg.sequence() == o.sequence()
        assert (mc, strat) == o.result()
        for i, v in enumerate(o.sequence()):
            assert pg.fingerprint(v) == o.fingerprint(i)
    _check_golden(P, "w1_residual_cnn", 0, p=64, bf=True, keep=False)
    _check_golden(P, "w1_residual_cnn", 0, p=64, bf=True, keep=True)


# ------------------------------------------------------------------ volume-intersection transfer model
@pytest.mark.parametrize("seed", range(8))
def test_volume_model_random_graphs(P, seed):
    """PASE_OPT_TRANSFER = 1: the device-computed edge matrices equal the
    oracle's cell-counting ones entry for entry (mismatched dim sizes,
    unmapped dims, both configuration sets), and so do the search and every
    table entry."""
    p, all_int = ((4, False), (8, False), (6, True), (16, False), (12, True), (5, True), (8, False),
                  (2, False))[seed]
    g = random_graph(seed + 600, n=4 + seed % 4, p=p, max_dims=3, extra_edges=1 + seed % 3, max_size=200)
    say(f"volume model random graph seed={seed + 600} p={p} all_integers={all_int}")
    o = _oracle(g, p=p, all_integers=all_int, volume=True)
    pg, mc, strat = _run(P, g, p=p, all_integers=all_int, volume=True)
    for e in range(len(g["edges"])):
        assert np.array_equal(pg.edge_costs(e), o.edge_costs(e)), e
    assert (mc, strat) == o.result()
    _compare_all_entries(pg, o, g, max_entries=512)


def test_volume_model_large_tensors(P):
    """Tensors of ~2^53 words at p = 64 (Q up to 4096, so elems * f passes
    2^64): the device's split ceil division (no 128-bit products) against the
    oracle's 128-bit one; uint64 keys."""
    vs = [{"name": f"v{k}", "dims": [1 << 20, 3 << 18, 7], "dim_names": ["a", "b", "c"], "reduce": [2],
           "flops_per_point": 1} for k in range(3)]
    big = (1 << 53) - 12345
    es = [{"src": 0, "dst": 1, "src_dim": [0, 1], "dst_dim": [1, 0], "elems": big},
          {"src": 1, "dst": 2, "src_dim": [1, -1], "dst_dim": [0, 2], "elems": big - 999},
          {"src": 0, "dst": 2, "src_dim": [2], "dst_dim": [1], "elems": 3 ** 33}]
    g = {"name": "big", "p": 64, "comm_weight": 1, "vertices": vs, "edges": es}
    for p, all_int in ((64, False), (12, True)):
        say(f"volume model large tensors p={p}")
        o = _oracle(g, p=p, all_integers=all_int, volume=True)
        pg, mc, strat = _run(P, g, p=p, all_integers=all_int, volume=True, key=1)
        for e in range(len(es)):
            assert np.array_equal(pg.edge_costs(e), o.edge_costs(e)), e
        assert (mc, strat) == o.result()


@pytest.mark.parametrize("name", ["w1_residual_cnn", "w2_inception", "w3_lstm_grid"])
def test_volume_model_workloads_against_golden(P, name):
    _check_golden(P, name, 0, volume=True)
    _check_golden(P, name, 0, volume=True, keep=False, schedule=4)


def test_volume_model_transformer_against_golden(P):
    """The measured Transformer with volume transfer costs, in the benchmark's
    configuration and with every table kept and fingerprinted."""
    _check_golden(P, "w4_transformer", 0, volume=True, keep=False)
    _check_golden(P, "w4_transformer", 0, volume=True, keep=True)


# ------------------------------------------------------------------ fused minimum (PASE_OPT_FUSED_MIN)
def _fused_graph():
    """A Transformer with one encoder and two decoder layers at p = 16 (4.1e8
    cells): its last cross-attention key/value projection takes a minimum
    over the whole table of its predecessor, which the plan fuses."""
    from workloads import transformer
    return transformer(p=16, enc_layers=1, dec_layers=2)


@pytest.mark.parametrize("schedule,key", [(0, 0), (1, 0), (4, 0), (5, 0), (0, 1), (5, 1)])
def test_fused_minimum_every_entry(P, schedule, key):
    """The fused producer/reader pair against the oracle entry by entry (every
    table, with tables kept so the producer also writes its own), under each
    schedule and both 64-bit key types; and the same search with fusion off."""
    g = _fused_graph()
    say(f"fused minimum schedule={schedule} key={key}")
    o = _oracle(g)
    pg, mc, strat = _run(P, g, schedule=schedule, key=key, direct=None, bulk_us=5)
    fused = [v for v in range(pg.nv) if pg.vertex_info(v)["fused"]]
    assert len(fused) == 2, fused
    assert (mc, strat) == o.result()
    _compare_all_entries(pg, o, g, max_entries=4096)
    pg2, mc2, strat2 = _run(P, g, schedule=schedule, key=key, direct=None, bulk_us=5, fuse=False)
    assert not any(pg2.vertex_info(v)["fused"] for v in range(pg2.nv))
    assert (mc2, strat2) == (mc, strat)


@pytest.mark.parametrize("key", [0, 1])
def test_hoisted_preps_every_entry(P, key):
    """Every eligible prep hoisted to the side stream (PASE_OPT_HOIST_ELEMS =
    1) on the fused graph: every table against the oracle, and the same
    result with hoisting off."""
    g = _fused_graph()
    say(f"hoisted preps key={key}")
    o = _oracle(g)
    pg = P.Graph(g)
    pg.set_option(P.OPT_HOIST_ELEMS, 1)
    pg.set_option(P.OPT_KEY_TYPE, key)
    pg.enumerate_configs(16)
    pg.set_option(P.OPT_KEEP_TABLES, 1)
    hoisted = [v for v in range(pg.nv) if pg.vertex_info(v)["prep_after"] >= -1]
    assert hoisted
    mc, strat = pg.find_best_strategy()
    assert (mc, strat) == o.result()
    _compare_all_entries(pg, o, g, max_entries=4096)
    pg.set_option(P.OPT_HOIST_ELEMS, 0)
    assert not any(pg.vertex_info(v)["prep_after"] >= -1 for v in range(pg.nv))
    assert pg.find_best_strategy() == (mc, strat)


@pytest.mark.parametrize("seed", range(3))
def test_fused_minimum_random_costs(P, seed):
    """Caller-given costs in [0, 4) on the fused graph (dense ties: the atomic
    minimum must still keep the lowest configuration), tables kept and not."""
    g = _fused_graph()
    say(f"fused minimum random costs seed={seed}")
    o0 = _oracle(g)
    K = [int(k) for k in o0.K]
    shapes = [(K[e["src"]], K[e["dst"]]) for e in g["edges"]]
    costs = random_costs(seed + 900, K, shapes, hi=4)
    o = _oracle(g, costs=costs)
    pg, mc, strat = _run(P, g, costs=costs, direct=None)
    assert any(pg.vertex_info(v)["fused"] == 2 for v in range(pg.nv))
    assert (mc, strat) == o.result()
    _compare_all_entries(pg, o, g, max_entries=4096)
    pg2, mc2, strat2 = _run(P, g, costs=costs, keep=False, direct=None)
    assert (mc2, strat2) == o.result()


# ------------------------------------------------------------------ device assignment of the found strategy
@pytest.mark.parametrize("name,seed", [("random", 0), ("random", 1), ("random", 2), ("w1_residual_cnn", 0),
                                       ("w2_inception", 0), ("w4_transformer", 0)])
def test_assign_devices_after_search(P, name, seed):
    """The strategy the GPU search returns, placed on devices by
    pase_assign_devices: devices, localities and transfers equal the oracle's
    assignment of the oracle's own optimum (the same strategy); where both
    ends of an edge keep the grid numbering, the transfer equals the device's
    volume-model matrix entry."""
    if name == "random":
        p = (4, 8, 16)[seed]
        g = random_graph(seed + 720, n=5 + seed, p=p, max_dims=3, extra_edges=2, max_size=200)
        volume = True
    else:
        g = workload(name, seed)
        p, volume = g["p"], name != "w4_transformer"
    say(f"device assignment after search {name} seed={seed} p={p} volume={volume}")
    if name == "random":
        o = _oracle(g, p=p, volume=True)
        want = o.result()
    else:
        gold = _golden(name, seed, volume=volume)
        want = (int(gold["min_cost"]), gold["strategy"])
        from oracle.oracle import Oracle
        o = Oracle(g)
        o.configs(p)
    pg, mc, strat = _run(P, g, p=p, keep=False, volume=volume)
    assert (mc, strat) == want
    dev, loc, xfer = pg.assign_devices(strat)
    odev, oloc, oxfer = o.assign_devices(want[1])
    assert np.array_equal(dev, odev) and np.array_equal(loc, oloc) and np.array_equal(xfer, oxfer)
    assert pg.stats()["assign_ms"] > 0
    if volume:
        def grid(w):
            n = int((dev[w] >= 0).sum())
            return dev[w].tolist() == list(range(n)) + [-1] * (p - n)
        for e, ed in enumerate(g["edges"]):
            u, v = ed["src"], ed["dst"]
            if grid(u) and grid(v):
                assert int(xfer[e]) == int(pg.edge_costs(e)[strat[u], strat[v]]), e


# ------------------------------------------------------------------ weight-gradient all-reduce
@pytest.mark.parametrize("seed", range(8))
def test_grad_sync_random_graphs(P, seed):
    """PASE_OPT_GRAD_SYNC = 1 on random graphs with random weight tensors: the
    device layer costs equal the oracle's, and so do the search and every
    table entry (both configuration sets, with and without volume costs)."""
    p, all_int, volume = ((4, False, False), (8, False, False), (6, True, False), (16, False, True),
                          (12, True, True), (32, False, False), (5, True, False), (2, False, True))[seed]
    g = random_graph(seed + 640, n=4 + seed % 4, p=p, max_dims=3, extra_edges=1 + seed % 3, max_size=300)
    say(f"gradient term random graph seed={seed + 640} p={p} all_integers={all_int} volume={volume}")
    o = _oracle(g, p=p, all_integers=all_int, volume=volume, grad=True)
    pg, mc, strat = _run(P, g, p=p, all_integers=all_int, volume=volume, grad=True)
    for v in range(len(g["vertices"])):
        assert np.array_equal(pg.layer_costs(v), o.layer_costs(v)), v
    assert (mc, strat) == o.result()
    _compare_all_entries(pg, o, g, max_entries=512)


# ------------------------------------------------------------------ halo exchange of convolutions
def _halo_graph(seed, **kw):
    """The first random graph from seed on with at least two haloed layers."""
    while True:
        g = random_graph(seed, **kw)
        if sum(1 for v in g["vertices"] if any(v.get("halo", []))) >= 2:
            return g
        seed += 1000


@pytest.mark.parametrize("seed", range(8))
def test_halo_random_graphs(P, seed):
    """PASE_OPT_HALO = 1 on random graphs with random convolution geometry:
    the device layer costs equal the oracle's, and so do the search and every
    table entry (both configuration sets, with the gradient term on some)."""
    p, all_int, grad = ((4, False, False), (8, False, True), (6, True, False), (16, False, False),
                        (12, True, True), (32, False, False), (5, True, False), (64, False, True))[seed]
    g = _halo_graph(seed + 1500, n=4 + seed % 4, p=p, max_dims=5, extra_edges=1 + seed % 3, max_size=300)
    say(f"halo term random graph p={p} all_integers={all_int} grad={grad}")
    o = _oracle(g, p=p, all_integers=all_int, grad=grad, halo=True)
    for direct in (None, 0):
        pg, mc, strat = _run(P, g, p=p, all_integers=all_int, grad=grad, halo=True, direct=direct)
        for v in range(len(g["vertices"])):
            assert np.array_equal(pg.layer_costs(v), o.layer_costs(v)), v
        assert (mc, strat) == o.result()
        _compare_all_entries(pg, o, g, max_entries=512)


@pytest.mark.parametrize("name", ["w1_residual_cnn", "w2_inception"])
@pytest.mark.parametrize("grad", [False, True])
def test_halo_workloads_against_golden(P, name, grad):
    _check_golden(P, name, 0, halo=True, grad=grad)
    _check_golden(P, name, 0, halo=True, grad=grad, keep=False, direct=0)


def test_grad_sync_fc_chain(P):
    """W0 with the gradient term: 8 486 912, every layer split 4 ways over out."""
    g = workload("w0_fc_chain")
    pg, mc, strat = _run(P, g, grad=True)
    assert mc == 8_486_912
    assert [pg.config_splits(v, c) for v, c in enumerate(strat)] == [[1, 4, 1]] * 4


@pytest.mark.parametrize("name", ["w1_residual_cnn", "w2_inception", "w3_lstm_grid"])
def test_grad_sync_workloads_against_golden(P, name):
    _check_golden(P, name, 0, grad=True)


def test_grad_sync_transformer_against_golden(P):
    _check_golden(P, "w4_transformer", 0, grad=True, keep=False)
    _check_golden(P, "w4_transformer", 0, grad=True, keep=True)


# ------------------------------------------------------------------ direct fill
ALL_DIRECT = 1 << 62


@pytest.mark.parametrize("seed", range(10))
@pytest.mark.parametrize("key", [0, 1])
def test_direct_fill_random_graphs(P, seed, key):
    """Every vertex on the direct fill (each term summed per cell from its
    source arrays): every table entry equals the oracle's, with model costs,
    dense ties (odd seeds), volume transfer costs and the gradient term."""
    g = random_graph(seed + 660, n=4 + seed % 6, p=8, max_dims=3, extra_edges=1 + seed % 4)
    volume, grad = seed % 3 == 2, seed % 4 == 3
    costs = None
    if seed % 2:
        o0 = _oracle(g)
        K = [int(k) for k in o0.K]
        costs = random_costs(seed, K, [(K[e["src"]], K[e["dst"]]) for e in g["edges"]], hi=4)
    say(f"direct fill random graph seed={seed + 660} key={key} ties={costs is not None} volume={volume} grad={grad}")
    o = _oracle(g, costs=costs, volume=volume, grad=grad)
    pg, mc, strat = _run(P, g, key=key, costs=costs, volume=volume, grad=grad, direct=ALL_DIRECT)
    assert all(pg.vertex_info(v)["kernel"] == 2 for v in range(len(g["vertices"])))
    assert (mc, strat) == o.result()
    _compare_all_entries(pg, o, g, max_entries=1024)


def test_direct_fill_schedules_and_orders(P):
    """The direct fill under the level, sequential and bulk lane schedules,
    the breadth-first order and every-integer configurations; the generic-only
    kernel mode does not use it."""
    g = random_graph(680, n=9, p=16, max_dims=3, extra_edges=4, max_size=256)
    o = _oracle(g)
    for sched in (0, 1, 4, 5):
        say(f"direct fill seed=680 schedule={sched}")
        pg, mc, strat = _run(P, g, schedule=sched, direct=ALL_DIRECT)
        assert (mc, strat) == o.result()
        _compare_all_entries(pg, o, g, max_entries=256)
    pg, mc, strat = _run(P, g, kernel=1, direct=ALL_DIRECT)
    assert (mc, strat) == o.result()
    assert all(pg.vertex_info(v)["kernel"] != 2 for v in range(len(g["vertices"])))
    ob = _oracle(g, bf=True)
    pg, mc, strat = _run(P, g, bf=True, direct=ALL_DIRECT)
    assert (mc, strat) == ob.result()
    _compare_all_entries(pg, ob, g, max_entries=256)
    oa = _oracle(g, p=12, all_integers=True)
    pg, mc, strat = _run(P, g, p=12, all_integers=True, direct=ALL_DIRECT)
    assert (mc, strat) == oa.result()


@pytest.mark.parametrize("name", ["w1_residual_cnn", "w2_inception", "w3_lstm_grid"])
def test_direct_fill_whole_workloads(P, name):
    """Every vertex of a workload on the direct fill, against the golden."""
    _check_golden(P, name, 0, direct=ALL_DIRECT)


# ------------------------------------------------------------------ key types at their edges (R10)
@pytest.mark.parametrize("seed", range(3))
def test_key_type_edges(P, seed):
    """Caller-given costs near a magnitude M (dense ties), placed so that the
    largest key bound sits just under 2^53 (fp64 keys), just over it (uint64),
    just under 2^64 (uint64), just over it (128-bit keys), and at the largest M
    whose cost bounds still fit 64 bits (128-bit keys, table values past
    2^63): every table entry against the oracle with the same costs.  The
    largest table value shifted by its position's argmin bits -- a key the
    fill formed -- lies within 1% of the edge, so the fp64 arithmetic runs
    next to 2^53 and the uint64 keys next to 2^64."""
    import keyedge
    g = random_graph(seed + 1200, n=5 + seed % 3, p=8, max_dims=3, extra_edges=2 + seed % 3)
    pg0 = P.Graph(g)
    pg0.enumerate_configs(8)
    K = pg0.K
    shapes = [(K[e["src"]], K[e["dst"]]) for e in g["edges"]]
    m53 = keyedge.largest_m(P, pg0, seed, K, shapes, lambda kt: kt == 0)
    m64 = keyedge.largest_m(P, pg0, seed, K, shapes, lambda kt: kt in (0, 1), lo=m53)
    mov = keyedge.largest_m(P, pg0, seed, K, shapes, lambda kt: kt >= 0, lo=m64)
    for M, kt, edge in ((m53, 0, 2 ** 53), (m53 + 1, 1, 2 ** 53), (m64, 1, 2 ** 64), (m64 + 1, 2, 2 ** 64),
                        (mov, 2, None)):
        say(f"key edge seed={seed + 1200} M={M} key_type={kt}")
        costs = keyedge.near_costs(seed, K, shapes, M)
        o = _oracle(g, costs=costs)
        for direct in (None, 0):
            pg, mc, strat = _run(P, g, costs=costs, direct=direct)
            assert pg.stats()["key_type"] == kt
            assert (mc, strat) == o.result()
            _compare_all_entries(pg, o, g)
        top = max(int(max(o.table(i)[0])) << max(0, (int(K[v]) - 1).bit_length())
                  for i, v in enumerate(o.sequence()))
        if edge is not None:
            assert 0.99 * edge < top <= edge * 1.01, (M, kt, top)
        else:
            assert max(int(max(o.table(i)[0])) for i in range(len(K))) > 2 ** 63


@pytest.mark.parametrize("seed", range(6))
def test_forced_wide_keys_random_costs(P, seed):
    """128-bit keys forced (PASE_OPT_KEY_TYPE 2) on random graphs with dense
    ties: prep + generic fill in 16-byte keys, every entry against the oracle."""
    g = random_graph(seed + 1300, n=4 + seed % 6, p=8, max_dims=3, extra_edges=1 + seed % 4)
    say(f"forced 128-bit keys seed={seed + 1300}")
    o0 = _oracle(g)
    K = [int(k) for k in o0.K]
    costs = random_costs(seed, K, [(K[e["src"]], K[e["dst"]]) for e in g["edges"]], hi=4)
    o = _oracle(g, costs=costs)
    pg, mc, strat = _run(P, g, key=2, costs=costs, direct=None)
    assert pg.stats()["key_type"] == 2
    assert (mc, strat) == o.result()
    _compare_all_entries(pg, o, g)
    pg, mc, strat = _run(P, g, key=2)
    assert pg.stats()["key_type"] == 2
    assert (mc, strat) == o0.result()
    _compare_all_entries(pg, o0, g)


@pytest.mark.parametrize("name", ["w1_residual_cnn", "w2_inception"])
def test_forced_wide_keys_against_golden(P, name):
    _check_golden(P, name, 0, key=2)


@pytest.mark.parametrize("block", range(4))
def test_random_graph_sweep_schedules(P, block):
    """Seeded sweep over random graphs (4-13 vertices, 2-5 loop dims, p from 4
    to 64, sizes up to 4096): the level schedule (shared level launches), the
    bulk lane with every row vertex on the bulk stream, the split chains
    schedule, the sequential schedule and the level schedule without the
    direct fill all give the oracle's minimum, strategy and every table
    (fingerprints).  No graph is
    refused: those whose packed keys pass 64 bits run on 128-bit keys."""
    checked = 0
    wide = 0
    for seed in range(block * 20, block * 20 + 20):
        rng = np.random.default_rng(seed)
        n = int(rng.integers(4, 14))
        p = int(rng.choice([4, 8, 16, 32, 64]))
        g = random_graph(seed + 5000, n=n, p=p, max_dims=int(rng.integers(2, 6)),
                         extra_edges=int(rng.integers(0, 6)), max_size=int(rng.choice([8, 64, 512, 4096])))
        say(f"random sweep seed={seed + 5000} n={n} p={p}")
        o = _oracle(g)
        fps = [o.fingerprint(i) for i in range(len(o.sequence()))]
        for sched, bulk, direct in ((0, None, None), (4, 0, None), (5, 0, None), (1, None, 0), (0, None, 0)):
            pg = P.Graph(g)
            pg.set_option(P.OPT_SCHEDULE, sched)
            if bulk is not None:
                pg.set_option(P.OPT_BULK_US, bulk)
            if direct is not None:
                pg.set_option(P.OPT_DIRECT_CELLS, direct)
            pg.set_option(P.OPT_KEEP_TABLES, 1)
            pg.enumerate_configs(p)
            mc, strat = pg.find_best_strategy()
            assert (mc, strat) == o.result(), (seed, sched)
            for i, v in enumerate(o.sequence()):
                assert pg.fingerprint(v) == fps[i], (seed, sched, v)
            checked += 1
            wide += pg.stats()["key_type"] == 2
    assert checked == 100
    say(f"   {wide} runs on 128-bit keys")
