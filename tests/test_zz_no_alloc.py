"""The allocation-free search (pase_find_best_strategy_noalloc) against the
ordinary entry point, through the C ABI: on two calls in a row, the second
with a smaller graph, the minimum, the strategy and every DP table
(fingerprints, and every entry of the small graph's tables) agree; a search
larger than the static workspace is refused before any device work."""
import numpy as np
import pytest

from workloads import random_graph, workload

pytestmark = pytest.mark.gpu


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


def _tables(P, pg, g):
    """Fingerprints of every table, and every entry of tables up to 512 entries."""
    out = {}
    for v in range(len(g["vertices"])):
        fp = pg.fingerprint(v)
        entries = []
        D = pg.dependent_set(v)
        n = int(np.prod([pg.K[w] for w in D])) if D else 1
        if n <= 512:
            for idx in range(n):
                cfg, x = [], idx
                for w in reversed(D):
                    cfg.append(x % pg.K[w])
                    x //= pg.K[w]
                cfg.reverse()
                entries.append(pg.table_entry(v, cfg))
        out[v] = (fp, entries)
    return out


def _both(P, g, p, schedule=0, direct=None, options=()):
    """The same graph through both entry points (two handles); returns
    (result, tables, handle) of each.  direct: PASE_OPT_DIRECT_CELLS (0 keeps
    small vertices on the prep + row / generic kernels and their scratch);
    options: further (option, value) pairs."""
    res = []
    for noalloc in (False, True):
        pg = P.Graph(g)
        pg.set_option(P.OPT_SCHEDULE, schedule)
        if direct is not None:
            pg.set_option(P.OPT_DIRECT_CELLS, direct)
        for opt, val in options:
            pg.set_option(opt, val)
        pg.enumerate_configs(p)
        pg.set_option(P.OPT_KEEP_TABLES, 1)
        assert pg.workspace_size() <= P.NOALLOC_WORKSPACE_BYTES
        if noalloc:
            r = P.pase_find_best_strategy_noalloc(pg.h, pg.nv)
        else:
            r = pg.find_best_strategy()
        res.append((r, _tables(P, pg, g), pg))
    return res


def test_noalloc_matches_the_allocating_search(P):
    big = workload("w2_inception")          # ~13 MB of workspace
    small = workload("w1_residual_cnn")     # ~1 MB: the second call has the smaller input
    for name, g in (("w2_inception", big), ("w1_residual_cnn", small)):
        say(f"noalloc vs allocating: {name}")
        (r0, t0, _), (r1, t1, pg1) = _both(P, g, g["p"])
        assert r1 == r0, name
        assert t1 == t0, name
        assert pg1.stats()["workspace_bytes"] <= P.NOALLOC_WORKSPACE_BYTES


def test_noalloc_random_graphs_and_schedules(P):
    """Random graphs in a row (each second one smaller), every table entry
    compared, with and without the direct fill (so the prep blocks and split
    scratch live in the array too); the bulk lane plan runs level by level in
    the static array."""
    for seed, n, sched, direct in ((901, 11, 0, 0), (902, 6, 0, 0), (901, 11, 0, None), (903, 9, 4, 0),
                                   (902, 6, 4, None)):
        g = random_graph(seed, n=n, p=16, max_dims=3, extra_edges=3, max_size=512)
        say(f"noalloc random graph seed={seed} n={n} schedule={sched} direct={direct}")
        (r0, t0, _), (r1, t1, pg1) = _both(P, g, 16, schedule=sched, direct=direct)
        assert r1 == r0
        assert t1 == t0
        # the same handle again: the array keeps the last call's contents, a
        # repeated call overwrites them with the same answer
        assert P.pase_find_best_strategy_noalloc(pg1.h, pg1.nv) == r0
        assert _tables(P, pg1, g) == t0


def test_noalloc_refuses_a_search_larger_than_the_array(P):
    g = workload("w4_transformer")
    pg = P.Graph(g)
    pg.enumerate_configs(g["p"])
    assert pg.workspace_size() > P.NOALLOC_WORKSPACE_BYTES
    with pytest.raises(P.PaseError) as e:
        P.pase_find_best_strategy_noalloc(pg.h, pg.nv)
    assert e.value.status == P.TOO_LARGE
    assert "allocation-free workspace" in str(e.value)
    # the handle stays usable through the ordinary entry point
    mc, _ = pg.find_best_strategy()
    assert mc == 146_670_616_576


def test_noalloc_fused_minimum_and_hoisted_preps(P):
    """A Transformer (one encoder, two decoder layers, p = 16) with a fused
    minimum and, with every eligible prep hoisted, side-stream preps in the
    allocating search -- which the allocation-free one builds in their own
    slots: both agree on every table."""
    from workloads import transformer
    g = transformer(p=16, enc_layers=1, dec_layers=2)
    say("noalloc vs allocating: fused minimum, hoisted preps")
    (r0, t0, pg0), (r1, t1, _) = _both(P, g, 16, options=((P.OPT_HOIST_ELEMS, 1),))
    assert any(pg0.vertex_info(v)["fused"] for v in range(pg0.nv))
    assert any(pg0.vertex_info(v)["prep_after"] >= -1 for v in range(pg0.nv))
    assert r1 == r0
    assert t1 == t0
