"""The dataflow schedule, checked on the host: for every workload and for
random graphs, the segments built for the one-launch search are simulated
with the kernel's worker protocol (two ticket queues, dependency waits) for
many worker counts and random item durations.  Every item must run, none
before its dependencies, and the workers must never deadlock -- the property
the device launch relies on to terminate."""
import pytest

from workloads import random_graph, workload


@pytest.fixture(scope="module")
def P():
    from paper_2407_04001_amd import pase
    pase.load()
    return pase


def _graph(P, g, p=None, schedule=3):
    pg = P.Graph(g)
    pg.set_option(P.OPT_SCHEDULE, schedule)
    pg.enumerate_configs(p or g["p"])
    return pg


@pytest.mark.parametrize("name", ["w0_fc_chain", "w1_residual_cnn", "w2_inception", "w3_lstm_grid",
                                  "w4_transformer"])
def test_workload_schedules_drain(P, name):
    g = workload(name)
    pg = _graph(P, g)
    for workers, lat in [(2, 1), (3, 1), (3, 2), (17, 2), (64, 8), (2048, 256)]:
        for seed in range(3):
            items = pg.flow_check(workers, lat, seed)
            assert items > 0


@pytest.mark.parametrize("seed", range(12))
def test_random_graph_schedules_drain(P, seed):
    g = random_graph(seed, n=3 + seed % 7)
    pg = _graph(P, g, p=4)
    for workers, lat in [(2, 1), (5, 1), (5, 4), (40, 5)]:
        pg.flow_check(workers, lat, seed)


def test_flow_check_arguments(P):
    g = workload("w0_fc_chain")
    pg = _graph(P, g)
    for workers, lat in [(1, 1), (4, 0), (4, 4)]:
        with pytest.raises(P.PaseError):
            pg.flow_check(workers, lat)
    other = _graph(P, g, schedule=2)
    with pytest.raises(P.PaseError, match="BAD_STATE"):
        other.flow_check(4, 1)
