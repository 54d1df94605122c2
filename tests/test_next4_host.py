"""Host-side checks of the richer collectives and latency (no GPU): the
library's tree and hierarchical all-reduce decompositions are the oracle's
flow for flow (sources, destinations, bytes, lags, routes and dependency
lists, in order) on three fabrics, alone, after other operations and with
per-rank streams; latency settings are validated and every bad call
appends nothing."""

import numpy as np
import pytest

from oracle import flows as oflows
from oracle import timeline as otl
from workloads import configs
from workloads.program import Hier, MiB, Program, Ring, Scenario, Send, Topology, Tree, gbit
from workloads.trace import Collective, Compute, Trace

from paper_2505_01616_amd import netsim as ns
from paper_2505_01616_amd import program as prog
from paper_2505_01616_amd import trace as ptr

from tests.test_lib_host import _compare


def _fabrics():
    yield Topology(kind="leaf_spine", servers=8, gpus_per_server=8, servers_per_leaf=2, spines=4,
                   nvlink_Bps=900e9, nic_Bps=gbit(400), fabric_Bps=gbit(800), ecmp_seed=17,
                   fabric_latency_s=1e-6, nvlink_latency_s=2e-7)
    yield Topology(kind="rail", servers=8, gpus_per_server=8, servers_per_leaf=4, spines=4,
                   nvlink_Bps=900e9, nic_Bps=gbit(400), fabric_Bps=gbit(400), ecmp_seed=3)
    yield configs.c3_topology(7)


@pytest.mark.parametrize("k", [0, 1, 2])
def test_tree_and_hier_bit_exact(k):
    topo = list(_fabrics())[k]
    rng = np.random.default_rng(k)
    sc = Scenario(topo)
    for p in (2, 3, 7, 16, 37):
        sc.add(Tree(rng.permutation(topo.endpoints)[:p].astype(np.int32), 24 * MiB,
                    lag=float(rng.random() * 1e-5)))
    for m, g in ((4, 8), (3, 1), (1, 5), (2, 2), (5, 3)):
        r = rng.permutation(topo.endpoints)[:m * g].reshape(m, g).astype(np.int32)
        sc.add(Hier(r, 40 * MiB, lag=1e-6, after=(len(sc.ops) - 1,)))
    sc.add(Send(0, topo.endpoints - 1, MiB, after=(len(sc.ops) - 1, (2, 5))))
    sc.add(Tree(np.arange(10, dtype=np.int32), 8 * MiB, after=(len(sc.ops) - 1,)))
    sc.add(Ring("allreduce", np.arange(12, dtype=np.int32), 12 * MiB, after=(len(sc.ops) - 1, 5)))
    _compare(Program("next4", [sc]))


def test_streams_tree_and_hier_match_the_oracle():
    from tests.test_trace_host import _compare as compare_trace
    topo = next(_fabrics())
    tr = Trace("next4 streams", topo)
    tr.add(Compute(3, 1e-4))
    a = tr.add(Collective("tree_allreduce", np.arange(9, dtype=np.int32), np.arange(9) * 2, 16 * MiB))
    r = np.arange(24, dtype=np.int32).reshape(3, 8)
    tr.add(Collective("hier_allreduce", r, r.astype(np.int64) * 2 + 1, 48 * MiB))
    tr.add(Compute(4, 2e-5, wait=[(a, 4)]))
    tr.add(Collective("hier_allreduce", r[:, :1].copy(), (r[:, :1] * 2).astype(np.int64), MiB))
    compare_trace(tr)


def test_latency_and_collective_errors_append_nothing():
    keep = []
    topo = next(_fabrics())
    h = ns.netsim_create_topology([prog.topology_struct(topo, keep)])
    try:
        before = ns.netsim_counts(h)
        bad = [
            lambda: ns.netsim_add_tree_allreduce(h, 0, [5], MiB),
            lambda: ns.netsim_add_tree_allreduce(h, 0, [5, 5], MiB),
            lambda: ns.netsim_add_tree_allreduce(h, 0, [5, 9999], MiB),
            lambda: ns.netsim_add_tree_allreduce(h, 0, [1, 2], -1.0),
            lambda: ns.netsim_add_hier_allreduce(h, 0, np.zeros((1, 1), np.int32), MiB),
            lambda: ns.netsim_add_hier_allreduce(h, 0, np.array([[1, 2], [2, 3]]), MiB),
            lambda: ns.netsim_add_hier_allreduce(h, 0, np.array([[1, 2], [3, 4]]), MiB, after=[7]),
            lambda: ns.netsim_set_link_latency(h, 0, np.zeros(5)),
            lambda: ns.netsim_set_link_latency(h, 0, -np.ones(ns.netsim_get_links(h, 0).size)),
            lambda: ns.netsim_set_link_latency(h, 3, np.zeros(1)),
            lambda: ns.netsim_stream_tree_allreduce(h, 0, [1, 2], [4, 4], MiB),
            lambda: ns.netsim_stream_hier_allreduce(h, 0, np.array([[1, 2]]), np.array([[4, 5]]), -2.0),
        ]
        for f in bad:
            with pytest.raises(ns.NetsimError) as e:
                f()
            assert e.value.status == ns.E_INVALID
            assert ns.netsim_counts(h) == before
        ns.netsim_set_link_latency(h, 0, np.full(ns.netsim_get_links(h, 0).size, 1e-6))
    finally:
        ns.netsim_destroy(h)
    bad_topo = next(_fabrics())
    bad_topo.fabric_latency_s = float("nan")
    with pytest.raises(ns.NetsimError) as e:
        ns.netsim_create_topology([prog.topology_struct(bad_topo, keep)])
    assert e.value.status == ns.E_INVALID
