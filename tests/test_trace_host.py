"""Host-side checks of the event-queue front end (no GPU): the flows the
library lays out for a trace through ``netsim_stream_*`` -- rendezvous,
routed collective flows, per-rank completions, computations -- are the
oracle timeline's, flow for flow (bytes, release lags, routes, dependency
sets); error paths append nothing."""

import numpy as np
import pytest

from oracle import flows as oflows
from oracle import timeline as otl
from workloads.program import MiB, Topology, gbit
from workloads.trace import Collective, Compute, SendRecv, StreamWait, Trace, training_step

from paper_2505_01616_amd import netsim as ns
from paper_2505_01616_amd import program as prog
from paper_2505_01616_amd import trace as ptr


def _compare(tr):
    fs = oflows.expand(otl.build(tr).scenario)
    tl = otl.build(tr)
    ld = ptr.load_trace(tr)
    try:
        ex = ns.netsim_export_flows(ld.handle)
        assert len(ex["nbytes"]) == fs.F
        np.testing.assert_array_equal(ex["nbytes"], fs.nbytes)
        np.testing.assert_array_equal(ex["start"], fs.start)
        routed = fs.src >= 0
        np.testing.assert_array_equal(ex["src"][routed], fs.src[routed])
        np.testing.assert_array_equal(ex["dst"][routed], fs.dst[routed])
        np.testing.assert_array_equal(ex["path_off"], fs.path_off)
        np.testing.assert_array_equal(ex["path_link"], fs.path_link)
        for f in range(fs.F):
            a = ex["dep_ids"][ex["dep_off"][f]:ex["dep_off"][f + 1]]
            b = fs.dep_ids[fs.dep_off[f]:fs.dep_off[f + 1]]
            assert sorted(set(a.tolist())) == sorted(set(b.tolist())), f"flow {f}"
        first = otl._first_flows(tl.scenario)
        for k, d in enumerate(ld.done):
            np.testing.assert_array_equal(d, first[np.asarray(tl.done_op[k])])
        assert ld.tails() == {s: int(first[k]) for s, k in tl.tail_op.items()}
    finally:
        ld.close()


def test_training_step_flows_match_the_oracle():
    _compare(training_step(seed=6, tp=4, pp=2, dp=2, microbatches=2, layers=2))


def test_full_training_step_flows_match_the_oracle():
    _compare(training_step())


def _topo():
    return Topology(kind="leaf_spine", servers=4, gpus_per_server=8, servers_per_leaf=2, spines=2,
                    nvlink_Bps=900e9, nic_Bps=gbit(400), fabric_Bps=gbit(800), ecmp_seed=99)


@pytest.mark.parametrize("mode", ["chained", "flat", "aggregated"])
def test_every_collective_kind(mode):
    tr = Trace("kinds", _topo())
    tr.add(Compute(0, 1e-3))
    tr.add(Compute(5, 2e-3))
    r = np.array([0, 9, 17, 30], np.int32)
    a = tr.add(Collective("allreduce", r, np.array([0, 5, 7, 8]), 8 * MiB, mode=mode))
    b = tr.add(Collective("reduce_scatter", r[::-1].copy(), np.array([8, 7, 5, 0]), 4 * MiB, mode=mode))
    tr.add(StreamWait(40, [(a, 1), (b, 3)]))
    c = tr.add(Collective("all_gather", np.array([1, 2, 25], np.int32), np.array([40, 41, 42]),
                          3 * MiB, mode=mode))
    n = np.arange(16, dtype=np.float64).reshape(4, 4) * MiB
    tr.add(Collective("all_to_all", r, np.array([41, 0, 8, 99]), n))
    tr.add(SendRecv(2, 42, 31, 5, 7 * MiB))
    tr.add(Compute(5, 1e-4, wait=[(c, 2)]))
    _compare(tr)


def test_errors_append_nothing():
    keep = []
    h = ns.netsim_create_topology([prog.topology_struct(_topo(), keep)])
    try:
        ns.netsim_stream_compute(h, 0, 3, 1e-3)
        before = ns.netsim_counts(h)
        tail = ns.netsim_stream_tail(h, 0, 3)
        bad = [
            lambda: ns.netsim_stream_ring(h, 0, ns.RING_ALLREDUCE, ns.MODE_CHAINED, [0, 1], [3, 3], MiB),
            lambda: ns.netsim_stream_ring(h, 0, ns.RING_ALLREDUCE, ns.MODE_CHAINED, [0, 999], [3, 4], MiB),
            lambda: ns.netsim_stream_ring(h, 0, ns.RING_ALLREDUCE, 7, [0, 1], [3, 4], MiB),
            lambda: ns.netsim_stream_ring(h, 0, ns.RING_ALLREDUCE, ns.MODE_CHAINED, [0], [3], MiB),
            lambda: ns.netsim_stream_all_to_all(h, 0, [0, 1], [3, 4], -np.ones(4)),
            lambda: ns.netsim_stream_send(h, 0, 0, 3, 1, 3, MiB),
            lambda: ns.netsim_stream_send(h, 0, 0, 3, 1, 4, -1.0),
            lambda: ns.netsim_stream_compute(h, 0, 3, -1.0),
            lambda: ns.netsim_stream_compute(h, 0, 3, float("nan")),
            lambda: ns.netsim_stream_compute(h, 1, 3, 1.0),
        ]
        for f in bad:
            with pytest.raises(ns.NetsimError) as e:
                f()
            assert e.value.status == ns.E_INVALID
            assert ns.netsim_counts(h) == before
            assert ns.netsim_stream_tail(h, 0, 3) == tail
        assert ns.netsim_stream_tail(h, 0, 12345) == -1
    finally:
        ns.netsim_destroy(h)
