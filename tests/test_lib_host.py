"""Host-side checks of libnetsim that need no GPU: every declared symbol is
exported; routes, capacities and collective decompositions are bit-exact
with the oracle's independent Python implementation; every error status is
reachable from the host."""

import ctypes
import math
import os
import re

import numpy as np
import pytest

from oracle import flows as oflows
from oracle.topology import Fabric
from workloads import configs, micro
from workloads.program import Program, Ring, Scenario, Send, Topology, MiB

from paper_2505_01616_amd import netsim as ns
from paper_2505_01616_amd import program as prog

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_exports_every_declared_symbol():
    with open(os.path.join(ROOT, "include", "netsim.h")) as fh:
        hdr = fh.read()
    names = sorted(set(re.findall(r"\b(netsim_[a-z_]+)\s*\(", hdr)))
    assert len(names) >= 17
    lib = ctypes.CDLL(ns.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


def _compare(program):
    """Library's stored flows == oracle's expansion, scenario by scenario."""
    ld = prog.load_program(program)
    try:
        ex = ns.netsim_export_flows(ld.handle)
        for s, sc in enumerate(program.scenarios):
            fs = oflows.expand(sc)
            a, n = ld.first_flow[s], ld.num_flows[s]
            assert n == fs.F
            assert np.all(ex["scen"][a:a + n] == s)
            np.testing.assert_array_equal(ex["nbytes"][a:a + n], fs.nbytes)
            np.testing.assert_array_equal(ex["start"][a:a + n], fs.start)
            routed = fs.src >= 0
            np.testing.assert_array_equal(ex["src"][a:a + n][routed], fs.src[routed])
            np.testing.assert_array_equal(ex["dst"][a:a + n][routed], fs.dst[routed])
            po = ex["path_off"][a:a + n + 1]
            np.testing.assert_array_equal(po - po[0], fs.path_off)
            np.testing.assert_array_equal(ex["path_link"][po[0]:po[-1]], fs.path_link)
            do = ex["dep_off"][a:a + n + 1]
            np.testing.assert_array_equal(do - do[0], fs.dep_off)
            np.testing.assert_array_equal(ex["dep_ids"][do[0]:do[-1]] - a, fs.dep_ids)
            np.testing.assert_array_equal(ns.netsim_get_links(ld.handle, s), fs.cap)
    finally:
        ld.close()


@pytest.mark.parametrize("mode", ["chained", "flat", "aggregated"])
def test_bit_exact_c1(mode):
    _compare(configs.c1(1, mode=mode))


def test_bit_exact_c2_c3():
    _compare(configs.c2(2))
    _compare(configs.c3(3))


def test_bit_exact_c4():
    _compare(configs.c4(4))


def test_bit_exact_c5_sample():
    _compare(configs.c5(5, scenarios=3))
    _compare(configs.c5(5, scenarios=2, first=100))


def test_bit_exact_explicit_micro():
    for seed in range(20):
        _compare(micro.random_dynamic(seed))


def test_rs_ag_chain_and_seed_sweep():
    for seed in (101, 105, 110):
        _compare(configs.c1(seed))
        topo = configs.c3_topology(seed)
        sc = Scenario(topo)
        ranks = np.arange(0, 1024, 37, dtype=np.int32)
        sc.add(Ring("reduce_scatter", ranks, 64 * MiB, lag=1e-6))
        sc.add(Ring("all_gather", ranks, 64 * MiB, mode="flat", after=(0,)))
        sc.add(Send(3, 999, 5 * MiB, after=(1,)))
        _compare(Program("rsag", [sc]))


# ------------------------------------------------------------ error paths
def _status(fn, *a):
    try:
        fn(*a)
    except ns.NetsimError as e:
        return e.status
    return ns.OK


def _small_topo():
    return prog.topology_struct(configs.c1_topology(1), [])


def test_error_invalid_arguments():
    lib = ns.load_library()
    h = ctypes.c_void_p()
    assert lib.netsim_create(ctypes.byref(h), 0, None, None, None) == ns.E_INVALID
    assert "scenario" in ns.netsim_last_error(None)
    lo = np.array([0, 2], np.int64)
    assert _status(ns.netsim_create, lo, np.array([1.0, -1.0])) == ns.E_INVALID
    assert _status(ns.netsim_create, lo, np.array([1.0, np.inf])) == ns.E_INVALID
    bad = _small_topo()
    bad.servers = 7
    bad.servers_per_leaf = 2
    assert _status(ns.netsim_create_topology, [bad]) == ns.E_INVALID
    bad = _small_topo()
    bad.nic_Bps = 0.0
    assert _status(ns.netsim_create_topology, [bad]) == ns.E_INVALID
    h = ns.netsim_create(np.array([0, 3], np.int64), np.array([1.0, 2.0, 3.0]))
    try:
        one, zero = np.ones(1), np.zeros(1)
        po = np.array([0, 1], np.int64)
        cases = [
            dict(path_off=po, path_link=np.array([3], np.int32)),          # link out of range
            dict(path_off=np.array([0, 0], np.int64), path_link=np.zeros(0, np.int32)),  # empty path
            dict(path_off=np.array([0, 2], np.int64), path_link=np.array([1, 1], np.int32)),  # repeated
            dict(path_off=po, path_link=np.array([0], np.int32), dep_off=po,
                 dep_ids=np.array([0], np.int64)),                         # depends on itself
        ]
        for kw in cases:
            assert _status(ns.netsim_add_flows, h, 0, one, zero, None, None,
                           kw.get("path_off"), kw.get("path_link"), kw.get("dep_off"),
                           kw.get("dep_ids")) == ns.E_INVALID, kw
        for b, s in ((-1.0, 0.0), (np.nan, 0.0), (1.0, -1.0), (1.0, np.inf)):
            assert _status(ns.netsim_add_flows, h, 0, [b], [s], None, None, po,
                           np.array([0], np.int32)) == ns.E_INVALID
        assert _status(ns.netsim_add_flows, h, 1, one, zero, None, None, po,
                       np.array([0], np.int32)) == ns.E_INVALID            # bad scenario
        assert _status(ns.netsim_add_flows, h, 0, one, zero, [0], [1]) == ns.E_INVALID  # no fabric
        assert ns.netsim_add_flows(h, 0, one, zero, path_off=po, path_link=np.array([2], np.int32)) == 0
        assert ns.netsim_counts(h) == (1, 1, 0)   # failed calls added nothing
    finally:
        ns.netsim_destroy(h)
    h = ns.netsim_create_topology([_small_topo()])
    try:
        assert _status(ns.netsim_add_flows, h, 0, [1.0], [0.0], [5], [5]) == ns.E_INVALID   # src == dst
        assert _status(ns.netsim_add_flows, h, 0, [1.0], [0.0], [5], [64]) == ns.E_INVALID  # endpoint range
        assert _status(ns.netsim_add_ring, h, 0, 7, 0, [0, 1], 1.0) == ns.E_INVALID          # kind
        assert _status(ns.netsim_add_ring, h, 0, 0, 0, [3], 1.0) == ns.E_INVALID             # p < 2
        assert _status(ns.netsim_add_ring, h, 0, 0, 0, [3, 3], 1.0) == ns.E_INVALID          # repeated rank
        assert _status(ns.netsim_add_ring, h, 0, 0, 0, [0, 1], 1.0, 0.0, [0]) == ns.E_INVALID  # 'after'
        assert _status(ns.netsim_add_all_to_all, h, 0, [0, 1], np.ones(4), -1.0) == ns.E_INVALID
        assert ns.netsim_add_flows(h, 0, [0.0], [0.0], [-1], [-1]) == 0                    # barrier
        assert ns.netsim_counts(h)[0] == 1
    finally:
        ns.netsim_destroy(h)


def test_error_state_limit_device():
    h = ns.netsim_create(np.array([0, 1], np.int64), np.array([1.0]))
    try:
        assert _status(ns.netsim_get_finish, h) == ns.E_STATE          # no run yet
        lib = ns.load_library()
        one = np.ones(1)
        rc = lib.netsim_add_flows(h, 0, (1 << 31), None, None, ns._ptr(one), ns._ptr(one), None,
                                  None, None, None, None)
        assert rc == ns.E_LIMIT                                          # too many flows
        assert _status(ns.netsim_set_limits, h, -1, math.inf) == ns.E_INVALID
    finally:
        ns.netsim_destroy(h)


def test_error_device_without_gpu():
    """Without a usable GPU, running reports NETSIM_E_DEVICE (not a crash)."""
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    h = ns.netsim_create(np.array([0, 1], np.int64), np.array([1.0]))
    try:
        ns.netsim_add_flows(h, 0, [1.0], [0.0], path_off=[0, 1], path_link=[0])
        assert _status(ns.netsim_run, h) == ns.E_DEVICE
    finally:
        ns.netsim_destroy(h)


def test_update_start_host_side():
    """Time-rollback entry points without a GPU: argument checks, and a start
    changed before the first run is what the flows hold (and export)."""
    h = ns.netsim_create(np.array([0, 2], np.int64), np.array([1.0, 2.0]))
    try:
        po = np.array([0, 1, 2], np.int64)
        ns.netsim_add_flows(h, 0, [4.0, 8.0], [0.0, 0.5], path_off=po,
                            path_link=np.array([0, 1], np.int32))
        assert _status(ns.netsim_update_start, h, 2, 1.0) == ns.E_INVALID     # no such flow
        assert _status(ns.netsim_update_start, h, -1, 1.0) == ns.E_INVALID
        assert _status(ns.netsim_update_start, h, 0, -1.0) == ns.E_INVALID    # negative start
        assert _status(ns.netsim_update_start, h, 0, np.nan) == ns.E_INVALID
        assert _status(ns.netsim_advance, h, np.nan, 0) == ns.E_INVALID
        assert _status(ns.netsim_advance, h, 1.0, -1) == ns.E_INVALID
        assert _status(ns.netsim_gc, h, np.nan) == ns.E_INVALID
        ns.netsim_update_start(h, 1, 0.25)
        np.testing.assert_array_equal(ns.netsim_export_flows(h)["start"], [0.0, 0.25])
        assert ns.netsim_num_checkpoints(h) == 0
        ns.netsim_gc(h, 1.0)
    finally:
        ns.netsim_destroy(h)


@pytest.mark.parametrize("kind", ["ring-chained", "ring-flat", "ring-aggregated", "rs-chained",
                                  "all-to-all", "tree", "hier"])
def test_last_exits_are_the_oracles(kind):
    """netsim_last_exits after each kind of operation equals the oracle's exit
    flows of that operation, read off the dependency list of a barrier the
    oracle places after it (ids relative to the operation's first flow)."""
    from workloads.program import AllToAll, Barrier, Hier, Tree
    topo = configs.c1_topology(1)
    ranks = np.array([0, 9, 17, 3, 40, 63], dtype=np.int32)
    if kind.startswith("ring") or kind.startswith("rs"):
        k = "reduce_scatter" if kind.startswith("rs") else "allreduce"
        op = Ring(k, ranks, 12 * MiB, mode=kind.split("-")[1])
    elif kind == "all-to-all":
        op = AllToAll(ranks, np.full((6, 6), 1.0 * MiB))
    elif kind == "tree":
        op = Tree(ranks, 8 * MiB)
    else:
        op = Hier(np.array([[0, 1, 2], [8, 9, 10], [16, 17, 18]], dtype=np.int32), 9 * MiB)
    sc = Scenario(topo)
    sc.add(Send(5, 6, 1.0))          # a flow before, so ids do not start at 0
    sc.add(op)
    sc.add(Barrier(after=(1,)))
    fs = oflows.expand(sc)
    want = fs.dep_ids[fs.dep_off[fs.F - 1]:fs.dep_off[fs.F]] - 1
    ld = prog.load_program(Program("x", [Scenario(topo, ops=sc.ops[:2])]))
    try:
        got = ns.netsim_last_exits(ld.handle) - 1
    finally:
        ld.close()
    assert np.array_equal(np.sort(got), np.sort(want))
    assert len(got) > 0


def test_last_exits_of_a_batch_and_before_any():
    h = ns.netsim_create(np.array([0, 2], np.int64), np.array([1.0, 2.0]))
    try:
        with pytest.raises(ns.NetsimError) as ei:
            ns.netsim_last_exits(h)
        assert ei.value.status == ns.E_STATE
        ns.netsim_add_flows(h, 0, np.array([1.0, 2.0, 0.0]), np.zeros(3),
                            path_off=np.array([0, 1, 2, 2], np.int64),
                            path_link=np.array([0, 1], np.int32))
        assert list(ns.netsim_last_exits(h)) == [0, 1, 2]
    finally:
        ns.netsim_destroy(h)


def test_negative_history_is_refused():
    opt = ns.make_options(history_mb=-1)
    with pytest.raises(ns.NetsimError) as ei:
        ns.netsim_create(np.array([0, 1], np.int64), np.array([1.0]), opt)
    assert ei.value.status == ns.E_INVALID
    assert "history_mb" in str(ei.value)
