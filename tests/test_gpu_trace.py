"""GPU parity of the event-queue front end: traces of stream operations fed
through ``netsim_stream_*`` and simulated by the HIP path, against the
oracle timeline on the same trace.  Per-flow completion times (and so every
stream synchronisation) agree within 1e-6 relative."""

import sys

import numpy as np
import pytest

from oracle import timeline as otl
from workloads.program import MiB, Topology, gbit
from workloads.trace import Collective, Compute, SendRecv, StreamWait, Trace, training_step

pytestmark = pytest.mark.gpu

TOL = 1e-6


def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2505_01616_amd import netsim as ns
    from paper_2505_01616_amd import trace as ptr
    return ns, ptr


def _say(*a):
    print(*a, file=sys.stderr, flush=True)

def _layout(ns, name):
    """Options of an execution layout; the cluster layout hands every
    re-solve to the helper workgroups (assist_min_flows = 1)."""
    if name == "cluster":
        return dict(exec=ns.EXEC_CLUSTER, assist_min_flows=1)
    return dict(exec={"block": ns.EXEC_BLOCK, "grid": ns.EXEC_GRID}[name])



def _rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    assert a.shape == b.shape
    assert np.all(np.isfinite(a)) and np.all(np.isfinite(b))
    return float(np.max(np.abs(a - b) / np.maximum(np.abs(b), 1e-300))) if a.size else 0.0


def _check(tr, **opt):
    ns, ptr = _gpu()
    ref = otl.simulate(tr)
    fin, done, sync, st = ptr.run_trace(tr, ns.make_options(**opt))
    assert st["complete"] == 1
    assert _rel(fin, ref.finish) < TOL
    for k in range(len(done)):
        assert _rel(done[k], ref.op_done[k]) < TOL, k
    assert sync.keys() == ref.stream_sync.keys()
    assert _rel([sync[s] for s in sorted(sync)], [ref.stream_sync[s] for s in sorted(sync)]) < TOL
    return st, ref


def _mixed(mode):
    topo = Topology(kind="leaf_spine", servers=4, gpus_per_server=8, servers_per_leaf=2, spines=2,
                    nvlink_Bps=900e9, nic_Bps=gbit(400), fabric_Bps=gbit(800), ecmp_seed=99)
    tr = Trace("kinds", topo)
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
    return tr


@pytest.mark.parametrize("mode", ["chained", "flat", "aggregated"])
def test_every_collective_kind(mode):
    _say(f"test_every_collective_kind mode={mode}")
    _check(_mixed(mode))


@pytest.mark.parametrize("single_clock", [0, 1])
@pytest.mark.parametrize("exec_", ["block", "grid", "cluster"])
def test_small_training_step(exec_, single_clock):
    ns, _ = _gpu()
    _say(f"test_small_training_step exec={exec_} single_clock={single_clock}")
    ex = _layout(ns, exec_)
    st, ref = _check(training_step(seed=6, tp=4, pp=2, dp=2, microbatches=3, layers=2),
                     **ex, single_clock=single_clock)
    if single_clock:
        assert st["events"] == ref.events and st["solves"] == ref.solves


def test_full_training_step():
    """128 ranks (TP 8 x PP 4 x DP 4), 8 micro-batches: ~14k operations,
    ~142k flows."""
    _say("test_full_training_step")
    _check(training_step())


def test_stream_calls_after_a_run_are_refused():
    ns, ptr = _gpu()
    ld = ptr.load_trace(_mixed("chained"))
    try:
        ns.netsim_run(ld.handle)
        with pytest.raises(ns.NetsimError) as e:
            ns.netsim_stream_compute(ld.handle, 0, 0, 1e-3)
        assert e.value.status == ns.E_STATE
    finally:
        ld.close()


@pytest.mark.parametrize("exec_", ["block", "grid", "cluster"])
def test_compute_duration_change_rolls_back(exec_):
    """A computation found longer than assumed after the simulation passed it
    (the situation time rollback exists for): its flow's start (the
    duration) is updated, the simulation goes back and continues; the result
    equals, bit for bit, a run of the trace with the right duration from the
    start, and the oracle's timeline of that trace."""
    import copy
    ns, ptr = _gpu()
    _say(f"test_compute_duration_change_rolls_back exec={exec_}")
    tr = training_step(seed=8, tp=4, pp=2, dp=2, microbatches=3, layers=2)
    ex = _layout(ns, exec_)
    computes = [k for k, op in enumerate(tr.ops) if type(op).__name__ == "Compute"]
    k = computes[len(computes) // 3]
    new_d = tr.ops[k].duration + 4e-4
    ld = ptr.load_trace(tr, ns.make_options(**ex))
    try:
        h = ld.handle
        ns.netsim_advance(h)
        before = ns.netsim_get_finish(h)
        x = int(ld.done[k][0])
        assert np.isfinite(before[x])
        ns.netsim_update_start(h, x, new_d)
        ns.netsim_advance(h)
        got = ns.netsim_get_finish(h)
    finally:
        ld.close()
    tr2 = copy.deepcopy(tr)
    tr2.ops[k].duration = new_d
    fin2, _, _, _ = ptr.run_trace(tr2, ns.make_options(**ex))
    assert np.array_equal(got, fin2)
    assert np.sum(got != before) > 0
    ref = otl.simulate(tr2)
    assert _rel(got, ref.finish) < TOL


@pytest.mark.parametrize("exec_", ["block", "grid"])
def test_compute_duration_change_rolls_back_from_history(exec_):
    """The same with tree all-reduce, link latencies and the rollback
    history: the part returns to its last event before the computation's
    new end instead of a checkpoint; the result equals, bit for bit, a run
    of the trace with the right duration from the start, and the oracle's
    timeline of that trace."""
    import copy
    ns, ptr = _gpu()
    _say(f"test_compute_duration_change_rolls_back_from_history exec={exec_}")
    tr = training_step(seed=9, tp=4, pp=2, dp=2, microbatches=3, layers=2, allreduce="tree",
                       fabric_latency_s=1e-6, nvlink_latency_s=3e-7)
    ex = _layout(ns, exec_)
    computes = [k for k, op in enumerate(tr.ops) if type(op).__name__ == "Compute"]
    k = computes[len(computes) // 2]
    new_d = tr.ops[k].duration + 3e-4
    ld = ptr.load_trace(tr, ns.make_options(history_mb=32, **ex))
    try:
        h = ld.handle
        ns.netsim_advance(h)
        before = ns.netsim_get_finish(h)
        x = int(ld.done[k][0])
        assert np.isfinite(before[x])
        ns.netsim_update_start(h, x, new_d)
        ns.netsim_advance(h)
        got = ns.netsim_get_finish(h)
        resim = ns.netsim_get_stats(h)["launch_events"]
        total = ns.netsim_get_stats(h)["events"]
    finally:
        ld.close()
    tr2 = copy.deepcopy(tr)
    tr2.ops[k].duration = new_d
    fin2, _, _, _ = ptr.run_trace(tr2, ns.make_options(**ex))
    assert np.array_equal(got, fin2)
    assert np.sum(got != before) > 0
    assert 0 < resim < total  # from the event before the change, not from t = 0
    ref = otl.simulate(tr2)
    assert _rel(got, ref.finish) < TOL
