"""GPU parity of the richer collectives and per-link latency: double binary
tree and hierarchical all-reduce on three fabrics with latencies, random
explicit cases with latencies and dependencies, the 128-GPU training step
with tree all-reduce and latencies through the event-queue front end, and
time rollback with latencies.  Per-flow completion times within 1e-6 of the
oracle; pieces and rollbacks bit for bit equal to one run."""

import sys

import numpy as np
import pytest

from oracle import flows as oflows
from oracle import sim as osim
from oracle import timeline as otl
from workloads import configs
from workloads.program import Hier, MiB, PathFlow, Program, Ring, Scenario, Send, Topology, Tree, gbit
from workloads.trace import training_step

pytestmark = pytest.mark.gpu

TOL = 1e-6


def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2505_01616_amd import netsim as ns
    from paper_2505_01616_amd import program as prog
    from paper_2505_01616_amd import trace as ptr
    return ns, prog, ptr


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
    fa, fb = np.isfinite(a), np.isfinite(b)
    assert np.array_equal(fa, fb), "different sets of finished flows"
    return float(np.max(np.abs(a[fa] - b[fa]) / np.maximum(np.abs(b[fa]), 1e-300))) if fa.any() else 0.0


def _scenarios():
    topos = [
        Topology(kind="leaf_spine", servers=8, gpus_per_server=8, servers_per_leaf=2, spines=4,
                 nvlink_Bps=900e9, nic_Bps=gbit(400), fabric_Bps=gbit(800), ecmp_seed=17,
                 fabric_latency_s=1e-6, nvlink_latency_s=2e-7),
        Topology(kind="rail", servers=8, gpus_per_server=8, servers_per_leaf=4, spines=4,
                 nvlink_Bps=900e9, nic_Bps=gbit(400), fabric_Bps=gbit(400), ecmp_seed=3,
                 fabric_latency_s=5e-7),
        configs.c3_topology(7),
    ]
    topos[2].fabric_latency_s = 2e-6
    out = []
    for k, topo in enumerate(topos):
        rng = np.random.default_rng(100 + k)
        sc = Scenario(topo)
        for p in (2, 5, 16, 37):
            sc.add(Tree(rng.permutation(topo.endpoints)[:p].astype(np.int32), 24 * MiB,
                        lag=float(rng.random() * 1e-5)))
        for m, g in ((4, 8), (3, 1), (1, 5), (5, 3)):
            r = rng.permutation(topo.endpoints)[:m * g].reshape(m, g).astype(np.int32)
            sc.add(Hier(r, 40 * MiB, lag=1e-6, after=(len(sc.ops) - 1,)))
        sc.add(Send(0, topo.endpoints - 1, MiB, after=(len(sc.ops) - 1, (2, 5))))
        sc.add(Ring("allreduce", np.arange(12, dtype=np.int32), 12 * MiB, after=(len(sc.ops) - 1,)))
        out.append(sc)
    return out


@pytest.mark.parametrize("single_clock", [0, 1])
@pytest.mark.parametrize("exec_", ["block", "grid", "cluster"])
def test_tree_hier_latency(exec_, single_clock):
    ns, pr, _ = _gpu()
    _say(f"test_tree_hier_latency exec={exec_} single_clock={single_clock}")
    scs = _scenarios()
    ex = _layout(ns, exec_)
    fins, st = pr.run_program(Program("next4", scs), ns.make_options(**ex, single_clock=single_clock))
    assert st["complete"] == 1
    for s, sc in enumerate(scs):
        ref = osim.run_scenario(sc)
        assert _rel(fins[s], ref.finish) < TOL, s


def _latency_micro(seed):
    rng = np.random.default_rng(seed)
    L = int(rng.integers(2, 7))
    topo = Topology(kind="explicit", capacities=rng.choice([1e9, 2e9, 5e8, 4e9], size=L),
                    latencies=rng.choice([0.0, 1e-4, 2.5e-4, 5e-4], size=L))
    sc = Scenario(topo)
    for k in range(int(rng.integers(2, 12))):
        path = sorted(rng.choice(L, size=int(rng.integers(1, min(L, 6) + 1)), replace=False).tolist())
        after = tuple(int(a) for a in rng.choice(k, size=min(k, int(rng.integers(0, 3))),
                                                 replace=False)) if k else ()
        sc.add(PathFlow(path, float(rng.choice([1e5, 3e5, 1e6])), lag=float(rng.choice([0.0, 1e-4])),
                        after=after))
    return sc


def test_latency_micro_batched():
    ns, pr, _ = _gpu()
    _say("test_latency_micro_batched")
    scs = [_latency_micro(s) for s in range(150)]
    fins, st = pr.run_program(Program("lat-micro", scs), ns.make_options(single_clock=1))
    for s, sc in enumerate(scs):
        ref = osim.run_scenario(sc)
        assert _rel(fins[s], ref.finish) < TOL, s


@pytest.mark.parametrize("alg", ["tree", "ring"])
def test_training_step_with_latency(alg):
    ns, _, ptr = _gpu()
    _say(f"test_training_step_with_latency alg={alg}")
    tr = training_step(allreduce=alg, fabric_latency_s=1e-6, nvlink_latency_s=3e-7)
    ref = otl.simulate(tr)
    fin, done, sync, st = ptr.run_trace(tr)
    assert st["complete"] == 1
    assert _rel(fin, ref.finish) < TOL
    assert _rel([sync[s] for s in sorted(sync)], [ref.stream_sync[s] for s in sorted(sync)]) < TOL


@pytest.mark.parametrize("exec_", ["block", "grid", "cluster"])
def test_latency_pieces_and_rollback(exec_):
    """With latencies: advancing in pieces equals one run bit for bit; moving
    a finished flow's start back in time, then advancing, equals a fresh
    run with that start."""
    ns, pr, _ = _gpu()
    _say(f"test_latency_pieces_and_rollback exec={exec_}")
    program = Program("next4", _scenarios()[:2])
    ex = _layout(ns, exec_)
    opt = dict(ex)

    def fresh(updates):
        ld = pr.load_program(program, ns.make_options(**opt))
        try:
            for fid, s in updates.items():
                ns.netsim_update_start(ld.handle, fid, s)
            ns.netsim_run(ld.handle)
            return ns.netsim_get_finish(ld.handle)
        finally:
            ld.close()

    ref = fresh({})
    T = float(np.nanmax(ref))
    ld = pr.load_program(program, ns.make_options(**opt))
    try:
        h = ld.handle
        for frac in (0.25, 0.6):
            ns.netsim_advance(h, until=frac * T)
        ns.netsim_advance(h)
        assert np.array_equal(ns.netsim_get_finish(h), ref)
        ex_ = ns.netsim_export_flows(h)
        cand = np.nonzero((ex_["nbytes"] > 0) & (ref > 0.5 * T) & (ex_["dep_off"][1:] == ex_["dep_off"][:-1]))[0]
        if len(cand) == 0:
            cand = np.nonzero(ex_["nbytes"] > 0)[0]
        x = int(cand[len(cand) // 2])
        new = float(ex_["start"][x]) + 3e-5
        ns.netsim_update_start(h, x, new)
        ns.netsim_advance(h)
        got = ns.netsim_get_finish(h)
    finally:
        ld.close()
    assert np.array_equal(got, fresh({x: new}))


@pytest.mark.parametrize("exec_", ["block", "grid"])
def test_latency_rollback_from_history(exec_):
    """With latencies and the rollback history: starts of flows with and
    without predecessors moved after the simulation passed them (each part
    goes back to its last event before the change, rebuilding the waiting
    flows' counts and, with latency, their bases from the arrivals of the
    predecessors finished by then); then advancing equals, bit for bit, a
    fresh run with those starts, and the rollback re-simulates fewer events
    than the one from the latest checkpoint."""
    ns, pr, _ = _gpu()
    _say(f"test_latency_rollback_from_history exec={exec_}")
    program = Program("next4", _scenarios()[:2])
    ex = _layout(ns, exec_)

    def fresh(updates):
        ld = pr.load_program(program, ns.make_options(**ex))
        try:
            for fid, s in updates.items():
                ns.netsim_update_start(ld.handle, fid, s)
            ns.netsim_run(ld.handle)
            return ns.netsim_get_finish(ld.handle)
        finally:
            ld.close()

    ref = fresh({})
    T = float(np.nanmax(ref))

    def rolled(history_mb):
        ld = pr.load_program(program, ns.make_options(history_mb=history_mb, **ex))
        try:
            h = ld.handle
            ns.netsim_advance(h, until=0.3 * T)
            ns.netsim_advance(h)
            ex_ = ns.netsim_export_flows(h)
            deps = ex_["dep_off"][1:] > ex_["dep_off"][:-1]
            upd = {}
            for want_deps, frac, d in ((True, 0.6, 2e-5), (False, 0.45, 3e-5)):
                # the flow of that kind finishing nearest to frac of the horizon
                c = np.nonzero((ex_["nbytes"] > 0) & (deps == want_deps))[0]
                assert len(c), want_deps
                x = int(c[np.argmin(np.abs(ref[c] - frac * T))])
                upd[x] = float(ex_["start"][x]) + d
                ns.netsim_update_start(h, x, upd[x])
            ns.netsim_advance(h)
            return ns.netsim_get_finish(h), ns.netsim_get_stats(h)["launch_events"], upd
        finally:
            ld.close()

    got, ev_hist, upd = rolled(64)
    alt, ev_ckpt, upd2 = rolled(0)
    assert upd == upd2
    want = fresh(upd)
    assert np.array_equal(got, want)
    assert np.array_equal(alt, want)
    assert not np.array_equal(want, ref)
    assert ev_hist < ev_ckpt
    _say("  continuation events: history", ev_hist, "checkpoint", ev_ckpt)
