"""Pins of the oracle's event-queue front end (stream semantics of Section
4.1) against closed forms: sequential streams add durations, an event wait
takes the later of two completions, a collective starts when its last
stream arrives and, on dedicated links, takes steps x chunk / capacity; a
whole contention-free training step equals the longest path through its
dependency graph, evaluated here directly from the trace."""

import math

import numpy as np
import pytest

from oracle import timeline as otl
from workloads.program import MiB, Topology, gbit
from workloads.trace import Collective, Compute, SendRecv, StreamWait, Trace, training_step

NV = 900e9
NIC = gbit(400)


def _topo(servers=2):
    return Topology(kind="leaf_spine", servers=servers, gpus_per_server=8, servers_per_leaf=servers,
                    spines=2, nvlink_Bps=NV, nic_Bps=NIC, fabric_Bps=gbit(800), ecmp_seed=7)


def _close(a, b, tol=1e-12):
    assert math.isclose(a, b, rel_tol=tol, abs_tol=1e-300), (a, b)


def test_one_stream_adds_durations():
    d = [0.25e-3, 1.5e-3, 0.0, 3.125e-4, 2e-3]
    tr = Trace("seq", _topo())
    for x in d:
        tr.add(Compute(0, x))
    r = otl.simulate(tr)
    for k in range(len(d)):
        _close(float(r.op_done[k][0]), math.fsum(d[:k + 1]))
    _close(r.stream_sync[0], math.fsum(d))


def test_event_waits_take_the_later_completion():
    tr = Trace("events", _topo())
    a0 = tr.add(Compute(10, 3.0))
    a1 = tr.add(Compute(10, 5.0))
    tr.add(Compute(11, 1.0))
    tr.add(Compute(11, 2.0, wait=[(a0, 0)]))      # max(1, 3) + 2
    tr.add(StreamWait(11, [(a1, 0)]))             # max(5, 8)
    tr.add(Compute(11, 1.0))                      # 9
    tr.add(Compute(12, 0.5))                      # an unrelated stream
    tr.add(Compute(12, 0.25, wait=[(3, 0)]))      # after stream 11's second op: 5 + 0.25
    r = otl.simulate(tr)
    got = [float(x[0]) for x in r.op_done]
    assert got == [3.0, 8.0, 1.0, 5.0, 8.0, 9.0, 0.5, 5.25]
    assert r.stream_sync == {10: 8.0, 11: 9.0, 12: 5.25}


@pytest.mark.parametrize("kind,steps", [("allreduce", 6), ("reduce_scatter", 3), ("all_gather", 3)])
@pytest.mark.parametrize("mode", ["chained", "flat", "aggregated"])
def test_ring_inside_a_server(kind, steps, mode):
    """Four ranks of one server, each ring edge its own NVLink link: the ring
    starts when the last stream arrives and takes steps x (bytes / p) / NV;
    every rank's stream continues from there."""
    tr = Trace("ring", _topo())
    ranks = np.array([0, 1, 2, 3], np.int32)
    for r, t in zip(ranks, [1e-3, 2e-3, 3e-3, 0.0]):
        if t:
            tr.add(Compute(int(r), t))
    nb = 64 * MiB
    k = tr.add(Collective(kind, ranks, ranks.astype(np.int64), nb, mode=mode))
    tr.add(Compute(2, 1e-4))
    r = otl.simulate(tr)
    want = 3e-3 + steps * (nb / 4) / NV
    for x in r.op_done[k]:
        _close(float(x), want, 1e-9)
    _close(r.stream_sync[2], want + 1e-4, 1e-9)
    _close(r.stream_sync[0], want, 1e-9)


def test_send_recv_across_servers():
    tr = Trace("send", _topo())
    tr.add(Compute(100, 2e-3))
    tr.add(Compute(201, 1e-3))
    k = tr.add(SendRecv(3, 100, 11, 201, 50 * MiB))
    tr.add(Compute(201, 1e-4))
    r = otl.simulate(tr)
    t = 2e-3 + 50 * MiB / NIC
    _close(float(r.op_done[k][0]), t, 1e-9)
    _close(float(r.op_done[k][1]), t, 1e-9)
    _close(r.stream_sync[201], t + 1e-4, 1e-9)


def test_all_to_all_rank_waits_for_row_and_column():
    """Inside one server every ordered pair has its own link: flow (i, j)
    takes n[i, j] / NV from the rendezvous, and rank i is done when both what
    it sends and what it receives have arrived."""
    n = np.array([[0, 1, 2], [9, 0, 1], [1, 3, 0]], np.float64) * MiB
    tr = Trace("a2a", _topo())
    tr.add(Compute(7, 1e-3))
    k = tr.add(Collective("all_to_all", np.array([5, 6, 7], np.int32), np.array([5, 6, 7]), n))
    r = otl.simulate(tr)
    for i in range(3):
        want = 1e-3 + max(np.max(n[i]), np.max(n[:, i])) / NV
        _close(float(r.op_done[k][i]), want, 1e-9)
    assert r.op_done[k][0] > 1e-3 + np.max(n[0]) / NV * 1.5   # rank 0 waits for its column


def _longest_path(tr):
    """Completion per (operation, position) of a contention-free trace, by
    walking the operations in issue order: each communication flow takes its
    bytes over the narrowest link of its path, and every link must be busy
    with one flow at a time (checked)."""
    topo = tr.topo
    G = topo.gpus_per_server
    tail, done, busy = {}, [], {}

    def links(a, b):
        if a // G == b // G:
            return [("nv", a, b)], NV
        return [("up", a), ("down", b)], NIC

    def occupy(a, b, t0, t1):
        ls, _ = links(a, b)
        for l in ls:
            for (s, e) in busy.get(l, []):
                assert t1 <= s or t0 >= e, f"link {l} shared: the check needs a contention-free trace"
            busy.setdefault(l, []).append((t0, t1))

    for op in tr.ops:
        if isinstance(op, (Compute, StreamWait)):
            t = max([tail.get(op.stream, 0.0)] + [done[k][j] for k, j in op.wait])
            t += op.duration if isinstance(op, Compute) else 0.0
            tail[op.stream] = t
            done.append([t])
        elif isinstance(op, Collective):
            assert op.kind == "allreduce" and op.mode == "chained"
            t0 = max(tail.get(int(s), 0.0) for s in op.streams)
            p = len(op.ranks)
            _, cap = links(int(op.ranks[0]), int(op.ranks[1]))
            step = (op.nbytes / p) / cap
            t1 = t0
            for _ in range(2 * (p - 1)):
                t1 = t1 + step
            for i in range(p):
                occupy(int(op.ranks[i]), int(op.ranks[(i + 1) % p]), t0, t1)
            for s in op.streams:
                tail[int(s)] = t1
            done.append([t1] * p)
        else:
            t0 = max(tail.get(op.src_stream, 0.0), tail.get(op.dst_stream, 0.0))
            _, cap = links(op.src, op.dst)
            t1 = t0 + op.nbytes / cap
            occupy(op.src, op.dst, t0, t1)
            tail[op.src_stream] = tail[op.dst_stream] = t1
            done.append([t1, t1])
    return done, tail


def test_training_step_is_its_longest_path():
    """Tensor parallelism inside each of two servers, a two-stage pipeline
    between them (dp = 1): no link ever carries two flows at once, so every
    completion is a longest path through the operations."""
    tr = training_step(seed=3, tp=8, pp=2, dp=1, microbatches=4, layers=2)
    want, tails = _longest_path(tr)
    r = otl.simulate(tr)
    for k, w in enumerate(want):
        np.testing.assert_allclose(r.op_done[k], w, rtol=1e-9, err_msg=f"operation {k}")
    assert set(r.stream_sync) == set(tails)
    for s, t in tails.items():
        _close(r.stream_sync[s], t, 1e-9)


def test_training_step_orders_every_stream():
    """Any trace: completions along a stream never go back in time, and a
    collective's flows start no earlier than its last stream's arrival."""
    tr = training_step(seed=5, tp=4, pp=2, dp=2, microbatches=3, layers=2)
    r = otl.simulate(tr)
    prev = {}
    for k, op in enumerate(tr.ops):
        streams = ([op.stream] if isinstance(op, (Compute, StreamWait)) else
                   list(op.streams) if isinstance(op, Collective) else [op.src_stream, op.dst_stream])
        for s, t in zip(streams, r.op_done[k]):
            assert t >= prev.get(int(s), 0.0)
            prev[int(s)] = float(t)
    assert np.all(np.isfinite(r.finish))
    assert prev == r.stream_sync
