"""Oracle for the event-queue front end: stream operations -> dependent flows.

Test infrastructure: only the tests, the smoke check and the benchmark's CPU
baseline use this module; the simulator library never does.

Section 4.1 (supporting unmodified ML frameworks) describes how CUDA
streams and events are emulated by dependencies in the event queue:
operations issued on one stream depend on each other in issue order;
operations on different streams are independent unless an event links
them; a synchronisation on a stream yields the completion time of its last
operation.  An NCCL collective forwarded to the simulator can only move data
once every rank of the communicator has issued it; each rank's stream then
continues when that rank's own part of the collective is over.

This module writes those rules out as a ``workloads.program.Scenario``:

* computation of d seconds on stream s: a zero-byte barrier released d
  after the completion of the previous operation on s and of every awaited
  event (with nothing to wait for, released at time d);
* an event wait on s: the same with d = 0;
* a collective (or send/recv) on streams s_1..s_p: a rendezvous barrier after
  the previous operation of every s_i, the collective's flows after the
  rendezvous, then one barrier per rank after the flows that leave or
  enter that rank and finish last -- a chained ring's last step, every step
  of a flat ring, both edges of an aggregated ring, the whole row and column
  of an all-to-all, the broadcasts into and out of it in both trees of a
  tree all-reduce, its last phase's last step in a hierarchical all-reduce,
  the single flow of a send -- which becomes the rank's stream completion.

The scenario then goes through ``oracle.flows.expand`` (decomposition and
routing) and ``oracle.sim`` (the event loop); nothing here computes a time.
"""

from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, List

import numpy as np

from workloads.program import AllToAll, Barrier, Hier, Ring, Scenario, Send, Tree
from workloads.trace import Collective, Compute, SendRecv, StreamWait, Trace

from . import flows as oflows
from . import sim as osim

_RING_STEPS = {"allreduce": lambda p: 2 * (p - 1), "reduce_scatter": lambda p: p - 1,
               "all_gather": lambda p: p - 1}


@dataclass
class Timeline:
    scenario: Scenario
    done_op: List[List[int]]     # per trace operation: the scenario op completing it per stream
    tail_op: Dict[int, int]      # stream -> scenario op of its last operation's completion


def _rank_flows(op: Collective, i: int) -> List[int]:
    """Flows (numbered as the collective lays them out) rank i waits for."""
    p = len(op.ranks)
    left = (i - 1) % p
    if op.kind == "all_to_all":
        def flow(a, b):        # row-major over ordered pairs without the diagonal
            return a * (p - 1) + (b if b < a else b - 1)
        return [flow(i, j) for j in range(p) if j != i] + [flow(j, i) for j in range(p) if j != i]
    steps = _RING_STEPS[op.kind](p)
    if op.mode == "aggregated":
        return [i, left]
    if op.mode == "chained":
        return [(steps - 1) * p + i, (steps - 1) * p + left]
    if op.mode == "flat":
        return [k * p + x for k in range(steps) for x in (i, left)]
    raise ValueError(op.mode)


def _last_flows_of(op: Collective, positions):
    """Tree / hierarchical all-reduce: per rank position (row-major), the
    collective's flows (numbered within it) among its last ones that leave
    or enter the rank."""
    ranks = np.asarray(op.ranks)
    mk = oflows._tree_flows if op.kind == "tree_allreduce" else oflows._hier_flows
    s, d, _, _, _, exits = mk(ranks.reshape(-1) if op.kind == "tree_allreduce" else ranks,
                              float(op.nbytes), 0.0, [], 0)
    flat = ranks.reshape(-1)
    return [[j for j in exits if s[j] == flat[i] or d[j] == flat[i]] for i in range(positions)]


def build(trace: Trace) -> Timeline:
    sc = Scenario(trace.topo)
    tail: Dict[int, int] = {}
    done: List[List[int]] = []

    def awaited(refs):
        return [done[k][j] for k, j in refs]

    for op in trace.ops:
        if isinstance(op, (Compute, StreamWait)):
            after = awaited(op.wait) + ([tail[op.stream]] if op.stream in tail else [])
            lag = float(op.duration) if isinstance(op, Compute) else 0.0
            k = sc.add(Barrier(lag=lag, after=tuple(after)))
            tail[op.stream] = k
            done.append([k])
            continue
        if isinstance(op, Collective) and op.kind in ("tree_allreduce", "hier_allreduce"):
            streams = [int(x) for x in np.ravel(op.streams)]
            rv = sc.add(Barrier(after=tuple(tail[s] for s in streams if s in tail)))
            kind = Tree if op.kind == "tree_allreduce" else Hier
            ranks = np.asarray(op.ranks)
            c = sc.add(kind(ranks.reshape(-1) if kind is Tree else ranks, float(op.nbytes),
                            after=(rv,)))
            per_rank = [tuple((c, j) for j in js)
                        for js in _last_flows_of(op, len(streams))]
        elif isinstance(op, Collective):
            streams = [int(x) for x in op.streams]
            rv = sc.add(Barrier(after=tuple(tail[s] for s in streams if s in tail)))
            if op.kind == "all_to_all":
                c = sc.add(AllToAll(np.asarray(op.ranks), np.asarray(op.nbytes, np.float64),
                                    after=(rv,)))
            else:
                c = sc.add(Ring(op.kind, np.asarray(op.ranks), float(op.nbytes), mode=op.mode,
                                after=(rv,)))
            per_rank = [tuple((c, j) for j in _rank_flows(op, i)) for i in range(len(streams))]
        elif isinstance(op, SendRecv):
            streams = [op.src_stream, op.dst_stream]
            rv = sc.add(Barrier(after=tuple(tail[s] for s in streams if s in tail)))
            c = sc.add(Send(op.src, op.dst, float(op.nbytes), after=(rv,)))
            per_rank = [((c, 0),), ((c, 0),)]
        else:
            raise TypeError(type(op).__name__)
        ids = [sc.add(Barrier(after=a)) for a in per_rank]
        for s, k in zip(streams, ids):
            tail[s] = k
        done.append(ids)
    return Timeline(sc, done, tail)


@dataclass
class TimelineResult:
    finish: np.ndarray            # per flow of the expanded scenario
    op_done: List[np.ndarray]     # per trace operation: completion time per stream
    stream_sync: Dict[int, float]  # what a synchronisation on each stream returns
    events: int
    solves: int


def simulate(trace: Trace, **kw) -> TimelineResult:
    tl = build(trace)
    fs = oflows.expand(tl.scenario)
    r = osim.run_flowset(fs, **kw)
    first = _first_flows(tl.scenario)
    op_done = [r.finish[first[np.asarray(d)]] for d in tl.done_op]
    sync = {s: float(r.finish[first[k]]) for s, k in tl.tail_op.items()}
    return TimelineResult(r.finish, op_done, sync, r.events, r.solves)


def _first_flows(sc: Scenario) -> np.ndarray:
    """Flow id of each scenario operation's first flow (barriers have one)."""
    counts = []
    for op in sc.ops:
        if isinstance(op, Ring):
            p = len(op.ranks)
            counts.append(p if op.mode == "aggregated" else _RING_STEPS[op.kind](p) * p)
        elif isinstance(op, Tree):
            counts.append(4 * (len(op.ranks) - 1))
        elif isinstance(op, Hier):
            m, g = np.asarray(op.ranks).shape
            counts.append(2 * m * g * (g - 1) + g * 2 * (m - 1) * m)
        elif isinstance(op, AllToAll):
            p = len(op.ranks)
            counts.append(p * (p - 1))
        else:
            counts.append(1)
    out = np.zeros(len(counts), np.int64)
    np.cumsum(counts[:-1], out=out[1:])
    return out
