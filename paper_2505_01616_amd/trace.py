"""Feeds a trace of stream operations into a libnetsim handle through the
event-queue front end (``netsim_stream_*``).

Marshalling only: each computation, event wait, collective and send/recv of
the trace becomes one library call; the library keeps the streams' tails,
lays out rendezvous and completion flows, decomposes and routes.  The trace
objects are duck-typed (the attributes of ``workloads.trace``).
"""

from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, List

import numpy as np

from . import netsim as ns
from .program import _MODE, _RING, topology_struct


@dataclass
class LoadedTrace:
    handle: int
    done: List[np.ndarray]       # per operation: completion flow id per stream
    streams: List[int]           # every stream the trace uses

    def close(self):
        ns.netsim_destroy(self.handle)
        self.handle = 0

    def tails(self) -> Dict[int, int]:
        return {s: ns.netsim_stream_tail(self.handle, 0, s) for s in self.streams}


def load_trace(trace, opt: ns.netsim_options = None) -> LoadedTrace:
    keep = []
    h = ns.netsim_create_topology([topology_struct(trace.topo, keep)], opt)
    done: List[np.ndarray] = []
    seen = set()
    try:
        for op in trace.ops:
            name = type(op).__name__
            wait = [int(done[k][j]) for k, j in getattr(op, "wait", ())]
            if name == "Compute":
                done.append(np.array([ns.netsim_stream_compute(h, 0, op.stream, op.duration, wait)]))
                seen.add(int(op.stream))
            elif name == "StreamWait":
                ns.netsim_stream_wait(h, 0, op.stream, wait)
                done.append(np.array([ns.netsim_stream_tail(h, 0, op.stream)]))
                seen.add(int(op.stream))
            elif name == "Collective" and op.kind == "tree_allreduce":
                done.append(ns.netsim_stream_tree_allreduce(h, 0, op.ranks, op.streams, op.nbytes))
                seen.update(int(s) for s in op.streams)
            elif name == "Collective" and op.kind == "hier_allreduce":
                done.append(ns.netsim_stream_hier_allreduce(h, 0, op.ranks, op.streams, op.nbytes))
                seen.update(int(s) for s in np.ravel(op.streams))
            elif name == "Collective":
                if op.kind == "all_to_all":
                    d = ns.netsim_stream_all_to_all(h, 0, op.ranks, op.streams, op.nbytes)
                else:
                    d = ns.netsim_stream_ring(h, 0, _RING[op.kind], _MODE[op.mode], op.ranks,
                                              op.streams, op.nbytes)
                done.append(d)
                seen.update(int(s) for s in op.streams)
            elif name == "SendRecv":
                a = ns.netsim_stream_send(h, 0, op.src, op.src_stream, op.dst, op.dst_stream,
                                          op.nbytes)
                done.append(np.array([a, ns.netsim_stream_tail(h, 0, op.dst_stream)]))
                seen.update((int(op.src_stream), int(op.dst_stream)))
            else:
                raise TypeError(f"unknown trace operation {name}")
    except Exception:
        ns.netsim_destroy(h)
        raise
    return LoadedTrace(h, done, sorted(seen))


def run_trace(trace, opt: ns.netsim_options = None, stream=None):
    """Loads and runs a trace; returns (finish per flow, completion per
    operation and stream, synchronisation time per stream, stats)."""
    ld = load_trace(trace, opt)
    try:
        ns.netsim_run(ld.handle, stream)
        fin = ns.netsim_get_finish(ld.handle)
        stats = ns.netsim_get_stats(ld.handle)
        sync = {s: float(fin[f]) for s, f in ld.tails().items()}
    finally:
        ld.close()
    return fin, [fin[d] for d in ld.done], sync, stats
