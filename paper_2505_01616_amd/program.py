"""Feeds a workload description into a libnetsim handle.

Marshalling only: topology parameters become ``netsim_topology`` structs,
ring, all-to-all, tree and hierarchical all-reduce operations become
``netsim_add_ring`` / ``netsim_add_all_to_all`` / ``netsim_add_tree_allreduce``
/ ``netsim_add_hier_allreduce`` calls (the library decomposes and routes
them), link latencies ``netsim_topology`` fields or ``netsim_set_link_latency``,
and point-to-point sends, barriers and explicit-path flows are batched into
``netsim_add_flows`` calls.  The description objects are duck-typed (any
object with the attributes of ``workloads.program``).
"""

from __future__ import annotations

import math
from dataclasses import dataclass
from typing import List

import numpy as np

from . import netsim as ns

_KINDS = {"leaf_spine": ns.TOPO_LEAF_SPINE, "rail": ns.TOPO_RAIL, "fat_tree": ns.TOPO_FAT_TREE}
_RING = {"allreduce": ns.RING_ALLREDUCE, "reduce_scatter": ns.RING_REDUCE_SCATTER,
         "all_gather": ns.RING_ALL_GATHER}
_MODE = {"chained": ns.MODE_CHAINED, "flat": ns.MODE_FLAT, "aggregated": ns.MODE_AGGREGATED}


def topology_struct(t, keep: list) -> ns.netsim_topology:
    d = ns.netsim_topology()
    d.kind = _KINDS[t.kind]
    d.servers, d.gpus_per_server, d.servers_per_leaf = t.servers, t.gpus_per_server, t.servers_per_leaf
    d.spines, d.pods, d.edges_per_pod = t.spines, t.pods, t.edges_per_pod
    d.aggs_per_pod, d.agg_uplinks = t.aggs_per_pod, t.agg_uplinks
    d.nvlink_Bps, d.nic_Bps, d.fabric_Bps = t.nvlink_Bps, t.nic_Bps, t.fabric_Bps
    d.ecmp_seed = int(t.ecmp_seed) & ((1 << 64) - 1)
    deg = np.ascontiguousarray(t.degraded, dtype=np.int64)
    keep.append(deg)
    d.num_degraded = len(deg)
    if len(deg):
        d.degraded_cables = deg.ctypes.data_as(ns.ctypes.POINTER(ns.ctypes.c_int64))
    d.degraded_Bps = t.degraded_Bps
    d.fabric_latency_s = float(getattr(t, "fabric_latency_s", 0.0))
    d.nvlink_latency_s = float(getattr(t, "nvlink_latency_s", 0.0))
    return d


@dataclass
class Loaded:
    handle: int
    num_scenarios: int
    first_flow: List[int]     # first flow id of each scenario
    num_flows: List[int]

    def close(self):
        ns.netsim_destroy(self.handle)
        self.handle = 0


class _Batch:
    """Consecutive single-flow operations, added with one call."""

    def __init__(self, h, scen, explicit):
        self.h, self.scen, self.explicit = h, scen, explicit
        self.reset()

    def reset(self):
        self.src, self.dst, self.nb, self.st = [], [], [], []
        self.doff, self.dids = [0], []
        self.poff, self.plink = [0], []

    def __len__(self):
        return len(self.nb)

    def add(self, src, dst, nbytes, lag, deps, path=()):
        self.src.append(src)
        self.dst.append(dst)
        self.nb.append(float(nbytes))
        self.st.append(float(lag))
        self.dids.extend(int(x) for x in deps)
        self.doff.append(len(self.dids))
        self.plink.extend(path)
        self.poff.append(len(self.plink))

    def flush(self):
        if not self.nb:
            return
        kw = {}
        if self.explicit:
            kw = dict(path_off=np.array(self.poff, np.int64), path_link=np.array(self.plink, np.int32))
        ns.netsim_add_flows(self.h, self.scen, np.array(self.nb), np.array(self.st),
                            src=np.array(self.src, np.int32), dst=np.array(self.dst, np.int32),
                            dep_off=np.array(self.doff, np.int64),
                            dep_ids=np.array(self.dids, np.int64), **kw)
        self.reset()


def load_program(program, opt: ns.netsim_options = None) -> Loaded:
    scs = program.scenarios
    explicit = [sc.topo.kind == "explicit" for sc in scs]
    if any(explicit) and not all(explicit):
        raise ValueError("a program mixes explicit and built-in topologies")
    keep = []
    if explicit[0]:
        caps = [np.asarray(sc.topo.capacities, np.float64) for sc in scs]
        off = np.zeros(len(scs) + 1, np.int64)
        np.cumsum([len(c) for c in caps], out=off[1:])
        h = ns.netsim_create(off, np.concatenate(caps), opt)
        for s, sc in enumerate(scs):
            if getattr(sc.topo, "latencies", None) is not None:
                ns.netsim_set_link_latency(h, s, sc.topo.latencies)
    else:
        h = ns.netsim_create_topology([topology_struct(sc.topo, keep) for sc in scs], opt)
    first_flow, nflows = [], []
    try:
        for s, sc in enumerate(scs):
            next_id = ns.netsim_counts(h)[0]
            first_flow.append(next_id)
            batch = _Batch(h, s, explicit[0])
            exits, firsts = [], []
            for op in sc.ops:
                after = []
                for a in op.after:   # an operation's exits, or one flow (op, j) of it
                    if isinstance(a, tuple):
                        after.append(firsts[a[0]] + a[1])
                    else:
                        after.extend(exits[a])
                name = type(op).__name__
                if name in ("Send", "Barrier", "PathFlow"):
                    fid = next_id + len(batch)
                    firsts.append(fid)
                    if name == "Send":
                        batch.add(op.src, op.dst, op.nbytes, op.lag, after)
                    elif name == "Barrier":
                        batch.add(-1, -1, 0.0, op.lag, after)
                    else:
                        batch.add(-1, -1, op.nbytes, op.lag, after, path=list(op.path))
                    exits.append([fid])
                    continue
                batch.flush()
                next_id = ns.netsim_counts(h)[0]
                if name == "Ring":
                    first, n = ns.netsim_add_ring(h, s, _RING[op.kind], _MODE[op.mode], op.ranks,
                                                  op.nbytes, op.lag, after)
                elif name == "AllToAll":
                    first, n = ns.netsim_add_all_to_all(h, s, op.ranks, op.nbytes, op.lag, after)
                elif name == "Tree":
                    first, n = ns.netsim_add_tree_allreduce(h, s, op.ranks, op.nbytes, op.lag, after)
                elif name == "Hier":
                    first, n = ns.netsim_add_hier_allreduce(h, s, op.ranks, op.nbytes, op.lag, after)
                else:
                    raise TypeError(f"unknown operation {name}")
                # what a later operation waits for: the library's exit flows
                firsts.append(first)
                exits.append(ns.netsim_last_exits(h).tolist())
                next_id = first + n
            batch.flush()
            nflows.append(ns.netsim_counts(h)[0] - first_flow[-1])
    except Exception:
        ns.netsim_destroy(h)
        raise
    return Loaded(h, len(scs), first_flow, nflows)


def run_program(program, opt: ns.netsim_options = None, stream=None):
    """Loads, runs and returns (finish per scenario, stats)."""
    ld = load_program(program, opt)
    try:
        ns.netsim_run(ld.handle, stream)
        fin = ns.netsim_get_finish(ld.handle)
        stats = ns.netsim_get_stats(ld.handle)
    finally:
        ld.close()
    out = [fin[f:f + n] for f, n in zip(ld.first_flow, ld.num_flows)]
    return out, stats


def default_options(**kw) -> ns.netsim_options:
    return ns.make_options(**kw)


__all__ = ["load_program", "run_program", "Loaded", "default_options", "math"]
