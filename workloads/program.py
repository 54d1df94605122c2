"""Workload description shared by the simulator binding and the oracle.

A ``Program`` is a list of independent ``Scenario`` objects.  A scenario is
a cluster topology (given by its parameters, not by its links) plus an
ordered list of communication operations.  Each side of a parity check
turns the same program into links, routes and flows with its own code;
nothing here decomposes, routes or simulates.

Operations and their dependencies:

* ``Ring``      -- a ring collective (all-reduce, reduce-scatter, all-gather)
                   over ``ranks`` of ``nbytes`` total, in one of three
                   decomposition modes ("chained", "flat", "aggregated").
* ``AllToAll``  -- one flow per ordered pair of distinct ranks, sizes from a
                   p x p matrix (row = sender).
* ``Tree``      -- a double binary tree all-reduce of ``nbytes`` over ``ranks``:
                   two binary trees over the rank positions, each carrying
                   half the bytes, reduced up and broadcast down.
* ``Hier``      -- a hierarchical all-reduce over ``ranks`` given as an m x g
                   array (row = server, g ranks each): reduce-scatter inside
                   every server, a ring all-reduce across the servers for
                   each local position, all-gather inside every server.
* ``Send``      -- one point-to-point flow.
* ``Barrier``   -- a zero-byte flow with no route; completes as soon as it
                   is released.
* ``PathFlow``  -- one flow over an explicit list of link ids (only on
                   ``explicit`` topologies).

``after`` lists earlier operations of the same scenario: an index names
an operation (its first flows wait for its last flows), a pair (index, j)
names flow j of that operation (flows numbered as the operation lays them
out: a ring step-major, an all-to-all row-major without the diagonal, a
tree as tree A reduce, tree A broadcast, tree B reduce, tree B broadcast, a
hierarchical all-reduce as its three phases in order).  The
first flows of an operation wait for everything in ``after``; ``lag``
seconds are added after that (with no ``after`` the lag is the absolute
start time).
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Union

import numpy as np

MiB = float(1 << 20)
GiB = float(1 << 30)


def gbit(x: float) -> float:
    """x Gb/s in bytes per second."""
    return x * 1e9 / 8.0


@dataclass
class Topology:
    """Cluster fabric parameters.

    kind:
      * ``leaf_spine`` -- each server's GPUs hang off one leaf (ToR) through
        one NIC per GPU; ``servers_per_leaf`` servers share a leaf; every
        leaf has one cable to each of ``spines`` spines.
      * ``rail``       -- rail-optimised: local GPU g of the
        ``servers_per_leaf`` servers of a group shares leaf (g, group);
        every leaf has one cable to each spine.
      * ``fat_tree``   -- three tiers: ``pods`` pods of ``edges_per_pod``
        edge and ``aggs_per_pod`` aggregation switches; ``servers_per_leaf``
        servers per edge switch; every edge switch has one cable to every
        aggregation switch of its pod; aggregation switch a of every pod has
        ``agg_uplinks`` cables, to cores a*agg_uplinks .. +agg_uplinks-1.
      * ``explicit``   -- links given by ``capacities``; flows carry paths.

    Inside a server every ordered GPU pair has its own link (``nvlink_Bps``).
    ``fabric_Bps`` is the rate of every switch-to-switch cable.
    ``degraded`` lists cable indices (canonical cable order) whose two
    directions run at ``degraded_Bps``.
    Latency: every NVLink link takes ``nvlink_latency_s``, every other link
    ``fabric_latency_s`` (explicit topologies: ``latencies`` per link, or
    none); a flow finishes its path's summed latency after its last byte
    leaves.
    """

    kind: str
    servers: int = 0
    gpus_per_server: int = 8
    servers_per_leaf: int = 1
    spines: int = 0
    pods: int = 0
    edges_per_pod: int = 0
    aggs_per_pod: int = 0
    agg_uplinks: int = 0
    nvlink_Bps: float = 900e9
    nic_Bps: float = gbit(400)
    fabric_Bps: float = gbit(800)
    ecmp_seed: int = 0
    degraded: np.ndarray = field(default_factory=lambda: np.zeros(0, np.int64))
    degraded_Bps: float = 0.0
    capacities: Optional[np.ndarray] = None
    fabric_latency_s: float = 0.0
    nvlink_latency_s: float = 0.0
    latencies: Optional[np.ndarray] = None

    @property
    def endpoints(self) -> int:
        return self.servers * self.gpus_per_server

    def num_cables(self) -> int:
        """Number of switch cables (NIC cables first); NVLink pairs excluded."""
        n = self.endpoints
        if self.kind == "leaf_spine":
            return n + (self.servers // self.servers_per_leaf) * self.spines
        if self.kind == "rail":
            leaves = self.gpus_per_server * (self.servers // self.servers_per_leaf)
            return n + leaves * self.spines
        if self.kind == "fat_tree":
            p, e, a, u = self.pods, self.edges_per_pod, self.aggs_per_pod, self.agg_uplinks
            return n + p * e * a + p * a * u
        return 0


@dataclass
class Ring:
    kind: str            # "allreduce" | "reduce_scatter" | "all_gather"
    ranks: np.ndarray
    nbytes: float
    mode: str = "chained"  # "chained" | "flat" | "aggregated"
    lag: float = 0.0
    after: Sequence[int] = ()


@dataclass
class AllToAll:
    ranks: np.ndarray
    nbytes: np.ndarray   # p x p, row = sender; diagonal ignored
    lag: float = 0.0
    after: Sequence[int] = ()


@dataclass
class Tree:
    ranks: np.ndarray
    nbytes: float
    lag: float = 0.0
    after: Sequence[int] = ()


@dataclass
class Hier:
    ranks: np.ndarray    # m x g: row s holds the g ranks of server s
    nbytes: float
    lag: float = 0.0
    after: Sequence[int] = ()


@dataclass
class Send:
    src: int
    dst: int
    nbytes: float
    lag: float = 0.0
    after: Sequence[int] = ()


@dataclass
class Barrier:
    lag: float = 0.0
    after: Sequence[int] = ()


@dataclass
class PathFlow:
    path: Sequence[int]
    nbytes: float
    lag: float = 0.0
    after: Sequence[int] = ()


Op = Union[Ring, AllToAll, Tree, Hier, Send, Barrier, PathFlow]


@dataclass
class Scenario:
    topo: Topology
    ops: List[Op] = field(default_factory=list)

    def add(self, op: Op) -> int:
        for a in op.after:
            k = a[0] if isinstance(a, tuple) else a
            if not (0 <= k < len(self.ops)) or (isinstance(a, tuple) and a[1] < 0):
                raise ValueError("'after' must name an earlier operation")
        self.ops.append(op)
        return len(self.ops) - 1


@dataclass
class Program:
    name: str
    scenarios: List[Scenario] = field(default_factory=list)
    notes: str = ""
