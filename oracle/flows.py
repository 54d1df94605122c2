"""Oracle side: communication operations -> flows.

TEST INFRASTRUCTURE (see ``oracle/__init__.py``).

The paper models each collective by the communication pattern NCCL would
use, all-reduce as a ring (Section 4.1, netsim description; Section 6
describes it as a plain ring algorithm).  Reading taken here, for a ring over
ranks r_0..r_{p-1} of S bytes in total:

  * all-reduce has 2(p-1) steps, reduce-scatter and all-gather p-1 steps;
  * in every step position i sends S/p bytes (fp64 division) from r_i to
    r_{(i+1) mod p};
  * "chained": the step-k send out of position i waits for the step-(k-1)
    send into position i (the one from position i-1); the first step waits
    for the operation's predecessors;
  * "flat": every step's flow is released together;
  * "aggregated": one flow per ring edge carrying steps*(S/p) bytes.

Flow numbering inside a ring: step-major, id = first + k*p + i.  An
all-to-all over p ranks gives flows (i, j), j != i, in row-major order.
Zero-byte flows get no route.  The last flows of an operation (what a
later operation's ``after`` waits for) are the last step's p flows for a
chained ring and all flows otherwise.
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from workloads.program import AllToAll, Barrier, PathFlow, Ring, Send
from .topology import Fabric

_STEPS = {"allreduce": lambda p: 2 * (p - 1),
          "reduce_scatter": lambda p: p - 1,
          "all_gather": lambda p: p - 1}


@dataclass
class FlowSet:
    """Flat arrays for one scenario."""
    cap: np.ndarray        # [L] f64 link capacities (B/s)
    src: np.ndarray        # [F] i64 (-1 for barriers / explicit paths)
    dst: np.ndarray        # [F] i64
    nbytes: np.ndarray     # [F] f64
    start: np.ndarray      # [F] f64 lag (absolute start when no deps)
    path_off: np.ndarray   # [F+1] i64
    path_link: np.ndarray  # [nnz] i32
    dep_off: np.ndarray    # [F+1] i64
    dep_ids: np.ndarray    # [ndeps] i64

    @property
    def F(self):
        return len(self.nbytes)

    @property
    def L(self):
        return len(self.cap)


def expand(scenario) -> FlowSet:
    fab = Fabric(scenario.topo)
    srcs, dsts, nbs, starts = [], [], [], []
    dep_lists = []          # per op: (counts array, flat ids array)
    explicit_paths = {}     # flow id -> list of links (explicit topologies)
    exits = []
    firsts = []
    nflows = 0
    for op in scenario.ops:
        # an entry of `after` names an operation (its exits) or one flow of it
        pred = (np.concatenate([np.array([firsts[a[0]] + a[1]]) if isinstance(a, tuple) else exits[a]
                                for a in op.after]).astype(np.int64)
                if len(op.after) else np.zeros(0, np.int64))
        first = nflows
        firsts.append(first)
        if isinstance(op, Ring):
            ranks = np.asarray(op.ranks, dtype=np.int64)
            p = len(ranks)
            steps = _STEPS[op.kind](p)
            chunk = float(op.nbytes) / float(p)
            nxt = np.roll(ranks, -1)
            if op.mode == "aggregated":
                n = p
                s, d = ranks, nxt
                nb = np.full(p, float(steps) * chunk)
                st = np.full(p, float(op.lag))
                cnt = np.full(p, len(pred), np.int64)
                ids = np.tile(pred, p)
                ex = first + np.arange(p, dtype=np.int64)
            else:
                n = steps * p
                s = np.tile(ranks, steps)
                d = np.tile(nxt, steps)
                nb = np.full(n, chunk)
                if op.mode == "flat":
                    st = np.full(n, float(op.lag))
                    cnt = np.full(n, len(pred), np.int64)
                    ids = np.tile(pred, n)
                    ex = first + np.arange(n, dtype=np.int64)
                elif op.mode == "chained":
                    st = np.zeros(n)
                    st[:p] = float(op.lag)
                    cnt = np.ones(n, np.int64)
                    cnt[:p] = len(pred)
                    k = np.arange(1, steps, dtype=np.int64)[:, None]
                    i = np.arange(p, dtype=np.int64)[None, :]
                    prev = first + (k - 1) * p + (i - 1) % p   # flow into position i
                    ids = np.concatenate([np.tile(pred, p), prev.reshape(-1)])
                    ex = first + (steps - 1) * p + np.arange(p, dtype=np.int64)
                else:
                    raise ValueError(op.mode)
        elif isinstance(op, AllToAll):
            ranks = np.asarray(op.ranks, dtype=np.int64)
            p = len(ranks)
            ii, jj = np.meshgrid(np.arange(p), np.arange(p), indexing="ij")
            off = ii != jj
            s, d = ranks[ii[off]], ranks[jj[off]]
            nb = np.asarray(op.nbytes, dtype=np.float64)[ii[off], jj[off]]
            n = len(s)
            st = np.full(n, float(op.lag))
            cnt = np.full(n, len(pred), np.int64)
            ids = np.tile(pred, n)
            ex = first + np.arange(n, dtype=np.int64)
        elif isinstance(op, (Send, Barrier, PathFlow)):
            n = 1
            if isinstance(op, Send):
                s, d, nb = np.array([op.src]), np.array([op.dst]), np.array([float(op.nbytes)])
            elif isinstance(op, Barrier):
                s, d, nb = np.array([-1]), np.array([-1]), np.array([0.0])
            else:
                s, d, nb = np.array([-1]), np.array([-1]), np.array([float(op.nbytes)])
                explicit_paths[first] = list(op.path)
            st = np.array([float(op.lag)])
            cnt = np.array([len(pred)], np.int64)
            ids = pred
            ex = np.array([first], np.int64)
        else:
            raise TypeError(type(op))
        srcs.append(np.asarray(s, np.int64))
        dsts.append(np.asarray(d, np.int64))
        nbs.append(np.asarray(nb, np.float64))
        starts.append(np.asarray(st, np.float64))
        dep_lists.append((cnt, ids))
        exits.append(ex)
        nflows += n
    if nflows == 0:
        z = np.zeros(0, np.int64)
        return FlowSet(fab.cap, z, z, np.zeros(0), np.zeros(0), np.zeros(1, np.int64),
                       np.zeros(0, np.int32), np.zeros(1, np.int64), z)
    src = np.concatenate(srcs)
    dst = np.concatenate(dsts)
    nbytes = np.concatenate(nbs)
    start = np.concatenate(starts)
    dep_off = np.zeros(nflows + 1, np.int64)
    np.cumsum(np.concatenate([c for c, _ in dep_lists]), out=dep_off[1:])
    dep_ids = np.concatenate([i for _, i in dep_lists]).astype(np.int64)
    # routes
    routed = (nbytes > 0) & (src >= 0)
    lens = np.zeros(nflows, np.int64)
    links = np.zeros(0, np.int32)
    if fab.kind == "explicit":
        for f, pth in explicit_paths.items():
            if nbytes[f] > 0:
                lens[f] = len(pth)
        path_off = np.zeros(nflows + 1, np.int64)
        np.cumsum(lens, out=path_off[1:])
        links = np.zeros(int(path_off[-1]), np.int32)
        for f, pth in explicit_paths.items():
            if nbytes[f] > 0:
                links[path_off[f]:path_off[f + 1]] = pth
    else:
        idx = np.nonzero(routed)[0]
        r_off, r_link = fab.route(src[idx], dst[idx])
        lens[idx] = np.diff(r_off)
        path_off = np.zeros(nflows + 1, np.int64)
        np.cumsum(lens, out=path_off[1:])
        links = r_link
    return FlowSet(fab.cap, src, dst, nbytes, start, path_off, links.astype(np.int32),
                   dep_off, dep_ids)
