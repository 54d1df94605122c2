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
chained ring, the broadcast flows for a tree, the last phase's last step for
a hierarchical all-reduce, and all flows otherwise.

Double binary tree (the ``Tree`` operation; an NCCL-like alternative to
the ring, cf. the paper's Section 6 on replacing its ring algorithm): with
node numbers u = 1..p for positions u - 1, node u of level l (the number of
trailing zero bits of u) has, for l >= 1, a left child u - 2^(l-1) and a
right child u + 2^j for the largest j < l with u + 2^j <= p (if any); the
root is the largest power of two <= p; odd nodes are leaves (a parent's
level always exceeds its child's).  Tree A puts position u - 1 at node u,
tree B (its mirror) position p - u.  Per tree and edge (child c, parent q):
a reduce flow c -> q of half the bytes after the reduce flows into c (a
leaf: after the operation's predecessors, with its lag), and a broadcast
flow q -> c after the broadcast flow into q (q the root: after the reduce
flows into the root).  Reduce flows are laid out by child level, lowest
first, broadcast flows highest first, each level by child node.

Hierarchical all-reduce (``Hier``, ranks m x g): phase 1, per server, a
chained ring reduce-scatter of chunks S/g over its g ranks; phase 2, per
local position j, a chained ring all-reduce of chunks S/(g*m) over the m
servers; phase 3, per server, a chained ring all-gather of chunks S/g.  The
first step of a phase out of rank (s, i) waits for that rank's previous
phase: the previous phase's last-step flows out of and into it.  Phases
of one rank (g = 1: phases 1 and 3; m = 1: phase 2) are left out.

Latency: a flow's latency is the sum over its path, in path order, of its
links' latencies.
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from workloads.program import AllToAll, Barrier, Hier, PathFlow, Ring, Send, Tree
from .topology import Fabric

_STEPS = {"allreduce": lambda p: 2 * (p - 1),
          "reduce_scatter": lambda p: p - 1,
          "all_gather": lambda p: p - 1}


def _level(u: int) -> int:
    return (u & -u).bit_length() - 1


def btree(p: int):
    """The binary tree over nodes 1..p described above: (root, edges (c, q)
    ordered by child c, children of each node)."""
    kids = {u: [] for u in range(1, p + 1)}
    for u in range(2, p + 1, 2):
        lvl = (u & -u).bit_length() - 1
        kids[u].append(u - (1 << (lvl - 1)))
        for j in range(lvl - 1, -1, -1):
            if u + (1 << j) <= p:
                kids[u].append(u + (1 << j))
                break
    parent = {c: q for q, cs in kids.items() for c in cs}
    root = 1 << (p.bit_length() - 1)
    return root, sorted(parent.items()), kids


def _tree_flows(ranks, nbytes, lag, pred, first):
    """Flows of a double binary tree all-reduce (see the module notes)."""
    p = len(ranks)
    root, edges, kids = btree(p)
    red = sorted(edges, key=lambda e: (_level(e[0]), e[0]))    # leaves first
    bc = sorted(edges, key=lambda e: (-_level(e[0]), e[0]))    # top first
    rslot = {c: k for k, (c, _) in enumerate(red)}
    bslot = {c: k for k, (c, _) in enumerate(bc)}
    half = float(nbytes) / 2.0
    s, d, nb, st, deps = [], [], [], [], []
    exits = []
    for t in range(2):
        pos = (lambda u: u - 1) if t == 0 else (lambda u: p - u)
        red0 = first + t * 2 * (p - 1)
        bc0 = red0 + (p - 1)
        for c, q in red:
            s.append(ranks[pos(c)])
            d.append(ranks[pos(q)])
            into = [red0 + rslot[x] for x in kids[c]]
            deps.append(into if into else list(pred))
            st.append(0.0 if into else float(lag))
        for c, q in bc:
            s.append(ranks[pos(q)])
            d.append(ranks[pos(c)])
            deps.append([red0 + rslot[x] for x in kids[root]] if q == root else [bc0 + bslot[q]])
            st.append(0.0)
            exits.append(bc0 + bslot[c])
        nb.extend([half] * (2 * (p - 1)))
    return s, d, nb, st, deps, exits


def _hier_flows(ranks, nbytes, lag, pred, first):
    """Flows of a hierarchical all-reduce over an m x g rank array."""
    R = np.asarray(ranks)
    m, g = R.shape
    S = float(nbytes)
    s, d, nb, st, deps = [], [], [], [], []
    done = {}  # (server, local) -> the previous phase's flows out of and into the rank

    def start_deps(a, i):
        return done[(a, i)] if (a, i) in done else list(pred)

    def lag_of(a, i):
        return 0.0 if (a, i) in done else float(lag)

    def server_ring(steps_of, chunk):
        nonlocal first
        new_done = {}
        for a in range(m):
            base = first
            for k in range(steps_of):
                for i in range(g):
                    s.append(R[a, i])
                    d.append(R[a, (i + 1) % g])
                    nb.append(chunk)
                    if k == 0:
                        deps.append(start_deps(a, i))
                        st.append(lag_of(a, i))
                    else:
                        deps.append([base + (k - 1) * g + (i - 1) % g])
                        st.append(0.0)
            last = base + (steps_of - 1) * g
            for i in range(g):
                new_done[(a, i)] = [last + i, last + (i - 1) % g]
            first += steps_of * g
        done.clear()
        done.update(new_done)

    if g > 1:
        server_ring(g - 1, S / g)                      # reduce-scatter
    if m > 1:
        new_done = {}
        for j in range(g):                               # ring all-reduce per position
            base = first
            steps = 2 * (m - 1)
            for k in range(steps):
                for a in range(m):
                    s.append(R[a, j])
                    d.append(R[(a + 1) % m, j])
                    nb.append(S / (g * m))
                    if k == 0:
                        deps.append(start_deps(a, j))
                        st.append(lag_of(a, j))
                    else:
                        deps.append([base + (k - 1) * m + (a - 1) % m])
                        st.append(0.0)
            last = base + (steps - 1) * m
            for a in range(m):
                new_done[(a, j)] = [last + a, last + (a - 1) % m]
            first += steps * m
        done.clear()
        done.update(new_done)
    if g > 1:
        server_ring(g - 1, S / g)                      # all-gather
    exits = sorted({x for v in done.values() for x in v})
    return s, d, nb, st, deps, exits


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
    lat: np.ndarray = None  # [F] f64 path latency (None: all zero)

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
        elif isinstance(op, (Tree, Hier)):
            ranks = np.asarray(op.ranks, dtype=np.int64)
            mk = _tree_flows if isinstance(op, Tree) else _hier_flows
            fl = mk(ranks, op.nbytes, op.lag, pred, first)
            s, d, nb, st, dl, ex = fl
            n = len(nb)
            cnt = np.array([len(x) for x in dl], np.int64)
            ids = (np.concatenate([np.asarray(x, np.int64) for x in dl]) if n
                   else np.zeros(0, np.int64))
            ex = np.asarray(ex, np.int64)
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
    lat = None
    if np.any(fab.lat != 0.0):
        # summed in path order: ((0 + l_1) + l_2) + ...
        lens = np.diff(path_off)
        lat = np.zeros(nflows)
        for k in range(int(lens.max()) if nflows else 0):
            has = lens > k
            lat[has] = lat[has] + fab.lat[links[path_off[:-1][has] + k]]
    return FlowSet(fab.cap, src, dst, nbytes, start, path_off, links.astype(np.int32),
                   dep_off, dep_ids, lat)
