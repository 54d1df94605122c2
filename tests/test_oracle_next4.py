"""Pins of the oracle's richer collectives and per-link latency.

* The double binary tree: both trees span every rank with p - 1 edges, each
  flow carries half the bytes, and (p even) every leaf of tree A is interior
  in tree B; inside one server (a link per ordered GPU pair) trees of 2, 4
  and 8 ranks share no link, so each flow ends where the longest path
  through the dependencies puts it and the whole tree takes
  log2(p) * S / B_nvlink.
* The hierarchical all-reduce: on a single-leaf fabric (no flow shares a
  link) it takes 2(g-1)/g * S / B_nvlink + 2(m-1)/(g*m) * S / B_nic, and
  it reduces to the plain ring when g = 1 or m = 1.
* Latency: a flow finishes its path's latency after its last byte; the
  link is freed when the last byte leaves (two flows sharing a link); a
  chained ring pays one path latency per step; a flow after several
  predecessors starts after the latest finish, not after the last one to
  send its last byte; the fp64 oracle agrees with the exact-rational
  twin on random cases with latencies.
"""

import math

import numpy as np
import pytest

from oracle import flows as oflows
from oracle import plain
from oracle import sim as osim
from tests.helpers import rel_err
from workloads.program import Hier, MiB, PathFlow, Ring, Scenario, Send, Topology, Tree, gbit

NV = 900e9
NIC = gbit(400)


def _server(p=8, **kw):
    return Topology(kind="leaf_spine", servers=1, gpus_per_server=p, servers_per_leaf=1, spines=1,
                    nvlink_Bps=NV, nic_Bps=NIC, fabric_Bps=gbit(400), **kw)


def _one_leaf(m, g, **kw):
    return Topology(kind="leaf_spine", servers=m, gpus_per_server=g, servers_per_leaf=m, spines=1,
                    nvlink_Bps=NV, nic_Bps=NIC, fabric_Bps=gbit(400), ecmp_seed=5, **kw)


def _longest_path(fs):
    """Finish of every flow assuming none shares a link while sending
    (checked): start = latest predecessor finish + lag, then bytes over the
    narrowest link of the path, then the path latency."""
    fin = np.zeros(fs.F)
    busy = {}
    for f in range(fs.F):
        deps = fs.dep_ids[fs.dep_off[f]:fs.dep_off[f + 1]]
        t0 = (max(fin[deps]) if len(deps) else 0.0) + fs.start[f]
        links = fs.path_link[fs.path_off[f]:fs.path_off[f + 1]]
        dur = fs.nbytes[f] / min(fs.cap[links]) if len(links) else 0.0
        for l in map(int, links):
            for a, b in busy.get(l, []):
                assert t0 + dur <= a or t0 >= b, "a link carries two flows at once"
            busy.setdefault(l, []).append((t0, t0 + dur))
        fin[f] = t0 + dur + (fs.lat[f] if fs.lat is not None else 0.0)
    return fin


# ------------------------------------------------------------------ tree
@pytest.mark.parametrize("p", [2, 3, 5, 8, 13, 64, 100])
def test_tree_structure(p):
    root, edges, kids = oflows.btree(p)
    assert len(edges) == p - 1 and root == 1 << (p.bit_length() - 1)
    par = dict(edges)
    for u in range(1, p + 1):      # every node reaches the root
        x, d = u, 0
        while x != root:
            x, d = par[x], d + 1
            assert d < p
    sc = Scenario(_server(8) if p <= 8 else _one_leaf(p // 4 + 1, 4))
    ranks = np.arange(p)
    sc.add(Tree(ranks, 8 * MiB))
    fs = oflows.expand(sc)
    assert fs.F == 4 * (p - 1)
    assert np.all(fs.nbytes == 4 * MiB)
    # each tree and phase touches every rank
    for b in range(4):
        seg = slice(b * (p - 1), (b + 1) * (p - 1))
        assert set(fs.src[seg]) | set(fs.dst[seg]) == set(range(p))
    # dependencies, read off the flows' ends: a reduce flow out of x waits for
    # the reduce flows into x (a leaf: nothing); a broadcast flow out of x
    # waits for the broadcast flow into x (the root: every reduce flow into it)
    for t in range(2):
        red = range(2 * t * (p - 1), (2 * t + 1) * (p - 1))
        bc = range((2 * t + 1) * (p - 1), (2 * t + 2) * (p - 1))
        deps = lambda f: sorted(fs.dep_ids[fs.dep_off[f]:fs.dep_off[f + 1]].tolist())
        for f in red:
            assert deps(f) == sorted(h for h in red if fs.dst[h] == fs.src[f])
        root_rank = set(fs.src[list(bc)]) - set(fs.dst[list(bc)])
        assert len(root_rank) == 1
        for f in bc:
            if fs.src[f] in root_rank:
                assert deps(f) == sorted(h for h in red if fs.dst[h] == fs.src[f])
            else:
                assert deps(f) == [h for h in bc if fs.dst[h] == fs.src[f]]
    if p % 2 == 0:   # leaves of tree A (odd nodes) are interior in the mirror tree B
        leaves_a = {u - 1 for u in range(1, p + 1, 2)}
        senders_b_bcast = set(fs.src[3 * (p - 1):])
        assert leaves_a <= senders_b_bcast


@pytest.mark.parametrize("p", [2, 4, 8])
def test_tree_inside_a_server(p):
    sc = Scenario(_server(8))
    S = 64 * MiB
    sc.add(Tree(np.arange(p), S))
    fs = oflows.expand(sc)
    want = _longest_path(fs)
    r = osim.run_flowset(fs)
    assert rel_err(r.finish, want) < 1e-12
    assert math.isclose(r.makespan, math.log2(p) * S / NV, rel_tol=1e-12)


def test_tree_after_and_lag():
    """The leaves' reduce flows wait for the predecessors plus the lag."""
    sc = Scenario(_server(8))
    sc.add(Send(0, 1, 9 * MiB))
    sc.add(Tree(np.arange(4), 16 * MiB, lag=1e-5, after=(0,)))
    fs = oflows.expand(sc)
    r = osim.run_flowset(fs)
    t0 = 9 * MiB / NV + 1e-5
    assert math.isclose(r.makespan, t0 + 2 * 16 * MiB / NV, rel_tol=1e-12)
    assert rel_err(r.finish, _longest_path(fs)) < 1e-12


# ------------------------------------------------------------ hierarchical
@pytest.mark.parametrize("m,g", [(4, 4), (3, 8), (2, 2), (5, 1), (1, 6)])
def test_hier_closed_form(m, g):
    S = 96 * MiB
    sc = Scenario(_one_leaf(m, g))
    sc.add(Hier(np.arange(m * g).reshape(m, g), S))
    fs = oflows.expand(sc)
    r = osim.run_flowset(fs)
    want = 2 * (g - 1) / g * S / NV + 2 * (m - 1) / (g * m) * S / NIC
    assert math.isclose(r.makespan, want, rel_tol=1e-9)
    assert rel_err(r.finish, _longest_path(fs)) < 1e-12
    n = 2 * m * g * (g - 1) + g * 2 * (m - 1) * m
    assert fs.F == n


def test_hier_degenerates_to_ring():
    """g = 1: the inter-server ring all-reduce; m = 1: the in-server ring."""
    for m, g, bw in ((6, 1, NIC), (1, 6, NV)):
        S = 48 * MiB
        a = Scenario(_one_leaf(m, g))
        a.add(Hier(np.arange(m * g).reshape(m, g), S))
        b = Scenario(_one_leaf(m, g))
        b.add(Ring("allreduce", np.arange(m * g), S))
        fa, fb = oflows.expand(a), oflows.expand(b)
        ra, rb = osim.run_flowset(fa), osim.run_flowset(fb)
        assert math.isclose(ra.makespan, rb.makespan, rel_tol=1e-12)
        assert math.isclose(ra.makespan, 2 * (m * g - 1) / (m * g) * S / bw, rel_tol=1e-12)


# ---------------------------------------------------------------- latency
def _explicit(caps, lats):
    return Topology(kind="explicit", capacities=np.asarray(caps, np.float64),
                    latencies=np.asarray(lats, np.float64))


def test_latency_single_flow():
    sc = Scenario(_explicit([4e9, 1e9, 2e9], [1e-6, 3e-6, 0.5e-6]))
    sc.add(PathFlow([0, 1, 2], 1e6, lag=2e-3))
    r = osim.run_scenario(sc)
    assert math.isclose(r.finish[0], 2e-3 + 1e6 / 1e9 + 4.5e-6, rel_tol=1e-14)


def test_latency_frees_the_link_at_the_last_byte():
    """A (1 MB, latency 1 ms) and B (2 MB, no latency) share a 1 GB/s link:
    both run at 0.5 GB/s until A's last byte leaves at 2 ms; A arrives at
    3 ms; B then runs alone and ends at 3 ms."""
    sc = Scenario(_explicit([1e9, 1e12, 1e12], [0.0, 1e-3, 0.0]))
    sc.add(PathFlow([0, 1], 1e6))
    sc.add(PathFlow([0, 2], 2e6))
    r = osim.run_scenario(sc)
    assert math.isclose(r.finish[0], 3e-3, rel_tol=1e-12)
    # freeing the link only on arrival would leave B at 0.5 GB/s until 3 ms: 3.5 ms
    assert math.isclose(r.finish[1], 3e-3, rel_tol=1e-12)


def test_latency_release_after_the_latest_finish():
    """C waits for A (sends by 1 ms, arrives at 6 ms) and B (sends by 3 ms,
    no latency): it is released at 6 ms, although B is the last to send."""
    sc = Scenario(_explicit([1e9, 1e9, 1e9], [5e-3, 0.0, 0.0]))
    sc.add(PathFlow([0], 1e6))
    sc.add(PathFlow([1], 3e6))
    sc.add(PathFlow([2], 1e6, lag=1e-4, after=(0, 1)))
    r = osim.run_scenario(sc)
    assert math.isclose(r.finish[0], 6e-3, rel_tol=1e-12)
    assert math.isclose(r.finish[1], 3e-3, rel_tol=1e-12)
    assert math.isclose(r.finish[2], 6e-3 + 1e-4 + 1e-3, rel_tol=1e-12)


@pytest.mark.parametrize("mode,steps_paid", [("chained", 14), ("flat", 1), ("aggregated", 1)])
def test_latency_ring_steps(mode, steps_paid):
    """Eight ranks of one server, NVLink latency lam: a chained ring pays it
    once per step, flat and aggregated rings once."""
    lam = 2e-6
    S = 64 * MiB
    sc = Scenario(_server(8, nvlink_latency_s=lam))
    sc.add(Ring("allreduce", np.arange(8), S, mode=mode))
    r = osim.run_scenario(sc)
    want = 14 * (S / 8) / NV + steps_paid * lam
    assert math.isclose(r.makespan, want, rel_tol=1e-9)


def test_latency_tree_and_hier():
    lam, mu = 1e-6, 4e-6
    S = 64 * MiB
    sc = Scenario(_server(8, nvlink_latency_s=lam))
    sc.add(Tree(np.arange(8), S))
    fs = oflows.expand(sc)
    r = osim.run_flowset(fs)
    assert math.isclose(r.makespan, 3 * S / NV + 6 * lam, rel_tol=1e-9)
    assert rel_err(r.finish, _longest_path(fs)) < 1e-12
    m, g = 3, 4
    sc = Scenario(_one_leaf(m, g, nvlink_latency_s=lam, fabric_latency_s=mu))
    sc.add(Hier(np.arange(m * g).reshape(m, g), S))
    fs = oflows.expand(sc)
    r = osim.run_flowset(fs)
    # NIC up + NIC down per inter-server step
    want = (2 * (g - 1) * ((S / g) / NV + lam) + 2 * (m - 1) * ((S / (g * m)) / NIC + 2 * mu))
    assert math.isclose(r.makespan, want, rel_tol=1e-9)
    assert rel_err(r.finish, _longest_path(fs)) < 1e-12


def test_latency_sum_in_path_order():
    topo = _one_leaf(2, 2, fabric_latency_s=3e-7, nvlink_latency_s=1e-7)
    sc = Scenario(topo)
    sc.add(Send(0, 3, MiB))
    sc.add(Send(0, 1, MiB))
    fs = oflows.expand(sc)
    assert fs.lat[0] == (0.0 + 3e-7) + 3e-7 and fs.lat[1] == 1e-7


def test_latency_exact_twin_random():
    """fp64 oracle against exact rational arithmetic, random explicit cases
    with latencies, dependencies and shared links."""
    rng = np.random.default_rng(11)
    for case in range(25):
        L = int(rng.integers(2, 6))
        caps = rng.choice([1e9, 2e9, 5e8, 4e9], size=L)
        lats = rng.choice([0.0, 1e-4, 2.5e-4, 5e-4], size=L)
        sc = Scenario(_explicit(caps, lats))
        for k in range(int(rng.integers(2, 9))):
            path = sorted(rng.choice(L, size=int(rng.integers(1, L + 1)), replace=False).tolist())
            after = tuple(int(a) for a in rng.choice(k, size=min(k, int(rng.integers(0, 3))),
                                                     replace=False)) if k else ()
            sc.add(PathFlow(path, float(rng.choice([1e5, 3e5, 1e6])),
                            lag=float(rng.choice([0.0, 1e-4])), after=after))
        fs = oflows.expand(sc)
        r = osim.run_flowset(fs)
        ex, *_ = plain.simulate(fs, exact=True)
        assert rel_err(r.finish, [float(x) for x in ex]) < 1e-12, case
