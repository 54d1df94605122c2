"""Pins of the fp64 oracle against facts that do not come from the oracle:
closed forms, textbook max-min examples, an LP-free brute force, max-min
invariants, metamorphic relations and exact rational arithmetic."""

import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import flows, plain, sim
from workloads import configs, micro
from workloads.program import MiB, Program, Ring, Scenario, Topology, AllToAll

from helpers import explicit, rel_err

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def run(sc, **kw):
    return sim.run_flowset(flows.expand(sc), **kw)


# ----------------------------------------------------------- closed forms
def test_equal_flows_one_link():
    """N equal flows on one link of capacity C: rate C/N, all finish N*S/C."""
    N, S, C = 7, 3.0, 10.0
    sc = explicit([C], [dict(path=[0], nbytes=S) for _ in range(N)])
    fs = flows.expand(sc)
    rates = sim.solve_rates(fs.cap, fs.path_off, fs.path_link, np.arange(N))
    assert np.all(rates == C / N)
    r = sim.run_flowset(fs)
    assert rel_err(r.finish, np.full(N, N * S / C)) < 1e-15
    ex = plain.simulate(fs, exact=True)[0]
    assert all(x == Fraction(N) * Fraction(S) / Fraction(C) for x in ex)


def test_processor_sharing_distinct_sizes():
    """S_1 < ... < S_N on one link, all at t=0:
    t_k = t_{k-1} + (S_k - S_{k-1}) * (N - k + 1) / C."""
    sizes = [2.0, 5.0, 6.0, 11.0, 17.0, 30.0]
    C = 4.0
    sc = explicit([C], [dict(path=[0], nbytes=s) for s in sizes])
    fs = flows.expand(sc)
    N = len(sizes)
    expect, t, prev = [], Fraction(0), Fraction(0)
    for k, s in enumerate(sizes, start=1):
        t = t + (Fraction(s) - prev) * (N - k + 1) / Fraction(C)
        prev = Fraction(s)
        expect.append(t)
    ex = plain.simulate(fs, exact=True)[0]
    assert ex == expect
    r = sim.run_flowset(fs)
    assert rel_err(r.finish, [float(x) for x in expect]) < 1e-14
    assert r.events == N + 1 and r.solves == N   # one arrival event, N completions


def test_staggered_arrival():
    """a: 100 B at t=0, b: 30 B at t=4, link 10 B/s.  a alone sends 40 B by
    t=4; both then get 5 B/s, b ends at 10 with a holding 30 B; a ends at 13."""
    sc = explicit([10.0], [dict(path=[0], nbytes=100), dict(path=[0], nbytes=30, lag=4.0)])
    r = run(sc)
    assert list(r.finish) == [13.0, 10.0]
    assert plain.simulate(flows.expand(sc), exact=True)[0] == [13, 10]


def test_textbook_examples():
    """Fixtures in tests/golden/textbook_maxmin.json (hand-derived max-min
    allocations of standard examples)."""
    with open(os.path.join(GOLDEN, "textbook_maxmin.json")) as fh:
        cases = json.load(fh)["cases"]
    assert len(cases) >= 3
    for case in cases:
        caps = case["capacities"]
        paths = case["paths"]
        sc = explicit(caps, [dict(path=p, nbytes=1.0) for p in paths])
        fs = flows.expand(sc)
        rates = sim.solve_rates(fs.cap, fs.path_off, fs.path_link, np.arange(len(paths)))
        want = [float(Fraction(x)) for x in case["rates"]]
        assert rel_err(rates, want) < 1e-15, case["name"]
        ex, _ = plain.maxmin(paths, caps, list(range(len(paths))), exact=True)
        assert [ex[f] for f in range(len(paths))] == [Fraction(x) for x in case["rates"]]


def _ring_scenario(p, S, B, mode, across_servers):
    if across_servers:
        topo = Topology(kind="leaf_spine", servers=p, gpus_per_server=1, servers_per_leaf=1,
                        spines=1, nic_Bps=B, fabric_Bps=B, ecmp_seed=7)
    else:
        topo = Topology(kind="leaf_spine", servers=1, gpus_per_server=p, servers_per_leaf=1,
                        spines=1, nvlink_Bps=B, ecmp_seed=7)
    sc = Scenario(topo)
    sc.add(Ring("allreduce", np.arange(p, dtype=np.int32), S, mode=mode))
    return sc


@pytest.mark.parametrize("mode", ["chained", "flat", "aggregated"])
@pytest.mark.parametrize("across", [False, True])
def test_ring_allreduce_homogeneous(mode, across):
    """Ring all-reduce over p ranks on a ring whose every hop is its own
    link of rate B: 2(p-1)/p * S/B in every decomposition mode; in chained
    mode step k (1-based) ends at k*S/(pB)."""
    p, S, B = 6, 96 * MiB, 50e9
    r = run(_ring_scenario(p, S, B, mode, across))
    want = 2 * (p - 1) / p * S / B
    assert abs(r.makespan - want) / want < 1e-12
    if mode == "chained":
        steps = r.finish.reshape(2 * (p - 1), p)
        for k in range(2 * (p - 1)):
            assert rel_err(steps[k], np.full(p, (k + 1) * S / (p * B))) < 1e-12


def test_c1_flat_closed_form():
    """C1 flat: each fabric hop carries 126 flows of 4 MiB over a 50e9 B/s
    NIC: 10.5696 ms; each NVLink hop 126 flows over 900e9 B/s: 0.5872 ms.
    The aggregated form gives the same makespan."""
    r = run(configs.c1(1, mode="flat").scenarios[0])
    assert abs(r.makespan - 126 * 4 * MiB / 50e9) / r.makespan < 1e-12
    assert abs(np.min(r.finish) - 126 * 4 * MiB / 900e9) / np.min(r.finish) < 1e-12
    ra = run(configs.c1(1, mode="aggregated").scenarios[0])
    assert abs(ra.makespan - r.makespan) / r.makespan < 1e-12
    rc = run(configs.c1(1, mode="chained").scenarios[0])
    assert rc.makespan >= r.makespan * (1 - 1e-12)   # link-load lower bound


def test_all_to_all_star():
    """Uniform all-to-all of S bytes per pair among n hosts on one switch:
    every NIC carries n-1 flows, all finish at (n-1)*S/C."""
    n, S, C = 9, 3 * MiB, 25e9
    topo = Topology(kind="leaf_spine", servers=n, gpus_per_server=1, servers_per_leaf=n,
                    spines=1, nic_Bps=C, fabric_Bps=C, ecmp_seed=3)
    sc = Scenario(topo)
    m = np.full((n, n), S)
    sc.add(AllToAll(np.arange(n, dtype=np.int32), m))
    r = run(sc)
    assert rel_err(r.finish, np.full(n * (n - 1), (n - 1) * S / C)) < 1e-12


def test_dependency_chain_and_barrier():
    """Chained flows on one link finish at prefix sums of S_i/C; a barrier
    after a flow finishes at (its finish + lag); a flow after the barrier
    starts lag later."""
    sizes = [10.0, 4.0, 6.0, 20.0]
    C = 2.0
    fl = [dict(path=[0], nbytes=sizes[0])]
    for i in range(1, len(sizes)):
        fl.append(dict(path=[0], nbytes=sizes[i], after=[i - 1]))
    r = run(explicit([C], fl))
    assert list(r.finish) == list(np.cumsum(sizes) / C)
    sc = explicit([10.0], [dict(path=[0], nbytes=10.0),
                           dict(barrier=True, lag=0.5, after=[0]),
                           dict(path=[0], nbytes=5.0, lag=0.25, after=[1])])
    r = run(sc)
    assert list(r.finish) == [1.0, 1.5, 2.25]


# ------------------------------------------------------------ brute force
@pytest.mark.parametrize("seed", range(24))
def test_bruteforce_maxmin(seed):
    """Random static cases (<= 7 links, <= 9 flows): exactly one candidate
    allocation is feasible with the bottleneck property; progressive
    filling in exact arithmetic equals it; the fp64 oracle is within 1e-12."""
    prog = micro.random_static(seed, max_links=7, max_flows=9)
    fs = flows.expand(prog.scenarios[0])
    paths = [list(map(int, fs.path_link[fs.path_off[f]:fs.path_off[f + 1]])) for f in range(fs.F)]
    fl, found = plain.brute_force_maxmin(paths, list(fs.cap))
    assert len(found) == 1
    ex, _ = plain.maxmin(paths, list(fs.cap), fl, exact=True)
    assert tuple(ex[f] for f in fl) == found[0]
    got = sim.solve_rates(fs.cap, fs.path_off, fs.path_link, np.array(fl))
    assert rel_err(got, [float(x) for x in found[0]]) < 1e-12


# --------------------------------------------------------- exact vs fp64
@pytest.mark.parametrize("block", range(4))
def test_exact_and_plain_vs_c_oracle(block):
    """Random dynamic cases: the C oracle equals the plain fp64 Python form
    bit for bit (finish times and event / solve / iteration counts) and the
    exact rational form within 1e-12."""
    for seed in range(block * 50, block * 50 + 50):
        for integer_caps in (True, False):
            fs = flows.expand(micro.random_dynamic(seed, integer_caps=integer_caps).scenarios[0])
            r = sim.run_flowset(fs)
            ff, ev, so, it = plain.simulate(fs, exact=False)
            assert np.array_equal(np.array(ff, float), r.finish), seed
            assert (ev, so, it) == (r.events, r.solves, r.iterations), seed
            fe = np.array([float(x) for x in plain.simulate(fs, exact=True)[0]])
            assert rel_err(r.finish, fe) < 1e-12, seed


# ------------------------------------------------------------- invariants
def check_maxmin_invariants(fs, rates, tol=1e-9):
    act = np.nonzero(rates > 0)[0]
    deg = np.diff(fs.path_off)[act]
    rows = np.repeat(act, deg)
    links = np.concatenate([fs.path_link[fs.path_off[f]:fs.path_off[f + 1]] for f in act])
    load = np.bincount(links, weights=rates[rows], minlength=fs.L)
    assert np.all(load <= fs.cap * (1 + tol))
    rmax = np.zeros(fs.L)
    np.maximum.at(rmax, links, rates[rows])
    sat = load >= fs.cap * (1 - tol)
    ok = sat[links] & (rates[rows] >= rmax[links] * (1 - tol))
    has = np.zeros(len(fs.nbytes), bool)
    np.logical_or.at(has, rows, ok)
    assert np.all(has[act])


@pytest.mark.parametrize("name,kw,snaps", [
    ("c1", dict(mode="chained"), [1, 50, 500, 900]),
    ("c1", dict(mode="flat"), [1, 2]),
    ("c2", dict(tp_reps=4), [1, 100, 1000]),
    ("c3", dict(groups=1, background=100), [1, 500, 3000]),
    ("c4", dict(blocks=1, locals_=1), [1, 2, 64, 200]),
])
def test_invariants_at_sampled_solves(name, kw, snaps):
    fs = flows.expand(configs.build(name, **kw).scenarios[0])
    for s in snaps:
        r = sim.run_flowset(fs, snap_solve=s)
        assert r.solves >= s
        check_maxmin_invariants(fs, r.snap_rates)


def test_lower_bounds_c2():
    """finish >= release + bytes / (slowest link on the path); flows with
    no dependencies are released at their start time."""
    fs = flows.expand(configs.c2(2, tp_reps=6).scenarios[0])
    r = sim.run_flowset(fs)
    assert np.all(np.isfinite(r.finish))
    for f in range(fs.F):
        deps = fs.dep_ids[fs.dep_off[f]:fs.dep_off[f + 1]]
        rel = fs.start[f] + (np.max(r.finish[deps]) if len(deps) else 0.0)
        if fs.nbytes[f] > 0:
            cmin = np.min(fs.cap[fs.path_link[fs.path_off[f]:fs.path_off[f + 1]]])
            assert r.finish[f] >= (rel + fs.nbytes[f] / cmin) * (1 - 1e-12)
        else:
            assert r.finish[f] == rel


# ------------------------------------------------------------ metamorphic
def _scaled(fs, k):
    return flows.FlowSet(fs.cap.copy(), fs.src, fs.dst, fs.nbytes * 2.0 ** k, fs.start * 2.0 ** k,
                         fs.path_off, fs.path_link, fs.dep_off, fs.dep_ids)


@pytest.mark.parametrize("seed", range(10))
def test_metamorphic_scale_by_power_of_two(seed):
    fs = flows.expand(micro.random_dynamic(seed, integer_caps=False).scenarios[0])
    base = sim.run_flowset(fs).finish
    for k in (-7, 3, 20):
        assert np.array_equal(sim.run_flowset(_scaled(fs, k)).finish, base * 2.0 ** k)


def _permute(fs, seed):
    """A random topological re-numbering of the flows."""
    rng = np.random.default_rng(seed)
    F = fs.F
    deps = [list(fs.dep_ids[fs.dep_off[f]:fs.dep_off[f + 1]]) for f in range(F)]
    indeg = [len(d) for d in deps]
    succ = [[] for _ in range(F)]
    for g in range(F):
        for d in deps[g]:
            succ[d].append(g)
    ready = [f for f in range(F) if indeg[f] == 0]
    order = []
    while ready:
        i = int(rng.integers(len(ready)))
        f = ready.pop(i)
        order.append(f)
        for g in succ[f]:
            indeg[g] -= 1
            if indeg[g] == 0:
                ready.append(g)
    new_of = np.empty(F, np.int64)
    new_of[order] = np.arange(F)
    paths = [fs.path_link[fs.path_off[f]:fs.path_off[f + 1]] for f in order]
    dl = [sorted(new_of[d] for d in deps[f]) for f in order]
    poff = np.zeros(F + 1, np.int64)
    np.cumsum([len(p) for p in paths], out=poff[1:])
    doff = np.zeros(F + 1, np.int64)
    np.cumsum([len(d) for d in dl], out=doff[1:])
    cat = lambda xs, dt: np.concatenate(xs).astype(dt) if xs and sum(map(len, xs)) else np.zeros(0, dt)
    return flows.FlowSet(fs.cap, fs.src[order], fs.dst[order], fs.nbytes[order], fs.start[order],
                         poff, cat(paths, np.int32), doff, cat(dl, np.int64)), new_of


@pytest.mark.parametrize("seed", range(10))
def test_metamorphic_flow_order_and_unused_link(seed):
    fs = flows.expand(micro.random_dynamic(seed).scenarios[0])
    base = sim.run_flowset(fs).finish
    pf, new_of = _permute(fs, seed)
    assert np.array_equal(sim.run_flowset(pf).finish[new_of], base)
    extra = flows.FlowSet(np.append(fs.cap, 123.0), fs.src, fs.dst, fs.nbytes, fs.start,
                          fs.path_off, fs.path_link, fs.dep_off, fs.dep_ids)
    assert np.array_equal(sim.run_flowset(extra).finish, base)


def test_until_horizon_is_a_prefix():
    """Stopping at a time horizon gives exactly the finish times <= horizon
    of the full run."""
    fs = flows.expand(configs.c1(1, mode="chained").scenarios[0])
    full = sim.run_flowset(fs)
    T = float(np.median(full.finish))
    part = sim.run_flowset(fs, until=T)
    assert not part.complete
    done = np.isfinite(part.finish)
    assert np.array_equal(done, full.finish <= T)
    assert np.array_equal(part.finish[done], full.finish[done])


def test_c3_is_ill_conditioned_in_fp64():
    """The chained rings of C3 over degraded links amplify rounding: one ulp
    on every capacity moves the oracle's own finish times by far more than
    1e-6, whereas C1 and C2 move by about 1e-14.  (This is why C3 parity is
    checked against the oracle's own one-ulp spread past a horizon.)"""
    def spread(fs):
        base = sim.run_flowset(fs).finish
        pert = flows.FlowSet(np.nextafter(fs.cap, np.inf), fs.src, fs.dst, fs.nbytes, fs.start,
                             fs.path_off, fs.path_link, fs.dep_off, fs.dep_ids)
        return np.max(np.abs(sim.run_flowset(pert).finish - base) / base)
    assert spread(flows.expand(configs.c3(3, groups=2, background=400).scenarios[0])) > 1e-3
    assert spread(flows.expand(configs.c1(1).scenarios[0])) < 1e-12
    assert spread(flows.expand(configs.c2(2, tp_reps=6).scenarios[0])) < 1e-12
