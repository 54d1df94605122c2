"""GPU parity of exact mode (``netsim_options.exact = 1``) against the fp64
oracle, through the C ABI.

Exact mode carries out the oracle's own arithmetic (one clock per scenario,
one bottleneck level per progressive-filling iteration with the 1e-12 tie
band on the minimum share, remaining bytes updated at every event), so the
bar is the method's 1e-6 relative per flow and the target is bit-identity:
every test asserts both, and the event, solve, iteration and swept-work
counts equal the oracle's.  C3 is compared flow by flow over its whole
horizon against the stored complete oracle run (tests/golden/c3_finish.npz).
"""

import json
import math
import os
import sys

import numpy as np
import pytest

from oracle import flows as oflows
from oracle import sim as osim
from workloads import configs, micro
from workloads.program import Program

sys.path.insert(0, os.path.join(os.path.dirname(__file__), "golden"))
import f64store  # noqa: E402

pytestmark = pytest.mark.gpu

TOL = 1e-6
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2505_01616_amd import netsim as ns
    from paper_2505_01616_amd import program as prog
    return ns, prog


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


def _rel(a, b):
    a, b = np.asarray(a), np.asarray(b)
    assert a.shape == b.shape
    fa, fb = np.isfinite(a), np.isfinite(b)
    assert np.array_equal(fa, fb), "different sets of finished flows"
    if not fa.any():
        return 0.0
    return float(np.max(np.abs(a[fa] - b[fa]) / np.maximum(np.abs(b[fa]), 1e-300)))


def _same(gpu, ref):
    """1e-6 per flow (the bar), then bit for bit (the target)."""
    assert _rel(gpu, ref) < TOL
    assert np.array_equal(np.asarray(gpu), np.asarray(ref), equal_nan=True)


def _counts(stats, ref):
    assert stats["events"] == ref.events
    assert stats["solves"] == ref.solves
    assert stats["rounds"] == ref.iterations
    assert stats["flows_swept"] == ref.flows_swept
    assert stats["incidences_swept"] == ref.incidences_swept


@pytest.mark.parametrize("mode", ["chained", "flat", "aggregated"])
@pytest.mark.parametrize("links", ["shared", "global"])
def test_c1_exact(mode, links):
    ns, pr = _gpu()
    _say(f"test_c1_exact mode={mode} links={links}")
    program = configs.c1(1, mode=mode)
    ref = osim.run_scenario(program.scenarios[0])
    fins, stats = pr.run_program(program, ns.make_options(exact=1, debug=16 if links == "global" else 0))
    _same(fins[0], ref.finish)
    _counts(stats, ref)
    assert stats["layout"] == ns.EXEC_EXACT and stats["parts"] == 1 and stats["complete"] == 1


@pytest.mark.parametrize("threads", [64, 256, 1024])
def test_exact_independent_of_workgroup_size(threads):
    ns, pr = _gpu()
    _say(f"test_exact_independent_of_workgroup_size threads={threads}")
    program = configs.c2(2, tp_reps=6)
    ref = osim.run_scenario(program.scenarios[0])
    fins, stats = pr.run_program(program, ns.make_options(exact=1, block_threads=threads))
    _same(fins[0], ref.finish)
    _counts(stats, ref)


@pytest.mark.parametrize("links", ["shared", "global"])
def test_micro_batched_exact(links):
    """200 random dynamic cases (releases, dependencies, zero-byte flows,
    integer and random capacities) as 200 scenarios of one batched run."""
    ns, pr = _gpu()
    _say(f"test_micro_batched_exact links={links}")
    scs = []
    for seed in range(200):
        scs += micro.random_dynamic(seed, integer_caps=(seed % 2 == 0)).scenarios
    program = Program("micro-batch", scs)
    fins, stats = pr.run_program(program, ns.make_options(exact=1, debug=16 if links == "global" else 0))
    tot = dict(events=0, solves=0, iterations=0, flows_swept=0, incidences_swept=0)
    for s, sc in enumerate(scs):
        ref = osim.run_scenario(sc)
        _same(fins[s], ref.finish)
        for k in tot:
            tot[k] += getattr(ref, k)
    assert stats["events"] == tot["events"] and stats["solves"] == tot["solves"]
    assert stats["rounds"] == tot["iterations"]
    assert stats["flows_swept"] == tot["flows_swept"]
    assert stats["incidences_swept"] == tot["incidences_swept"]
    assert stats["parts"] == len(scs)


def test_c2_exact():
    ns, pr = _gpu()
    _say("test_c2_exact")
    program = configs.c2(2)
    ref = osim.run_scenario(program.scenarios[0])
    fins, stats = pr.run_program(program, ns.make_options(exact=1))
    _same(fins[0], ref.finish)
    _counts(stats, ref)
    _say("c2 exact: device s", stats["device_seconds"])


def test_c3_exact_every_flow():
    """C3 at full size, all 262,096 flows over the whole horizon, against the
    stored complete oracle run (the C3 trajectory is ill-conditioned in fp64:
    only the oracle's own arithmetic reproduces it to 1e-6)."""
    ns, pr = _gpu()
    _say("test_c3_exact_every_flow")
    ref = f64store.load(os.path.join(GOLDEN, "c3_finish.npz"))["finish"]
    with open(os.path.join(GOLDEN, "c3_full.json")) as fh:
        meta = json.load(fh)
    program = configs.c3(3)
    fins, stats = pr.run_program(program, ns.make_options(exact=1))
    assert len(fins[0]) == meta["flows"] == len(ref)
    _say("c3 exact: device s", stats["device_seconds"], "events", stats["events"],
         "max rel", _rel(fins[0], ref))
    _same(fins[0], ref)
    assert stats["events"] == meta["events"] and stats["solves"] == meta["solves"]
    assert stats["rounds"] == meta["iterations"]
    assert stats["flows_swept"] == meta["flows_swept"]
    assert stats["incidences_swept"] == meta["incidences_swept"]


def test_c5_exact_makespans():
    """All 256 what-if scenarios of C5 as one batched run: every scenario's
    makespan, event and solve count equal the stored oracle values."""
    ns, pr = _gpu()
    _say("test_c5_exact_makespans")
    with open(os.path.join(GOLDEN, "c5_makespans.json")) as fh:
        stored = json.load(fh)["scenarios"]
    program = configs.c5(5)
    ld = pr.load_program(program, ns.make_options(exact=1))
    try:
        ns.netsim_run(ld.handle)
        ms = ns.netsim_get_makespan(ld.handle, ld.num_scenarios)
        stats = ns.netsim_get_stats(ld.handle)
    finally:
        ld.close()
    ref = np.array([s["makespan"] for s in stored])
    _say("c5 exact: device s", stats["device_seconds"], "max rel", _rel(ms, ref))
    _same(ms, ref)
    assert stats["events"] == sum(s["events"] for s in stored)
    assert stats["solves"] == sum(s["solves"] for s in stored)


def test_c5_exact_sampled_scenarios_every_flow():
    """Eight C5 scenarios run through the oracle here, flow by flow."""
    ns, pr = _gpu()
    _say("test_c5_exact_sampled_scenarios_every_flow")
    program = configs.c5(5, scenarios=8, first=100)
    fins, stats = pr.run_program(program, ns.make_options(exact=1))
    for s, sc in enumerate(program.scenarios):
        ref = osim.run_scenario(sc)
        _same(fins[s], ref.finish)


@pytest.mark.parametrize("mode", ["chained", "flat"])
def test_exact_with_latency(mode):
    """Per-link latencies (a dependant waits for the latest arrival)."""
    ns, pr = _gpu()
    _say(f"test_exact_with_latency mode={mode}")
    program = configs.c1(1, mode=mode)
    program.scenarios[0].topo.fabric_latency_s = 2e-6
    program.scenarios[0].topo.nvlink_latency_s = 5e-7
    ref = osim.run_scenario(program.scenarios[0])
    fins, stats = pr.run_program(program, ns.make_options(exact=1))
    _same(fins[0], ref.finish)
    _counts(stats, ref)


def test_exact_advance_in_pieces_and_until():
    """Advancing in time pieces gives the one-run result bit for bit; a run
    stopped at a time equals the oracle stopped there."""
    ns, pr = _gpu()
    _say("test_exact_advance_in_pieces_and_until")
    program = configs.c2(2, tp_reps=6)
    one, _ = pr.run_program(program, ns.make_options(exact=1))
    ld = pr.load_program(program, ns.make_options(exact=1))
    try:
        for u in (1e-3, 4e-3, 9e-3, math.inf):
            ns.netsim_advance(ld.handle, until=u)
            if u == 4e-3:
                part = ns.netsim_get_finish(ld.handle)
                refp = osim.run_scenario(program.scenarios[0], until=u)
                _same(part, refp.finish)
        fin = ns.netsim_get_finish(ld.handle)
    finally:
        ld.close()
    assert np.array_equal(fin, one[0])


def test_exact_rollback_equals_fresh_run():
    """Moving a finished flow's start after the simulation passed it, then
    advancing to the end, equals a fresh run with that start, bit for bit,
    and the oracle's run of the modified flows."""
    ns, pr = _gpu()
    _say("test_exact_rollback_equals_fresh_run")
    program = configs.c2(2, tp_reps=6)
    fs = oflows.expand(program.scenarios[0])
    ld = pr.load_program(program, ns.make_options(exact=1))
    try:
        ns.netsim_advance(ld.handle, until=2e-3)
        ns.netsim_advance(ld.handle, until=5e-3)
        ns.netsim_advance(ld.handle)
        fin0 = ns.netsim_get_finish(ld.handle)
        roots = np.nonzero((np.diff(fs.dep_off) == 0) & (fs.nbytes > 0))[0]
        fid = int(roots[len(roots) // 2])
        new_start = float(fs.start[fid]) + 3e-3
        ns.netsim_update_start(ld.handle, fid, new_start)
        ns.netsim_advance(ld.handle)
        fin = ns.netsim_get_finish(ld.handle)
    finally:
        ld.close()
    st = fs.start.copy()
    st[fid] = new_start
    mod = oflows.FlowSet(fs.cap, fs.src, fs.dst, fs.nbytes, st, fs.path_off, fs.path_link,
                         fs.dep_off, fs.dep_ids)
    ref = osim.run_flowset(mod)
    _same(fin, ref.finish)
    assert not np.array_equal(fin, fin0)


def test_exact_solve_once_full_width():
    """One solve of every flow of one all-to-all phase of the 4096-GPU
    workload (258,048 flows; link state in global memory) against the
    oracle's solve of the same set."""
    ns, pr = _gpu()
    _say("test_exact_solve_once_full_width")
    program = configs.c4(4, phases=1)
    fs = oflows.expand(program.scenarios[0])
    act = np.nonzero(fs.nbytes > 0)[0]
    ref = osim.solve_rates(fs.cap, fs.path_off, fs.path_link, act)
    ld = pr.load_program(program, ns.make_options(exact=1))
    try:
        rates = ns.netsim_solve_once(ld.handle, 0, act)
        stats = ns.netsim_get_stats(ld.handle)
    finally:
        ld.close()
    _say("full-width exact solve (whole GPU): device s", stats["device_seconds"], "levels",
         stats["rounds"], "links swept", stats["links_swept"])
    _same(rates, ref)
    assert stats["layout"] == ns.EXEC_EXACT


def test_exact_watchdog_and_empty():
    ns, pr = _gpu()
    _say("test_exact_watchdog_and_empty")
    program = configs.c1(1, mode="flat")
    with pytest.raises(ns.NetsimError) as ei:
        pr.run_program(program, ns.make_options(exact=1, max_rounds=1))
    assert ei.value.status == ns.E_LIMIT
    # a scenario without flows next to one with flows
    from helpers import explicit
    empty = explicit([1.0, 2.0], [])
    one = explicit([1.0, 2.0], [{"path": [0, 1], "nbytes": 3.0}, {"barrier": True, "after": (0,)}])
    fins, stats = pr.run_program(Program("e", [empty, one]), ns.make_options(exact=1))
    assert len(fins[0]) == 0
    assert np.array_equal(fins[1], np.array([3.0, 3.0]))


@pytest.mark.parametrize("mode", ["flat", "chained"])
def test_wide_solve_on_the_whole_gpu_equals_one_workgroup(mode):
    """The whole-GPU exact solve (count, links and freezing kernels) forced on
    C1's first solve gives the one-workgroup exact solve's rates bit for bit,
    with the same iteration, flow, incidence and link counts, and the
    oracle's rates."""
    ns, pr = _gpu()
    _say(f"test_wide_solve_on_the_whole_gpu_equals_one_workgroup mode={mode}")
    program = configs.c1(1, mode=mode)
    fs = oflows.expand(program.scenarios[0])
    act = np.nonzero((fs.nbytes > 0) & (np.diff(fs.dep_off) == 0))[0]
    ref = osim.solve_rates(fs.cap, fs.path_off, fs.path_link, act)
    out = {}
    for name, dbg in (("block", 0), ("grid", 32)):
        ld = pr.load_program(program, ns.make_options(exact=1, debug=dbg))
        try:
            out[name] = (ns.netsim_solve_once(ld.handle, 0, act), ns.netsim_get_stats(ld.handle))
        finally:
            ld.close()
    (rb, sb), (rg, sg) = out["block"], out["grid"]
    _same(rg, ref)
    assert np.array_equal(rg, rb)
    for k in ("rounds", "flows_swept", "incidences_swept", "links_swept"):
        assert sg[k] == sb[k], k
    assert sg["rounds"] > 1


def test_wide_solve_long_paths():
    """Paths of up to 10 links (no 16-byte path records: the CSR form of the
    freezing sweep), random capacities, one wide solve against the oracle."""
    ns, pr = _gpu()
    _say("test_wide_solve_long_paths")
    rng = np.random.default_rng(7)
    L = 300
    caps = rng.uniform(1.0, 50.0, L)
    flows = []
    for i in range(20000):
        deg = int(rng.integers(1, 11))
        flows.append({"path": list(rng.choice(L, size=deg, replace=False)), "nbytes": 1.0})
    from helpers import explicit
    sc = explicit(caps, flows)
    fs = oflows.expand(sc)
    act = np.arange(fs.F)
    ref = osim.solve_rates(fs.cap, fs.path_off, fs.path_link, act)
    ld = pr.load_program(Program("long", [sc]), ns.make_options(exact=1))
    try:
        rates = ns.netsim_solve_once(ld.handle, 0, act)
        st = ns.netsim_get_stats(ld.handle)
    finally:
        ld.close()
    _same(rates, ref)
    assert st["rounds"] > 10


def test_bench_sweeps_runs_and_leaves_no_position():
    ns, pr = _gpu()
    _say("test_bench_sweeps_runs_and_leaves_no_position")
    program = configs.c4(4, blocks=1, locals_=8, phases=1)
    fs = oflows.expand(program.scenarios[0])
    act = np.nonzero(fs.nbytes > 0)[0]
    ld = pr.load_program(program, ns.make_options(exact=1))
    try:
        t = ns.netsim_bench_sweeps(ld.handle, 0, act, 3, 64 << 20)
        for k in ("count_ms", "freeze_ms", "count_kernel_ms", "freeze_kernel_ms"):
            assert np.all(t[k] > 0), k
        assert np.all(t["freeze_kernel_ms"] <= t["freeze_ms"] * 1.5)
        rates = ns.netsim_solve_once(ld.handle, 0, act)
    finally:
        ld.close()
    _same(rates, osim.solve_rates(fs.cap, fs.path_off, fs.path_link, act))
