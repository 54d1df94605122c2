"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle on
identical seeded inputs.  Per-flow completion times must agree within
1e-6 relative (the bar the method's description fixes); the observed gap
is ~1e-12, the two solvers differing only in rounding (see the solver
notes in kernels.hip)."""

import math
import sys

import numpy as np
import pytest

from oracle import flows as oflows
from oracle import sim as osim
from workloads import configs, micro
from workloads.program import Program

pytestmark = pytest.mark.gpu

TOL = 1e-6


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


def _run(prog, program, **opt):
    ns, pr = _gpu()
    fins, stats = pr.run_program(program, ns.make_options(**opt))
    return fins, stats


@pytest.mark.parametrize("mode", ["chained", "flat", "aggregated"])
@pytest.mark.parametrize("exec_", ["block", "grid"])
def test_c1(mode, exec_):
    """Per-flow finish times against the oracle, split into independent parts
    and with one clock; with one clock the event and solve counts are the
    oracle's too."""
    ns, pr = _gpu()
    _say(f"test_c1 mode={mode} exec={exec_}")
    program = configs.c1(1, mode=mode)
    ex = {"block": ns.EXEC_BLOCK, "grid": ns.EXEC_GRID}[exec_]
    ref = osim.run_scenario(program.scenarios[0])
    fins, stats = pr.run_program(program, ns.make_options(exec=ex))
    assert _rel(fins[0], ref.finish) < TOL
    assert stats["complete"] == 1
    one, s1 = pr.run_program(program, ns.make_options(exec=ex, single_clock=1))
    assert _rel(one[0], ref.finish) < TOL
    assert s1["events"] == ref.events and s1["solves"] == ref.solves and s1["parts"] == 1


@pytest.mark.parametrize("single_clock", [1, 0])
def test_micro_batched_vs_oracle(single_clock):
    """200 random dynamic cases as 200 scenarios of one batched run.  With one
    clock per scenario the event count is the oracle's exactly; split into
    independent parts the finish times still agree."""
    ns, pr = _gpu()
    _say(f"test_micro_batched_vs_oracle single_clock={single_clock}")
    scs = []
    for seed in range(200):
        scs += micro.random_dynamic(seed, integer_caps=(seed % 2 == 0)).scenarios
    program = Program("micro-batch", scs)
    fins, stats = pr.run_program(program, ns.make_options(exec=ns.EXEC_BLOCK,
                                                          single_clock=single_clock))
    ev = 0
    for s, sc in enumerate(scs):
        ref = osim.run_scenario(sc)
        assert _rel(fins[s], ref.finish) < TOL, s
        ev += ref.events
    if single_clock:
        assert stats["events"] == ev and stats["parts"] == len(scs)
    else:
        assert stats["events"] >= ev and stats["parts"] >= len(scs)


@pytest.mark.parametrize("single_clock", [0, 1])
def test_block_and_grid_agree_bitwise_and_deterministic(single_clock):
    """Integer link state makes the result independent of the layout (one
    workgroup per part with link state in shared memory, or the whole grid
    with link state in global memory) and of the run."""
    ns, pr = _gpu()
    _say(f"test_block_and_grid_agree single_clock={single_clock}")
    program = configs.c2(2, tp_reps=6)
    a, sa = pr.run_program(program, ns.make_options(exec=ns.EXEC_BLOCK, single_clock=single_clock))
    b, sb = pr.run_program(program, ns.make_options(exec=ns.EXEC_GRID, single_clock=single_clock))
    c, _ = pr.run_program(program, ns.make_options(exec=ns.EXEC_BLOCK, single_clock=single_clock))
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[0], c[0])
    assert sa["events"] == sb["events"] and sa["solves"] == sb["solves"]
    assert (sa["parts"] == 1) == bool(single_clock)


def test_c2_full():
    ns, pr = _gpu()
    _say("test_c2_full")
    program = configs.c2(2)
    ref = osim.run_scenario(program.scenarios[0])
    fins, stats = pr.run_program(program, ns.make_options())
    assert _rel(fins[0], ref.finish) < TOL
    one, s1 = pr.run_program(program, ns.make_options(single_clock=1))
    assert _rel(one[0], ref.finish) < TOL
    assert s1["events"] == ref.events and s1["solves"] == ref.solves
    _say("c2 events: parts", stats["events"], "one clock", s1["events"], "oracle", ref.events,
         "parts", stats["parts"])


def _perturbed(fs, k):
    """The flow set with every capacity moved k ulps (k may be negative)."""
    cap = fs.cap.copy()
    for _ in range(abs(k)):
        cap = np.nextafter(cap, np.inf if k > 0 else 0.0)
    return oflows.FlowSet(cap, fs.src, fs.dst, fs.nbytes, fs.start, fs.path_off, fs.path_link,
                          fs.dep_off, fs.dep_ids)


def _check_ill_conditioned(fs, gpu_finish):
    """For trajectories that fp64 does not determine to 1e-6 (the oracle
    itself moves by more when the capacities change by a few ulps):
    per-flow 1e-6 up to the horizon where the perturbed oracle runs still
    agree to 1e-9, and beyond it the GPU's deviation from the oracle must
    stay within 4x the spread of the oracle's own perturbed runs."""
    ref = osim.run_flowset(fs)
    runs = [osim.run_flowset(_perturbed(fs, k)).finish for k in (-3, -2, -1, 1, 2, 3)]
    dev = np.max([np.abs(r - ref.finish) / ref.finish for r in runs], axis=0)
    order = np.argsort(ref.finish)
    bad = order[dev[order] > 1e-9]
    horizon = ref.finish[bad[0]] if len(bad) else np.inf
    early = ref.finish < horizon
    gdev = np.abs(gpu_finish - ref.finish) / ref.finish
    assert early.sum() > 0.05 * len(early)
    assert np.max(gdev[early]) < TOL
    spread_ms = max(abs(np.max(r) - ref.makespan) for r in runs) / ref.makespan
    gpu_ms = abs(np.max(gpu_finish) - ref.makespan) / ref.makespan
    assert gpu_ms <= 4 * spread_ms + 1e-12
    assert np.quantile(gdev, 0.99) <= 4 * np.quantile(dev, 0.99) + 1e-12
    _say(f"horizon {horizon:.4g}s covers {early.mean():.1%} of flows; makespan dev gpu "
         f"{gpu_ms:.2e} vs oracle ulp spread {spread_ms:.2e}")


def test_c3_reduced():
    ns, pr = _gpu()
    _say("test_c3_reduced")
    program = configs.c3(3, groups=2, background=400)
    fins, stats = pr.run_program(program, ns.make_options())
    _check_ill_conditioned(oflows.expand(program.scenarios[0]), fins[0])


def test_c4_one_group_full_run():
    ns, pr = _gpu()
    _say("test_c4_one_group")
    program = configs.c4(4, blocks=1, locals_=1)
    for ex in (ns.EXEC_BLOCK, ns.EXEC_GRID):
        fins, stats = pr.run_program(program, ns.make_options(exec=ex))
        ref = osim.run_scenario(program.scenarios[0])
        assert _rel(fins[0], ref.finish) < TOL


@pytest.mark.parametrize("exec_", ["block", "grid", "cluster"])
def test_c4_full_size_prefix(exec_):
    """Full 4096-GPU C4 (8 independent parts of 8 expert groups each),
    simulated up to the last completion among the oracle's first 150 events
    (the 64 group arrivals, then the first completions); every flow finished
    by then must agree and the sets of finished flows must be equal."""
    ns, pr = _gpu()
    _say(f"test_c4_full_size_prefix exec={exec_}")
    program = configs.c4(4)
    fs = oflows.expand(program.scenarios[0])
    probe = osim.run_flowset(fs, max_events=150)
    assert np.isfinite(probe.finish).sum() >= 50
    # the horizon sits 1e-9 relative after the last completion: far above the
    # ~1e-12 GPU/oracle gap, far below the spacing of events there
    T = float(np.nanmax(probe.finish)) * (1 + 1e-9)
    ref = osim.run_flowset(fs, until=T)
    done = ref.finish[np.isfinite(ref.finish)]
    assert len(done) >= 50 and np.all(np.abs(done - T) > 1e-10 * T)
    ex = {"block": ns.EXEC_BLOCK, "grid": ns.EXEC_GRID, "cluster": ns.EXEC_CLUSTER}[exec_]
    fins, stats = pr.run_program(program, ns.make_options(exec=ex, until=T))
    assert stats["complete"] == 0 and stats["parts"] == 8
    assert _rel(fins[0], ref.finish) < TOL
    _say("c4 prefix T", T, "flows done", int(np.isfinite(ref.finish).sum()),
         "events", stats["events"], ref.events)


def test_c4_solve_once_full_size():
    """One solve with every phase-0 flow of full C4 active: rates within 1e-9
    of the oracle, and the max-min invariants hold."""
    ns, pr = _gpu()
    _say("test_c4_solve_once")
    program = configs.c4(4)
    fs = oflows.expand(program.scenarios[0])
    act = np.nonzero((fs.nbytes > 0) & (np.diff(fs.dep_off) == 0))[0]
    ref = osim.solve_rates(fs.cap, fs.path_off, fs.path_link, act)
    ld = pr.load_program(program)
    try:
        got = ns.netsim_solve_once(ld.handle, 0, act + ld.first_flow[0])
        st = ns.netsim_get_stats(ld.handle)
    finally:
        ld.close()
    assert _rel(got, ref) < 1e-9
    _say("c4 solve rounds", st["rounds"], "device s", st["device_seconds"])


def test_c5_sample_batched():
    ns, pr = _gpu()
    _say("test_c5_sample_batched")
    program = configs.c5(5, scenarios=8)
    fins, stats = pr.run_program(program, ns.make_options())
    for s, sc in enumerate(program.scenarios):
        ref = osim.run_scenario(sc)
        assert _rel(fins[s], ref.finish) < TOL, s


def _golden(name):
    import json
    import os
    with open(os.path.join(os.path.dirname(__file__), "golden", name)) as fh:
        return json.load(fh)


def test_c5_full_batched():
    """All 256 what-if scenarios in one batched run: per-scenario makespan
    and event count against the stored oracle values."""
    ns, pr = _gpu()
    _say("test_c5_full_batched")
    gold = _golden("c5_makespans.json")["scenarios"]
    program = configs.c5(5)
    want = np.array([g["makespan"] for g in gold])
    for single_clock in (0, 1):
        ld = pr.load_program(program, ns.make_options(single_clock=single_clock))
        try:
            ns.netsim_run(ld.handle)
            ms = ns.netsim_get_makespan(ld.handle, len(program.scenarios))
            st = ns.netsim_get_stats(ld.handle)
        finally:
            ld.close()
        assert _rel(ms, want) < TOL
        if single_clock:
            assert st["events"] == sum(g["events"] for g in gold)
        _say("c5 full: single_clock", single_clock, "device s", st["device_seconds"],
             "events", st["events"], "parts", st["parts"])


def test_c4_part_complete():
    """One part of the expert-parallel all-to-all at full width (the eight
    expert groups of one 64-server block, one dispatch phase, ~32k flows) run
    to the end: ~27k events, the large re-solves handed to the helper
    workgroups (AUTO picks the cluster layout) and many slot compactions.
    The event count equals the oracle's, the makespan and a seeded 3000-flow
    sample of finish times agree with the stored complete oracle run to 1e-6,
    and the block layout gives the same bits."""
    ns, pr = _gpu()
    _say("test_c4_part_complete")
    gold = _golden("c4_part_summary.json")
    program = configs.c4(4, blocks=1, locals_=8, phases=1)
    fins, st = pr.run_program(program, ns.make_options())
    assert st["layout"] == ns.EXEC_CLUSTER and st["assisted_solves"] > 0 and st["complete"] == 1
    assert st["parts"] == 1 and st["events"] == gold["events"]  # one part: the oracle's own events
    fin = fins[0]
    assert len(fin) == gold["flows"] and int(np.isfinite(fin).sum()) == gold["finished"]
    ids = np.array(gold["sample_ids"])
    assert _rel(fin[ids], np.array(gold["sample_finish"])) < TOL
    assert abs(float(np.max(fin)) - gold["makespan"]) <= TOL * gold["makespan"]
    bfins, _ = pr.run_program(program, ns.make_options(exec=ns.EXEC_BLOCK))
    assert np.array_equal(bfins[0], fin, equal_nan=True)
    _say(f"c4 part: device s {st['device_seconds']:.3f}, events {st['events']} (oracle {gold['events']}), "
         f"assisted {st['assisted_solves']}")


def test_c4_full_size_first_part_complete():
    """The full 4096-GPU all-to-all exactly as bench.py runs it (AUTO, 8
    parts, all four phases, to the end).  Its first 129,048 flows are the
    eight expert groups of the first 64-server block: they share no link and
    no dependency with the other flows, so the oracle's complete run of that
    block alone (stored: ~111k events) is their exact reference.  The
    makespan of the block and a seeded 3000-flow sample agree to 1e-6."""
    ns, pr = _gpu()
    _say("test_c4_full_size_first_part_complete")
    gold = _golden("c4_part4_summary.json")
    program = configs.c4(4)
    fins, st = pr.run_program(program, ns.make_options())
    assert st["complete"] == 1 and st["parts"] == 8 and st["layout"] == ns.EXEC_CLUSTER
    part = fins[0][:gold["flows"]]
    assert int(np.isfinite(part).sum()) == gold["finished"]
    ids = np.array(gold["sample_ids"])
    assert _rel(part[ids], np.array(gold["sample_finish"])) < TOL
    assert abs(float(np.max(part)) - gold["makespan"]) <= TOL * gold["makespan"]
    _say(f"c4 full, first part: device s {st['device_seconds']:.2f}, oracle events of the part "
         f"{gold['events']}, GPU part events (all parts) {st['events']}")


def test_c3_full_size():
    """Full C3 (ill-conditioned in fp64): sampled flows finishing before the
    horizon of the oracle's perturbed runs agree to 1e-6; the makespan and
    the spread of a seeded 4000-flow sample stay within 4x the oracle's own
    spread over eleven runs with every capacity moved by -5..6 ulps."""
    ns, pr = _gpu()
    _say("test_c3_full_size")
    gold = _golden("c3_summary.json")
    program = configs.c3(3)
    fins, st = pr.run_program(program, ns.make_options())
    fin = fins[0]
    assert len(fin) == gold["flows"]
    early = np.array(gold["early_ids"])
    assert _rel(fin[early], np.array(gold["early_finish"])) < TOL
    gm = abs(np.max(fin) - gold["makespan"]) / gold["makespan"]
    assert gm <= 4 * gold["ulp_spread_makespan"] + 1e-12
    ids = np.array(gold["sample_ids"])
    dev = np.abs(fin[ids] - np.array(gold["sample_finish"])) / np.array(gold["sample_finish"])
    assert np.quantile(dev, 0.99) <= 4 * gold["ulp_spread_q99"] + 1e-12
    _say(f"c3 full: makespan dev {gm:.2e} (oracle ulp spread {gold['ulp_spread_makespan']:.2e}), "
         f"device s {st['device_seconds']:.2f}, events {st['events']} (oracle {gold['events']})")
