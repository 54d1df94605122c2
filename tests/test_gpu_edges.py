"""GPU parity on edge cases and on the solve paths the headline workloads do
not reach: empty scenarios, a single flow, chains of zero-byte flows only,
paths longer than the 6-link path record (the general solve with global
work lists), a solve of more than 64 x 1024 flows in one part (the same
general solve), a part with more links than shared memory holds (link state
in global memory), and the per-solve round watchdog forced from the host.
Finish times within 1e-6 of the oracle."""

import sys

import numpy as np
import pytest

from oracle import sim as osim
from workloads import micro
from workloads.program import Barrier, PathFlow, Program, Scenario, Topology

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

def _layout(ns, name):
    """Options of an execution layout; the cluster layout hands every
    re-solve to the helper workgroups (assist_min_flows = 1)."""
    if name == "cluster":
        return dict(exec=ns.EXEC_CLUSTER, assist_min_flows=1)
    return dict(exec={"block": ns.EXEC_BLOCK, "grid": ns.EXEC_GRID}[name])



def _rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    assert a.shape == b.shape
    fa, fb = np.isfinite(a), np.isfinite(b)
    assert np.array_equal(fa, fb), "different sets of finished flows"
    return float(np.max(np.abs(a[fa] - b[fa]) / np.maximum(np.abs(b[fa]), 1e-300))) if fa.any() else 0.0


def _explicit(caps):
    return Topology(kind="explicit", capacities=np.asarray(caps, np.float64))


def degenerate_scenarios():
    out = [Scenario(_explicit([1.0, 2.0]))]                       # no flows at all
    sc = Scenario(_explicit([3.0]))
    sc.add(PathFlow([0], 12.0, lag=1.5))                          # one flow: 1.5 + 4
    out.append(sc)
    sc = Scenario(_explicit([1.0]))                                # zero-byte flows only
    sc.add(Barrier(lag=0.25))
    sc.add(Barrier(lag=0.5, after=(0,)))
    sc.add(Barrier(lag=0.0, after=(1,)))
    sc.add(Barrier(lag=2.0))
    sc.add(Barrier(lag=0.125, after=(2, 3)))
    out.append(sc)
    sc = Scenario(_explicit([2.0, 2.0]))                           # barriers between flows
    sc.add(PathFlow([0, 1], 4.0))
    sc.add(Barrier(lag=1.0, after=(0,)))
    sc.add(PathFlow([1], 6.0, after=(1,)))
    sc.add(Barrier(after=(2, 0)))
    out.append(sc)
    return out


def wide_scenario(n=70000, links=100, seed=1):
    """n flows over link 0 (the narrowest) and one other link each: all at
    the same rate, so the first solve holds every flow of the part."""
    rng = np.random.default_rng(seed)
    caps = np.full(links, 1e12)
    caps[0] = 1e9
    sc = Scenario(_explicit(caps))
    other = rng.integers(1, links, size=n)
    size = rng.choice([1e5, 2e5], size=n)
    for k in range(n):
        sc.add(PathFlow([0, int(other[k])], float(size[k])))
    return sc


def many_links_scenario(L=6000, n=3000, seed=2):
    """One part over more links than shared memory holds: every flow crosses
    link 0 and two random others."""
    rng = np.random.default_rng(seed)
    caps = rng.choice([1e9, 2e9, 4e9], size=L)
    sc = Scenario(_explicit(caps))
    for k in range(n):
        a, b = sorted(rng.choice(np.arange(1, L), size=2, replace=False).tolist())
        sc.add(PathFlow([0, a, b], float(rng.choice([1e5, 3e5])), lag=float(rng.random() * 1e-4)))
    return sc


def test_degenerate_cases():
    ns, pr = _gpu()
    _say("test_degenerate_cases")
    scs = degenerate_scenarios()
    fins, st = pr.run_program(Program("degenerate", scs))
    assert st["complete"] == 1
    assert len(fins[0]) == 0
    assert abs(fins[1][0] - 5.5) < 1e-12
    np.testing.assert_array_equal(fins[2], [0.25, 0.75, 0.75, 2.0, 2.125])
    for s, sc in enumerate(scs):
        assert _rel(fins[s], osim.run_scenario(sc).finish) < TOL


@pytest.mark.parametrize("exec_", ["block", "grid", "cluster"])
def test_long_paths(exec_):
    """Paths of up to 14 links: beyond the 16-byte path record."""
    ns, pr = _gpu()
    _say(f"test_long_paths exec={exec_}")
    scs = [micro.random_dynamic(s, max_links=14, max_flows=16).scenarios[0] for s in range(60)]
    assert max(max(len(op.path) for op in sc.ops if hasattr(op, "path")) for sc in scs) > 6
    ex = _layout(ns, exec_)
    fins, st = pr.run_program(Program("long", scs), ns.make_options(**ex, single_clock=1))
    for s, sc in enumerate(scs):
        ref = osim.run_scenario(sc)
        assert _rel(fins[s], ref.finish) < TOL, s


def test_wide_solve():
    ns, pr = _gpu()
    _say("test_wide_solve")
    sc = wide_scenario()
    fins, st = pr.run_program(Program("wide", [sc]), ns.make_options(exec=ns.EXEC_BLOCK))
    assert st["wide_solves"] >= 1
    assert _rel(fins[0], osim.run_scenario(sc).finish) < TOL


def test_links_beyond_shared_memory():
    ns, pr = _gpu()
    _say("test_links_beyond_shared_memory")
    sc = many_links_scenario()
    fins, st = pr.run_program(Program("many-links", [sc]), ns.make_options(exec=ns.EXEC_BLOCK))
    assert st["parts"] == 1
    assert _rel(fins[0], osim.run_scenario(sc).finish) < TOL


def test_round_watchdog_reports_limit():
    """A solve that needs several rounds with the watchdog set to one: the
    kernel stops the part normally and the run reports NETSIM_E_LIMIT."""
    ns, pr = _gpu()
    _say("test_round_watchdog_reports_limit")
    sc = Scenario(_explicit([1.0, 2.0, 4.0]))
    sc.add(PathFlow([0], 1.0))
    sc.add(PathFlow([0, 1], 1.0))
    sc.add(PathFlow([1, 2], 1.0))
    sc.add(PathFlow([2], 1.0))
    with pytest.raises(ns.NetsimError) as e:
        pr.run_program(Program("watchdog", [sc]), ns.make_options(max_rounds=1))
    assert e.value.status == ns.E_LIMIT
    fins, st = pr.run_program(Program("watchdog", [sc]))
    assert _rel(fins[0], osim.run_scenario(sc).finish) < TOL


def test_more_groups_than_parts():
    """3,000 independent flows (each on a link of its own): more groups than
    the 1,024 parts a scenario is split into, so groups share parts; every
    flow still ends at start + bytes / capacity."""
    ns, pr = _gpu()
    _say("test_more_groups_than_parts")
    rng = np.random.default_rng(5)
    n = 3000
    caps = rng.choice([1e9, 2e9, 4e9], size=n)
    size = rng.choice([1e5, 2e5, 3e5], size=n)
    lag = rng.choice([0.0, 1e-4], size=n)
    sc = Scenario(_explicit(caps))
    for k in range(n):
        sc.add(PathFlow([k], float(size[k]), lag=float(lag[k])))
    fins, st = pr.run_program(Program("groups", [sc]))
    assert st["parts"] == 1024
    want = lag + size / caps
    assert _rel(fins[0], want) < 1e-12
    assert _rel(fins[0], osim.run_scenario(sc).finish) < TOL
