"""GPU tests of the cluster layout (NETSIM_EXEC_CLUSTER): one leader
workgroup per XCD runs the parts' event loops as the block layout does and
hands re-solves of at least assist_min_flows flows to the other workgroups of
its XCD, which run the multi-workgroup solve over link state in global memory.

The re-solve is the same computation on the same integer link state, so the
finish times and the solve statistics must equal the block layout's bit for
bit (the block layout is held to the oracle in test_gpu_parity); with
assist_min_flows = 1 every re-solve goes to the helpers, which exercises the
hand-over on every event.  One case also goes straight to the oracle."""

import sys

import numpy as np
import pytest

from oracle import sim as osim
from workloads import configs, micro
from workloads.program import Program

pytestmark = pytest.mark.gpu

TOL = 1e-6
# statistics that do not depend on where a solve ran (a re-solve of more than
# 64 x 1024 flows is "wide" in the block layout only)
SAME = ("events", "solves", "rounds", "flows_swept", "incidences_swept", "active_swept",
        "pending_swept", "reselected", "completed_flows")


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
    fa, fb = np.isfinite(a), np.isfinite(b)
    assert np.array_equal(fa, fb), "different sets of finished flows"
    return float(np.max(np.abs(a[fa] - b[fa]) / np.maximum(np.abs(b[fa]), 1e-300))) if fa.any() else 0.0


def _both(program, assist_min, helpers=0, **opt):
    ns, pr = _gpu()
    a, sa = pr.run_program(program, ns.make_options(exec=ns.EXEC_BLOCK, **opt))
    b, sb = pr.run_program(program, ns.make_options(exec=ns.EXEC_CLUSTER, assist_min_flows=assist_min,
                                                    assist_helpers=helpers, **opt))
    for x, y in zip(a, b):
        assert np.array_equal(x, y, equal_nan=True)
    for k in SAME:
        assert sa[k] == sb[k], (k, sa[k], sb[k])
    assert sa["assisted_solves"] == 0
    assert sb["complete"] == 1
    return sa, sb


@pytest.mark.parametrize("single_clock", [0, 1])
@pytest.mark.parametrize("assist_min", [1, 256])
@pytest.mark.parametrize("helpers", [0, 1, 31])
def test_cluster_equals_block(single_clock, assist_min, helpers):
    """Tensor-parallel rings and pipeline sends (several parts, or one):
    every re-solve (assist_min = 1) or the larger ones handed to the
    default number of helpers, to one, or to every other workgroup of the
    XCD."""
    _say(f"test_cluster_equals_block single_clock={single_clock} assist_min={assist_min} "
         f"helpers={helpers}")
    sa, sb = _both(configs.c2(2, tp_reps=6), assist_min, helpers, single_clock=single_clock)
    assert 0 <= sb["assisted_solves"] <= sb["solves"]
    if assist_min == 1:
        assert sb["assisted_solves"] > 0
    _say("  solves", sb["solves"], "assisted", sb["assisted_solves"], "parts", sb["parts"])


def test_cluster_against_oracle():
    """One clock per scenario: finish times within 1e-6 of the oracle's and
    the oracle's event and solve counts, every re-solve run by the helpers."""
    ns, pr = _gpu()
    _say("test_cluster_against_oracle")
    program = configs.c2(2, tp_reps=6)
    ref = osim.run_scenario(program.scenarios[0])
    fins, st = pr.run_program(program, ns.make_options(exec=ns.EXEC_CLUSTER, assist_min_flows=1,
                                                       single_clock=1))
    assert _rel(fins[0], ref.finish) < TOL
    assert st["events"] == ref.events and st["solves"] == ref.solves
    assert st["assisted_solves"] > 0


def test_cluster_expert_parallel_alltoall():
    """The expert-parallel all-to-all (fat tree, Zipf dispatch) reduced to two
    server blocks of four groups: re-solves of ~16k flows at every phase
    start, with the default threshold."""
    _say("test_cluster_expert_parallel_alltoall")
    sa, sb = _both(configs.c4(4, blocks=2, locals_=4, phases=2), 0)
    assert sb["assisted_solves"] > 0
    _say("  block s", sa["device_seconds"], "cluster s", sb["device_seconds"],
         "assisted", sb["assisted_solves"], "of", sb["solves"])


def test_cluster_link_state_in_global_memory():
    """One clock over the whole 4096-GPU fat tree: the part has ~20k links,
    more than shared memory holds, so the leader's link state and stamps
    are in global memory and shared with the helpers."""
    _say("test_cluster_link_state_in_global_memory")
    sa, sb = _both(configs.c4(4, blocks=2, locals_=2, phases=2), 1024, single_clock=1)
    assert sa["parts"] == 1 and sb["assisted_solves"] > 0


def test_cluster_many_parts_few_leaders():
    """200 random dynamic cases as 200 scenarios, far more parts than XCDs:
    leaders claim parts one after another; each scenario against the oracle."""
    _say("test_cluster_many_parts_few_leaders")
    scs = []
    for seed in range(200):
        scs += micro.random_dynamic(seed, integer_caps=(seed % 2 == 0)).scenarios
    sa, sb = _both(Program("micro-batch", scs), 1, single_clock=1)
    assert sb["parts"] == len(scs) and sb["assisted_solves"] > 0
    ns, pr = _gpu()
    fins, _ = pr.run_program(Program("micro-batch", scs),
                             ns.make_options(exec=ns.EXEC_CLUSTER, assist_min_flows=1, single_clock=1))
    for s, sc in enumerate(scs):
        assert _rel(fins[s], osim.run_scenario(sc).finish) < TOL, s


def test_cluster_advance_in_pieces():
    """Runs continued over several launches keep the helpers' counters and
    stamps consistent: pieces equal one run and the block layout's run."""
    ns, pr = _gpu()
    _say("test_cluster_advance_in_pieces")
    program = configs.c2(2, tp_reps=6)
    ref, _ = pr.run_program(program, ns.make_options(exec=ns.EXEC_BLOCK))
    ref = np.concatenate(ref)
    T = float(np.nanmax(ref))
    ld = pr.load_program(program, ns.make_options(exec=ns.EXEC_CLUSTER, assist_min_flows=1))
    try:
        h = ld.handle
        for frac in (0.25, 0.5, 0.75):
            ns.netsim_advance(h, until=frac * T)
            got = ns.netsim_get_finish(h)
            assert np.array_equal(np.isfinite(got), ref <= frac * T)
            assert np.array_equal(got[np.isfinite(got)], ref[np.isfinite(got)])
        ns.netsim_advance(h)
        assert np.array_equal(ns.netsim_get_finish(h), ref)
        assert ns.netsim_get_stats(h)["assisted_solves"] > 0
    finally:
        ld.close()


def test_auto_picks_the_layout():
    """AUTO: the cluster layout for the 4096-GPU all-to-all (8 parts, each
    starting with 32k flows), one workgroup per part for many small parts,
    the whole grid for one very wide part; solve-only runs never use the
    cluster layout."""
    ns, pr = _gpu()
    _say("test_auto_picks_the_layout")
    _, st = pr.run_program(configs.c4(4), ns.make_options(until=1e-4))
    assert st["layout"] == ns.EXEC_CLUSTER and st["parts"] == 8
    _, st = pr.run_program(configs.c2(2, tp_reps=6), ns.make_options())
    assert st["layout"] == ns.EXEC_BLOCK
    _, st = pr.run_program(configs.c4(4), ns.make_options(until=1e-4, single_clock=1))
    assert st["layout"] == ns.EXEC_GRID and st["parts"] == 1
    _, st = pr.run_program(configs.c4(4), ns.make_options(exec=ns.EXEC_CLUSTER, until=1e-4))
    assert st["layout"] == ns.EXEC_CLUSTER
    # the cluster kernel keeps no rollback history: with one, AUTO runs C4
    # one workgroup per part
    _, st = pr.run_program(configs.c4(4), ns.make_options(until=1e-4, history_mb=64))
    assert st["layout"] == ns.EXEC_BLOCK and st["parts"] == 8


def test_cluster_leader_solves_alone_when_helpers_leave():
    """Test hook (debug bit 2): helpers leave as soon as they have no job, so
    a leader's posts find the mailbox closed and it solves its re-solves
    itself; the result is still the block layout's, bit for bit."""
    ns, pr = _gpu()
    _say("test_cluster_leader_solves_alone_when_helpers_leave")
    program = configs.c2(2, tp_reps=6)
    a, sa = pr.run_program(program, ns.make_options(exec=ns.EXEC_BLOCK, single_clock=1))
    b, sb = pr.run_program(program, ns.make_options(exec=ns.EXEC_CLUSTER, assist_min_flows=1,
                                                    single_clock=1, debug=4))
    assert np.array_equal(a[0], b[0]) and sb["complete"] == 1
    for k in SAME:
        assert sa[k] == sb[k], k
    assert sb["assisted_solves"] < sb["solves"] // 2
    _say("  assisted", sb["assisted_solves"], "of", sb["solves"])


def test_cluster_helper_barrier_timeout_is_an_error():
    """Test hook (debug bit 3): the helpers' barrier gives up at once, which
    aborts the launch; every wait of the kernel ends, the run reports the
    time-out as an error, and a later run is whole again."""
    ns, pr = _gpu()
    _say("test_cluster_helper_barrier_timeout_is_an_error")
    program = configs.c2(2, tp_reps=6)
    ref, _ = pr.run_program(program, ns.make_options(exec=ns.EXEC_BLOCK, single_clock=1))
    ld = pr.load_program(program, ns.make_options(exec=ns.EXEC_CLUSTER, assist_min_flows=1,
                                                  single_clock=1, debug=8))
    try:
        with pytest.raises(ns.NetsimError, match="barrier timed out"):
            ns.netsim_run(ld.handle)
    finally:
        ld.close()
    fins, st = pr.run_program(program, ns.make_options(exec=ns.EXEC_CLUSTER, assist_min_flows=1,
                                                       single_clock=1))
    assert np.array_equal(fins[0], ref[0]) and st["complete"] == 1 and st["assisted_solves"] > 0


def test_cluster_phase_times_count_the_helpers():
    """Phase timers (debug bit 1): a re-solve run by the helpers counts with
    the first helper's phase times, so the solve phases are not empty and the
    phases add up to no more than the device time of every part."""
    ns, pr = _gpu()
    _say("test_cluster_phase_times_count_the_helpers")
    program = configs.c2(2, tp_reps=6)
    _, st = pr.run_program(program, ns.make_options(exec=ns.EXEC_CLUSTER, assist_min_flows=1,
                                                    single_clock=1, debug=2))
    ph = st["phase_seconds"]
    assert st["assisted_solves"] > 0
    assert ph[3] > 0 and ph[5] > 0 and ph[0] > 0
    assert sum(ph) <= st["device_seconds"] * st["parts"] * 1.01
    _say("  phases", [round(x, 5) for x in ph], "device", st["device_seconds"])


def _c4_batch(n, blocks=2, locals_=4, phases=2):
    """n expert-parallel all-to-all what-if scenarios (different seeds), each
    split into `blocks` parts."""
    return Program("c4-batch", [configs.c4(4 + k, blocks=blocks, locals_=locals_,
                                           phases=phases).scenarios[0] for k in range(n)])


@pytest.mark.parametrize("n", [5, 12])
def test_cluster_several_leaders_per_xcd(n):
    """More wide parts than XCDs (10 and 24 parts): two and three leaders per
    XCD, each with its own helpers; bit-identical to the block layout."""
    _say(f"test_cluster_several_leaders_per_xcd n={n}")
    sa, sb = _both(_c4_batch(n), 0)
    assert sb["parts"] == 2 * n and sb["assisted_solves"] > 0
    _say("  block s", sa["device_seconds"], "cluster s", sb["device_seconds"])


def test_auto_picks_the_cluster_layout_for_a_batch():
    """AUTO: 16 parts starting with 32k flows each (two full-size all-to-all
    scenarios) take the cluster layout with two leaders per XCD."""
    ns, pr = _gpu()
    _say("test_auto_picks_the_cluster_layout_for_a_batch")
    program = Program("c4x2", [configs.c4(4).scenarios[0], configs.c4(5).scenarios[0]])
    _, st = pr.run_program(program, ns.make_options(until=1e-4))
    assert st["layout"] == ns.EXEC_CLUSTER and st["parts"] == 16


def test_complete_alltoall_cluster_equals_block_and_is_causal():
    """The bench's workload, complete (4096 GPUs, 8 parts, every flow of the
    four phases): the cluster layout (AUTO's choice) equals the block layout
    bit for bit, every flow finishes, and no flow finishes before its release
    (its last predecessor's finish plus its lag) plus its bytes over the
    narrowest link of its path -- a bound that holds at any size."""
    from oracle import flows as oflows
    ns, pr = _gpu()
    _say("test_complete_alltoall_cluster_equals_block_and_is_causal")
    program = configs.c4(4)
    a, sa = pr.run_program(program, ns.make_options(exec=ns.EXEC_BLOCK))
    b, sb = pr.run_program(program, ns.make_options())
    assert sb["layout"] == ns.EXEC_CLUSTER and sb["complete"] == 1
    assert np.array_equal(a[0], b[0])
    for k in SAME:
        assert sa[k] == sb[k], k
    fin = b[0]
    assert np.all(np.isfinite(fin))
    fs = oflows.expand(program.scenarios[0])
    deg = np.diff(fs.dep_off)
    base = np.zeros(fs.F)
    has = deg > 0
    if has.any():
        seg = np.maximum.reduceat(fin[fs.dep_ids], fs.dep_off[:-1][has])
        base[has] = seg
    mincap = np.full(fs.F, np.inf)
    plen = np.diff(fs.path_off)
    wp = plen > 0
    mincap[wp] = np.minimum.reduceat(fs.cap[fs.path_link], fs.path_off[:-1][wp])
    lower = base + fs.start + np.where(wp, fs.nbytes / mincap, 0.0)
    assert np.all(fin >= lower * (1 - 1e-12))
    _say("  block s", sa["device_seconds"], "cluster s", sb["device_seconds"])


@pytest.mark.parametrize("case", ["c2-every-resolve", "global-link-state", "c4-complete"])
def test_formal_release_is_bit_identical(case):
    """Debug bit 6 makes every release of the cluster layout (the helpers'
    barrier, the leader's hand-over, a helper's end of job) an agent-scope
    release fence, the memory model's own form, instead of a drain of the
    wave's memory operations: the results and statistics are the same bit
    for bit."""
    ns, pr = _gpu()
    _say(f"test_formal_release_is_bit_identical {case}")
    if case == "c2-every-resolve":
        program, kw = configs.c2(2, tp_reps=6), dict(assist_min_flows=1)
    elif case == "global-link-state":
        program, kw = configs.c4(4, blocks=2, locals_=2, phases=2), dict(assist_min_flows=1024,
                                                                          single_clock=1)
    else:
        program, kw = configs.c4(4), {}
    a, sa = pr.run_program(program, ns.make_options(exec=ns.EXEC_CLUSTER, **kw))
    b, sb = pr.run_program(program, ns.make_options(exec=ns.EXEC_CLUSTER, debug=64, **kw))
    for x, y in zip(a, b):
        assert np.array_equal(x, y, equal_nan=True)
    for k in SAME + ("assisted_solves",):
        assert sa[k] == sb[k], k
    assert sb["assisted_solves"] > 0
    _say("  drain s", sa["device_seconds"], "formal release s", sb["device_seconds"])


@pytest.mark.parametrize("assist_min", [1, 256])
@pytest.mark.parametrize("single_clock", [0, 1])
def test_cluster_random_micro_batch(assist_min, single_clock):
    """100 random dynamic micro cases (random fabrics, releases,
    dependencies, zero-byte flows) in one batched handle: the cluster layout,
    with every re-solve handed to the helpers or with the leaders solving
    what is smaller than 256 flows, gives the block layout's bits."""
    ns, pr = _gpu()
    _say(f"test_cluster_random_micro_batch assist_min={assist_min} single_clock={single_clock}")
    scs = []
    for seed in range(100):
        scs += micro.random_dynamic(900 + seed, integer_caps=(seed % 3 == 0)).scenarios
    program = Program("micro-cluster", scs)
    a, sa = pr.run_program(program, ns.make_options(exec=ns.EXEC_BLOCK, single_clock=single_clock))
    b, sb = pr.run_program(program, ns.make_options(exec=ns.EXEC_CLUSTER, assist_min_flows=assist_min,
                                                    single_clock=single_clock))
    assert sb["layout"] == ns.EXEC_CLUSTER
    assert all(np.array_equal(x, y) for x, y in zip(a, b))
    assert sa["events"] == sb["events"] and sa["solves"] == sb["solves"]
    if assist_min == 1:
        assert sb["assisted_solves"] > 0
