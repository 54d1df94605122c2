"""GPU tests of time rollback (the paper's Section 4.2: an API that updates
an existing flow's start time, an API that advances the simulation step by
step or up to a time, and garbage collection of history).

Advancing in pieces must give, bit for bit, the finish times of one run;
after an update of a start the simulation continued to the end must give,
bit for bit, the finish times of a fresh run whose flows had that start all
along (the rollback restores an exact earlier state and the re-simulation is
deterministic), and they must match the oracle run on the modified flows."""

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

def _layout(ns, name):
    """Options of an execution layout; the cluster layout hands every
    re-solve to the helper workgroups (assist_min_flows = 1)."""
    if name == "cluster":
        return dict(exec=ns.EXEC_CLUSTER, assist_min_flows=1)
    return dict(exec={"block": ns.EXEC_BLOCK, "grid": ns.EXEC_GRID}[name])



def _rel(a, b):
    a, b = np.asarray(a), np.asarray(b)
    fa, fb = np.isfinite(a), np.isfinite(b)
    assert np.array_equal(fa, fb), "different sets of finished flows"
    return float(np.max(np.abs(a[fa] - b[fa]) / np.maximum(np.abs(b[fa]), 1e-300))) if fa.any() else 0.0


def _fresh(program, updates, **opt):
    """Finish times of a run whose flows carry the updated starts from the beginning."""
    ns, pr = _gpu()
    ld = pr.load_program(program, ns.make_options(**opt))
    try:
        for fid, st in updates.items():
            ns.netsim_update_start(ld.handle, fid, st)
        ns.netsim_run(ld.handle)
        return ns.netsim_get_finish(ld.handle)
    finally:
        ld.close()


def _oracle(sc, updates):
    fs = oflows.expand(sc)
    for fid, st in updates.items():
        fs.start[fid] = st
    return osim.run_flowset(fs).finish


@pytest.mark.parametrize("exec_", ["block", "grid", "cluster"])
def test_advance_in_pieces_equals_one_run(exec_):
    ns, pr = _gpu()
    _say(f"test_advance_in_pieces exec={exec_}")
    program = configs.c2(2, tp_reps=6)
    ex = _layout(ns, exec_)
    ref = _fresh(program, {}, **ex)
    T = float(np.nanmax(ref))
    ld = pr.load_program(program, ns.make_options(**ex))
    try:
        h = ld.handle
        for frac in (0.2, 0.5, 0.8):
            ns.netsim_advance(h, until=frac * T)
            got = ns.netsim_get_finish(h)
            assert np.array_equal(np.isfinite(got), ref <= frac * T)
            assert np.array_equal(got[np.isfinite(got)], ref[np.isfinite(got)])
        ns.netsim_advance(h)
        assert np.array_equal(ns.netsim_get_finish(h), ref)
        assert ns.netsim_get_stats(h)["complete"] == 1
        assert ns.netsim_num_checkpoints(h) == 4
    finally:
        ld.close()
    # by numbers of events
    ld = pr.load_program(program, ns.make_options(**ex))
    try:
        h = ld.handle
        for _ in range(100):
            ns.netsim_advance(h, max_events=97)
            if ns.netsim_get_stats(h)["complete"]:
                break
        assert np.array_equal(ns.netsim_get_finish(h), ref)
    finally:
        ld.close()


def _pick(fs, fin, lo, hi, with_deps):
    """A flow with bytes (with or without predecessors) finishing inside
    (lo, hi), else the one finishing closest to that window's middle."""
    has = np.diff(fs.dep_off) > 0
    ok = (fs.nbytes > 0) & (has == with_deps)
    cand = np.nonzero(ok & (fin > lo) & (fin < hi))[0]
    if len(cand):
        return int(cand[len(cand) // 2])
    cand = np.nonzero(ok)[0]
    return int(cand[np.argmin(np.abs(fin[cand] - 0.5 * (lo + hi)))])


@pytest.mark.parametrize("with_deps,delta", [(True, 30e-6), (True, -1.0), (False, 25e-6),
                                             (False, -1.0)])
def test_rollback_of_a_finished_flow(with_deps, delta):
    """The simulation has passed the flow's completion; its start moves (later,
    or as early as possible): the part rolls back and re-simulates."""
    ns, pr = _gpu()
    _say(f"test_rollback deps={with_deps} delta={delta}")
    program = configs.c2(2, tp_reps=6)
    sc = program.scenarios[0]
    fs = oflows.expand(sc)
    ref = _fresh(program, {})
    T = float(np.nanmax(ref))
    x = _pick(fs, ref, 0.2 * T, 0.4 * T, with_deps)
    new = max(0.0, float(fs.start[x]) + delta)
    if new == fs.start[x]:
        new = float(fs.start[x]) + 5e-6
    upd = {x: new}
    ld = pr.load_program(program)
    try:
        h = ld.handle
        ns.netsim_advance(h, until=0.3 * T)
        ns.netsim_advance(h, until=0.6 * T)
        ns.netsim_update_start(h, x, new)
        ns.netsim_advance(h)
        got = ns.netsim_get_finish(h)
    finally:
        ld.close()
    want = _fresh(program, upd)
    assert np.array_equal(got, want)
    assert not np.array_equal(want, ref)
    assert _rel(got, _oracle(sc, upd)) < TOL


def test_update_of_a_pending_flow_and_gc():
    """A flow not yet released whose new release stays in the future needs
    no rollback; garbage collection frees checkpoints without changing any
    later result; several updates in a row give the run with all of them."""
    ns, pr = _gpu()
    _say("test_update_pending_and_gc")
    program = configs.c2(2, tp_reps=6)
    sc = program.scenarios[0]
    fs = oflows.expand(sc)
    ref = _fresh(program, {})
    T = float(np.nanmax(ref))
    late = _pick(fs, ref, 0.85 * T, 0.95 * T, True)
    early = _pick(fs, ref, 0.5 * T, 0.7 * T, False)
    other = _pick(fs, ref, 0.75 * T, 0.8 * T, True)
    upd = {}
    ld = pr.load_program(program)
    try:
        h = ld.handle
        for frac in (0.1, 0.2, 0.3, 0.4):
            ns.netsim_advance(h, until=frac * T)
        upd[late] = float(fs.start[late]) + 40e-6
        ns.netsim_update_start(h, late, upd[late])
        n0 = ns.netsim_num_checkpoints(h)
        ns.netsim_gc(h, 0.35 * T)
        assert ns.netsim_num_checkpoints(h) < n0
        ns.netsim_advance(h, until=0.9 * T)
        upd[early] = float(fs.start[early]) + 10e-6
        ns.netsim_update_start(h, early, upd[early])
        ns.netsim_advance(h, until=0.95 * T)
        upd[other] = float(fs.start[other]) + 15e-6
        ns.netsim_update_start(h, other, upd[other])
        ns.netsim_advance(h)
        got = ns.netsim_get_finish(h)
    finally:
        ld.close()
    want = _fresh(program, upd)
    assert np.array_equal(got, want)
    assert _rel(got, _oracle(sc, upd)) < TOL


def test_rollback_random_micro_batch():
    """100 random dynamic micro cases in one batched handle: every case gets
    one flow's start moved after the simulation has passed half its horizon."""
    ns, pr = _gpu()
    _say("test_rollback_random_micro_batch")
    scs = []
    for seed in range(100):
        scs += micro.random_dynamic(500 + seed, integer_caps=(seed % 2 == 0)).scenarios
    program = Program("micro-rollback", scs)
    base = _fresh(program, {}, exec=ns.EXEC_BLOCK)
    ld = pr.load_program(program, ns.make_options(exec=ns.EXEC_BLOCK))
    try:
        h = ld.handle
        ms = np.array([np.nanmax(base[a:a + n]) for a, n in zip(ld.first_flow, ld.num_flows)])
        half = 0.5 * float(np.median(ms))
        rng = np.random.default_rng(7)
        upd = {}
        ns.netsim_advance(h, until=half)
        for s, sc in enumerate(scs):
            fs = oflows.expand(sc)
            loc = int(rng.integers(fs.F))
            upd[(s, loc)] = float(fs.start[loc]) + float(rng.uniform(0, 2.0)) * ms[s] / 10
            ns.netsim_update_start(h, ld.first_flow[s] + loc, upd[(s, loc)])
        ns.netsim_advance(h)
        got = ns.netsim_get_finish(h)
    finally:
        ld.close()
    want = _fresh(program, {ld.first_flow[s] + loc: v for (s, loc), v in upd.items()},
                  exec=ns.EXEC_BLOCK)
    assert np.array_equal(got, want)
    for s, sc in enumerate(scs):
        a = ld.first_flow[s]
        ref = _oracle(sc, {loc: v for (t, loc), v in upd.items() if t == s})
        assert _rel(got[a:a + ld.num_flows[s]], ref) < TOL, s
    assert not np.array_equal(got, base)


def _advance_update_finish(program, x, new, history_mb, **opt):
    """Advance to 30% and 60% of the horizon, move flow x's start, continue to
    the end: the finish times and the events the continuation processed."""
    ns, pr = _gpu()
    ref_T = opt.pop("T")
    ld = pr.load_program(program, ns.make_options(history_mb=history_mb, **opt))
    try:
        h = ld.handle
        ns.netsim_advance(h, until=0.3 * ref_T)
        ns.netsim_advance(h, until=0.6 * ref_T)
        ns.netsim_update_start(h, x, new)
        ns.netsim_advance(h)
        st = ns.netsim_get_stats(h)
        assert st["complete"] == 1
        return ns.netsim_get_finish(h), st["launch_events"]
    finally:
        ld.close()


@pytest.mark.parametrize("exec_", ["block", "grid", "cluster"])
@pytest.mark.parametrize("with_deps,delta", [(True, 30e-6), (True, -1.0), (False, 25e-6)])
def test_history_rollback_to_the_event_before(exec_, with_deps, delta):
    """With the rollback history the part goes back to the end of its last
    event before the changed release (not to the last checkpoint before it):
    the result equals, bit for bit, a fresh run with the new start and the
    rollback without history, and the continuation re-simulates no more
    events than the one from the checkpoint (fewer when the release is not
    at t = 0).  The cluster kernel keeps no history: there the rollback goes
    to the checkpoint either way."""
    ns, pr = _gpu()
    _say(f"test_history_rollback exec={exec_} deps={with_deps} delta={delta}")
    program = configs.c2(2, tp_reps=6)
    sc = program.scenarios[0]
    fs = oflows.expand(sc)
    lay = _layout(ns, exec_)
    ref = _fresh(program, {}, **lay)
    T = float(np.nanmax(ref))
    x = _pick(fs, ref, 0.2 * T, 0.4 * T, with_deps)
    new = max(0.0, float(fs.start[x]) + delta)
    if new == fs.start[x]:
        new = float(fs.start[x]) + 5e-6
    upd = {x: new}
    got, ev_hist = _advance_update_finish(program, x, new, 64, T=T, **lay)
    alt, ev_ckpt = _advance_update_finish(program, x, new, 0, T=T, **lay)
    want = _fresh(program, upd, **lay)
    assert np.array_equal(got, want)
    assert np.array_equal(alt, want)
    assert not np.array_equal(want, ref)
    if exec_ == "cluster":
        assert ev_hist == ev_ckpt
    else:
        assert ev_hist <= ev_ckpt
        if delta > 0:
            assert ev_hist < ev_ckpt
    _say("  continuation events: history", ev_hist, "checkpoint", ev_ckpt)
    assert _rel(got, _oracle(sc, upd)) < TOL


def test_history_several_updates_and_gc():
    """Several updates in a row (a pending flow, then finished flows after
    further advances) with the rollback history, garbage collection between
    them: the run with all of them, bit for bit."""
    ns, pr = _gpu()
    _say("test_history_several_updates_and_gc")
    program = configs.c2(2, tp_reps=6)
    sc = program.scenarios[0]
    fs = oflows.expand(sc)
    ref = _fresh(program, {})
    T = float(np.nanmax(ref))
    late = _pick(fs, ref, 0.85 * T, 0.95 * T, True)
    early = _pick(fs, ref, 0.5 * T, 0.7 * T, False)
    other = _pick(fs, ref, 0.75 * T, 0.8 * T, True)
    upd = {}
    ld = pr.load_program(program, ns.make_options(history_mb=64))
    try:
        h = ld.handle
        for frac in (0.1, 0.2, 0.3, 0.4):
            ns.netsim_advance(h, until=frac * T)
        upd[late] = float(fs.start[late]) + 40e-6
        ns.netsim_update_start(h, late, upd[late])
        ns.netsim_gc(h, 0.35 * T)
        ns.netsim_advance(h, until=0.9 * T)
        upd[early] = float(fs.start[early]) + 10e-6
        ns.netsim_update_start(h, early, upd[early])
        ns.netsim_advance(h, until=0.95 * T)
        upd[other] = float(fs.start[other]) + 15e-6
        ns.netsim_update_start(h, other, upd[other])
        ns.netsim_advance(h)
        got = ns.netsim_get_finish(h)
    finally:
        ld.close()
    want = _fresh(program, upd)
    assert np.array_equal(got, want)
    assert _rel(got, _oracle(sc, upd)) < TOL


def test_history_ring_too_small_falls_back_to_checkpoints():
    """A history of 1 MiB holds only the last few hundred events of C2: a
    rollback further back goes to the latest checkpoint instead, with the
    same result."""
    ns, pr = _gpu()
    _say("test_history_ring_too_small")
    program = configs.c2(2, tp_reps=6)
    sc = program.scenarios[0]
    fs = oflows.expand(sc)
    ref = _fresh(program, {})
    T = float(np.nanmax(ref))
    x = _pick(fs, ref, 0.2 * T, 0.4 * T, True)
    new = float(fs.start[x]) + 30e-6
    got, ev_small = _advance_update_finish(program, x, new, 1, T=T)
    _, ev_ckpt = _advance_update_finish(program, x, new, 0, T=T)
    assert np.array_equal(got, _fresh(program, {x: new}))
    assert ev_small == ev_ckpt


def test_history_rollback_random_micro_batch():
    """100 random dynamic micro cases in one batched handle with the rollback
    history: one flow's start moved in every case after half the horizon."""
    ns, pr = _gpu()
    _say("test_history_rollback_random_micro_batch")
    scs = []
    for seed in range(100):
        scs += micro.random_dynamic(500 + seed, integer_caps=(seed % 2 == 0)).scenarios
    program = Program("micro-rollback", scs)
    base = _fresh(program, {}, exec=ns.EXEC_BLOCK)
    ld = pr.load_program(program, ns.make_options(exec=ns.EXEC_BLOCK, history_mb=16))
    try:
        h = ld.handle
        ms = np.array([np.nanmax(base[a:a + n]) for a, n in zip(ld.first_flow, ld.num_flows)])
        half = 0.5 * float(np.median(ms))
        rng = np.random.default_rng(11)
        upd = {}
        ns.netsim_advance(h, until=half)
        for s, sc in enumerate(scs):
            fs = oflows.expand(sc)
            loc = int(rng.integers(fs.F))
            upd[(s, loc)] = float(fs.start[loc]) + float(rng.uniform(0, 2.0)) * ms[s] / 10
            ns.netsim_update_start(h, ld.first_flow[s] + loc, upd[(s, loc)])
        ns.netsim_advance(h)
        got = ns.netsim_get_finish(h)
    finally:
        ld.close()
    want = _fresh(program, {ld.first_flow[s] + loc: v for (s, loc), v in upd.items()},
                  exec=ns.EXEC_BLOCK)
    assert np.array_equal(got, want)
    for s, sc in enumerate(scs):
        a = ld.first_flow[s]
        ref = _oracle(sc, {loc: v for (t, loc), v in upd.items() if t == s})
        assert _rel(got[a:a + ld.num_flows[s]], ref) < TOL, s
    assert not np.array_equal(got, base)
