"""Plain pure-Python forms of the simulator, for small cases only.

TEST INFRASTRUCTURE (see ``oracle/__init__.py``).

``simulate(fs, exact=True)`` runs the fluid model in exact rational
arithmetic (``fractions.Fraction``): ties are exact equalities, so no
tolerance band is needed.  ``simulate(fs, exact=False)`` runs the same
steps in fp64 with the tie bands of the fp64 oracle (THR = 1 + 1e-12 on
the bottleneck share and on the completion time), in the sweep form
written in the paper's terms (Section 4.2: find the bottleneck link, give
its flows their share, repeat; rates constant between events).

``brute_force_maxmin`` checks the max-min allocation of a static active
set without progressive filling: it tries every order in which links could
be fixed, keeps the candidates that are feasible and satisfy the
bottleneck property, and returns all distinct survivors (the max-min fair
allocation is unique, so exactly one should survive; Bertsekas and
Gallager, Data Networks, 2nd ed., Section 6.5).
"""

from __future__ import annotations

import itertools
from fractions import Fraction

THR = 1.000000000001


def _paths(fs):
    return [list(map(int, fs.path_link[fs.path_off[f]:fs.path_off[f + 1]])) for f in range(fs.F)]


def maxmin(paths, caps, active, exact):
    """Progressive filling over ``active`` (flow indices); returns {f: rate}."""
    num = Fraction if exact else float
    R = {}
    n = {}
    for f in active:
        for l in paths[f]:
            if l not in R:
                R[l] = num(caps[l])
                n[l] = 0
            n[l] += 1
    U = set(active)
    rate = {}
    iters = 0
    while U:
        share = {l: R[l] / n[l] for l in R if n[l] > 0}
        s = min(share.values())
        assert s > 0
        iters += 1
        if exact:
            B = {l for l, v in share.items() if v == s}
        else:
            thr = s * THR
            B = {l for l, v in share.items() if v <= thr}
        frozen = [f for f in U if any(l in B for l in paths[f])]
        k = {}
        for f in frozen:
            rate[f] = s
            for l in paths[f]:
                k[l] = k.get(l, 0) + 1
        for l, kl in k.items():
            R[l] = R[l] - (num(kl) * s)
            n[l] -= kl
        U.difference_update(frozen)
    return rate, iters


def simulate(fs, exact: bool = True):
    """Event loop; returns (finish list, events, solves, iterations)."""
    num = Fraction if exact else float
    F = fs.F
    paths = _paths(fs)
    caps = [num(float(c)) for c in fs.cap]
    nbytes = [num(float(b)) for b in fs.nbytes]
    start = [num(float(s)) for s in fs.start]
    lat = ([num(float(x)) for x in fs.lat] if getattr(fs, "lat", None) is not None
           else [num(0)] * F)
    deps = [list(map(int, fs.dep_ids[fs.dep_off[f]:fs.dep_off[f + 1]])) for f in range(F)]
    succ = [[] for _ in range(F)]
    for g in range(F):
        for d in deps[g]:
            succ[d].append(g)
    cnt = [len(d) for d in deps]
    rel_base = [num(0)] * F
    finish = [None] * F
    pending = {f: start[f] for f in range(F) if cnt[f] == 0}
    active = {}
    rate = {}
    t = num(0)
    events = solves = iterations = 0
    while active or pending:
        t_arr = min(pending.values()) if pending else None
        tau = {f: t + active[f] / rate[f] for f in active}
        cands = list(tau.values()) + ([t_arr] if t_arr is not None else [])
        t_next = min(cands)
        events += 1
        if exact:
            done = [f for f in active if tau[f] == t_next]
        else:
            thr = t_next * THR
            done = [f for f in active if tau[f] <= thr]
        step = t_next - t
        for f in list(active):
            if f in done:
                finish[f] = t_next + lat[f]  # last byte sent at t_next, arrives lat later
                del active[f]
            else:
                active[f] = active[f] - rate[f] * step
        t = t_next
        changed = bool(done)
        queue = list(done)
        while True:
            while queue:
                f = queue.pop()
                for g in succ[f]:
                    if finish[f] > rel_base[g]:
                        rel_base[g] = finish[f]
                    cnt[g] -= 1
                    if cnt[g] == 0:
                        pending[g] = start[g] + rel_base[g]
            arrived = [g for g, r in pending.items() if r <= t]
            if not arrived:
                break
            for g in arrived:
                r = pending.pop(g)
                if nbytes[g] == 0:
                    finish[g] = r
                    queue.append(g)
                else:
                    active[g] = nbytes[g]
                    changed = True
        if changed and active:
            rate, it = maxmin(paths, caps, list(active), exact)
            solves += 1
            iterations += it
    return finish, events, solves, iterations


def _check_maxmin(paths, caps, alloc):
    """Feasibility and the bottleneck property, in exact arithmetic."""
    load = {}
    for f, r in alloc.items():
        for l in paths[f]:
            load[l] = load.get(l, 0) + r
    for l, v in load.items():
        if v > caps[l]:
            return False
    for f, r in alloc.items():
        ok = False
        for l in paths[f]:
            if load[l] == caps[l] and all(alloc[g] <= r for g in alloc if l in paths[g]):
                ok = True
                break
        if not ok:
            return False
    return True


def brute_force_maxmin(paths, caps):
    """All distinct feasible allocations with the bottleneck property among
    the 'fix links one at a time' candidates (exact arithmetic)."""
    caps = [Fraction(c) for c in caps]
    flows = [f for f in range(len(paths)) if paths[f]]
    links = sorted({l for f in flows for l in paths[f]})
    found = []
    for order in itertools.permutations(links):
        alloc = {}
        ok = True
        for l in order:
            on = [f for f in flows if l in paths[f]]
            free = [f for f in on if f not in alloc]
            if not free:
                continue
            rest = caps[l] - sum((alloc[f] for f in on if f in alloc), Fraction(0))
            if rest <= 0:
                ok = False
                break
            v = rest / len(free)
            for f in free:
                alloc[f] = v
        if not ok or len(alloc) != len(flows):
            continue
        if _check_maxmin(paths, caps, alloc):
            key = tuple(alloc[f] for f in flows)
            if key not in found:
                found.append(key)
    return flows, found
