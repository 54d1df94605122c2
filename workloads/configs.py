"""The five synthetic workloads (and scaled-down variants for tests).

Sizes are binary (MiB = 2**20 B, GiB = 2**30 B); link rates in bytes per
second ("X Gb/s" = X*1e9/8 B/s).  Every random quantity is drawn from a
named counter-based stream of ``workloads.rng`` keyed by the seed.

C1  64 GPUs, 2-tier leaf-spine, one 256 MiB ring all-reduce.
C2  128 GPUs, rail-optimised; TP=8 all-reduces (x24, barrier-chained),
    GPipe PP=4 sends, DP=4 ring all-reduce, start jitter U[0, 50 us].
C3  1024 GPUs, k=16 fat-tree, 10% degraded cables; 8 DP groups doing
    reduce-scatter + all-gather (one chained all-reduce) of 2 GiB, plus
    2000 log-uniform background sends.
C4  4096 GPUs, 3-tier fat-tree, 2:1 at the core; 64 expert-parallel groups
    of 64 ranks, 4 back-to-back all-to-all phases with Zipf(1.2) bytes.
C5  256 what-if scenarios on a 16384-GPU rail fabric (TP, PP, NIC rate and
    spine oversubscription drawn per scenario); aggregated DP ring plus
    aggregated PP sends.
"""

from __future__ import annotations

import numpy as np

from .program import (GiB, MiB, AllToAll, Barrier, Program, Ring, Scenario,
                      Send, Topology, gbit)
from .rng import Stream

JITTER = 50e-6


def _ecmp_seed(seed: int, tag: str = "ecmp") -> int:
    return int(Stream(seed, tag).u64(1)[0])


# --------------------------------------------------------------------- C1
def c1_topology(seed: int = 1) -> Topology:
    return Topology(kind="leaf_spine", servers=8, gpus_per_server=8,
                    servers_per_leaf=1, spines=4, nvlink_Bps=900e9,
                    nic_Bps=gbit(400), fabric_Bps=gbit(800),
                    ecmp_seed=_ecmp_seed(seed))


def c1(seed: int = 1, mode: str = "chained", nbytes: float = 256 * MiB) -> Program:
    """One ring all-reduce of 256 MiB over ranks 0..63 in rank order."""
    sc = Scenario(c1_topology(seed))
    sc.add(Ring("allreduce", np.arange(64, dtype=np.int32), nbytes, mode=mode))
    return Program(f"c1-{mode}", [sc])


# --------------------------------------------------------------------- C2
def c2(seed: int = 2, tp_reps: int = 24, microbatches: int = 8) -> Program:
    """3D-parallel step on 128 GPUs: rank = tp + 8*(dp + 4*pp)."""
    TP, DP, PP = 8, 4, 4
    topo = Topology(kind="rail", servers=16, gpus_per_server=8,
                    servers_per_leaf=16, spines=8, nvlink_Bps=900e9,
                    nic_Bps=gbit(400), fabric_Bps=gbit(800),
                    ecmp_seed=_ecmp_seed(seed))
    sc = Scenario(topo)
    jit = Stream(seed, "c2-jitter")
    nj = [0]

    def lag() -> float:
        v = float(jit.u01(1, nj[0])[0]) * JITTER
        nj[0] += 1
        return v

    def rank(tp, dp, pp):
        return tp + TP * (dp + DP * pp)

    # TP all-reduces inside each server, repeated and chained by barriers.
    for server in range(16):
        ranks = np.arange(8 * server, 8 * server + 8, dtype=np.int32)
        prev_barrier = None
        for rep in range(tp_reps):
            after = () if prev_barrier is None else (prev_barrier,)
            op = sc.add(Ring("allreduce", ranks, 32 * MiB, lag=lag(), after=after))
            if rep + 1 < tp_reps:
                prev_barrier = sc.add(Barrier(after=(op,)))
    # GPipe pipeline sends, forward then backward.
    for tp in range(TP):
        for dp in range(DP):
            fwd = {}
            for m in range(microbatches):
                for b in range(PP - 1):
                    after = []
                    if b > 0:
                        after.append(fwd[(b - 1, m)])
                    if m > 0:
                        after.append(fwd[(b, m - 1)])
                    lg = lag() if not after else 0.0
                    fwd[(b, m)] = sc.add(Send(rank(tp, dp, b), rank(tp, dp, b + 1),
                                              16 * MiB, lag=lg, after=tuple(after)))
            bwd = {}
            for m in range(microbatches):
                for b in range(PP - 2, -1, -1):
                    after = []
                    if b < PP - 2:
                        after.append(bwd[(b + 1, m)])
                    if m > 0:
                        after.append(bwd[(b, m - 1)])
                    if b == PP - 2 and m == 0:
                        after.append(fwd[(PP - 2, microbatches - 1)])
                    bwd[(b, m)] = sc.add(Send(rank(tp, dp, b + 1), rank(tp, dp, b),
                                              16 * MiB, after=tuple(after)))
    # DP ring all-reduce of the gradients.
    for tp in range(TP):
        for pp in range(PP):
            ranks = np.array([rank(tp, d, pp) for d in range(DP)], dtype=np.int32)
            sc.add(Ring("allreduce", ranks, 1 * GiB, lag=lag()))
    return Program("c2", [sc])


# --------------------------------------------------------------------- C3
def c3_topology(seed: int = 3, degrade_frac: float = 0.1) -> Topology:
    topo = Topology(kind="fat_tree", servers=128, gpus_per_server=8,
                    servers_per_leaf=1, pods=16, edges_per_pod=8,
                    aggs_per_pod=8, agg_uplinks=8, nvlink_Bps=900e9,
                    nic_Bps=gbit(400), fabric_Bps=gbit(400),
                    ecmp_seed=_ecmp_seed(seed), degraded_Bps=gbit(200))
    n = topo.num_cables()
    k = int(np.floor(degrade_frac * n))
    topo.degraded = Stream(seed, "c3-degrade").sample_without_replacement(n, k)
    return topo


def c3(seed: int = 3, groups: int = 8, background: int = 2000,
       nbytes: float = 2 * GiB) -> Program:
    sc = Scenario(c3_topology(seed))
    for g in range(groups):
        ranks = np.array([8 * s + g for s in range(128)], dtype=np.int32)
        # reduce-scatter followed by all-gather on the same ring, each step
        # waiting for the previous one = one chained ring all-reduce.
        sc.add(Ring("allreduce", ranks, nbytes))
    n = sc.topo.endpoints
    st = Stream(seed, "c3-background")
    u = st.u01(4 * background)
    for i in range(background):
        src = min(int(u[4 * i] * n), n - 1)
        dst = min(int(u[4 * i + 1] * (n - 1)), n - 2)
        if dst >= src:
            dst += 1
        nb = float(np.rint(2.0 ** (20.0 + 6.0 * u[4 * i + 2])))
        start = float(u[4 * i + 3]) * 0.1
        sc.add(Send(src, dst, nb, lag=start))
    return Program("c3", [sc])


# --------------------------------------------------------------------- C4
ZIPF_S = 1.2


def c4_topology(seed: int = 4) -> Topology:
    return Topology(kind="fat_tree", servers=512, gpus_per_server=8,
                    servers_per_leaf=2, pods=16, edges_per_pod=16,
                    aggs_per_pod=16, agg_uplinks=8, nvlink_Bps=900e9,
                    nic_Bps=gbit(400), fabric_Bps=gbit(400),
                    ecmp_seed=_ecmp_seed(seed))


def zipf_dispatch_bytes(seed: int, group: int, phase: int, p: int = 64,
                        mean: float = 4 * MiB, s: float = ZIPF_S) -> np.ndarray:
    """p x p dispatch matrix: bytes(i->j) = round(mean*p*w_j/W), w_j=(pi(j)+1)^-s.

    pi is a seeded permutation per (group, phase); W = sum_{k=1..p} k^-s.
    The diagonal is set to zero.
    """
    perm = Stream(seed, f"c4-zipf-{group}-{phase}").permutation(p)
    W = float(np.sum(np.arange(1, p + 1, dtype=np.float64) ** (-s)))
    w = (perm.astype(np.float64) + 1.0) ** (-s)
    col = np.rint(mean * p * w / W)
    m = np.tile(col, (p, 1))
    np.fill_diagonal(m, 0.0)
    return m


def c4(seed: int = 4, blocks: int = 8, locals_: int = 8, phases: int = 4,
       zipf_s: float = ZIPF_S) -> Program:
    """Expert-parallel all-to-all: group (b, l) = local GPU l on servers
    64b..64b+63.  Phases 0, 2 dispatch; 1, 3 are the transposes (combine).
    Phase k+1 of a group waits for a barrier over phase k of that group,
    plus a per-(group, phase) lag drawn from U[0, 50 us]."""
    sc = Scenario(c4_topology(seed))
    jit = Stream(seed, "c4-jitter")
    for b in range(blocks):
        for l in range(locals_):
            g = b * 8 + l
            ranks = np.array([8 * (64 * b + s) + l for s in range(64)], dtype=np.int32)
            lags = jit.u01(phases, start=g * 16) * JITTER
            prev_barrier = None
            disp = None
            for ph in range(phases):
                if ph % 2 == 0:
                    disp = zipf_dispatch_bytes(seed, g, ph, s=zipf_s)
                    mat = disp
                else:
                    mat = disp.T.copy()
                after = () if prev_barrier is None else (prev_barrier,)
                op = sc.add(AllToAll(ranks, mat, lag=float(lags[ph]), after=after))
                if ph + 1 < phases:
                    prev_barrier = sc.add(Barrier(after=(op,)))
    return Program("c4", [sc])


# --------------------------------------------------------------------- C5
def c5_params(seed: int, scen: int):
    u = Stream(seed, f"c5-scenario-{scen}").u01(4)
    tp = (4, 8)[min(int(u[0] * 2), 1)]
    pp = (4, 8, 16)[min(int(u[1] * 3), 2)]
    nic = (200, 400, 800)[min(int(u[2] * 3), 2)]
    rho = (1, 2, 4)[min(int(u[3] * 3), 2)]
    return tp, pp, nic, rho


def c5_scenario(seed: int, scen: int, servers: int = 2048,
                servers_per_leaf: int = 32) -> Scenario:
    tp, pp, nic, rho = c5_params(seed, scen)
    n = servers * 8
    dp = n // (tp * pp)
    topo = Topology(kind="rail", servers=servers, gpus_per_server=8,
                    servers_per_leaf=servers_per_leaf,
                    spines=max(1, servers_per_leaf // rho),
                    nvlink_Bps=900e9, nic_Bps=gbit(nic), fabric_Bps=gbit(nic),
                    ecmp_seed=_ecmp_seed(seed, f"c5-ecmp-{scen}"))
    sc = Scenario(topo)

    def rank(t, p, d):
        return t + tp * (p + pp * d)

    for t in range(tp):
        for p in range(pp):
            ranks = np.array([rank(t, p, d) for d in range(dp)], dtype=np.int32)
            sc.add(Ring("allreduce", ranks, 4 * GiB, mode="aggregated"))
    for t in range(tp):
        for d in range(dp):
            for b in range(pp - 1):
                sc.add(Send(rank(t, b, d), rank(t, b + 1, d), 8 * 16 * MiB))
                sc.add(Send(rank(t, b + 1, d), rank(t, b, d), 8 * 16 * MiB))
    return sc


def c5(seed: int = 5, scenarios: int = 256, servers: int = 2048,
       servers_per_leaf: int = 32, first: int = 0) -> Program:
    prog = Program("c5")
    for s in range(first, first + scenarios):
        prog.scenarios.append(c5_scenario(seed, s, servers, servers_per_leaf))
    return prog


CONFIGS = {"c1": c1, "c2": c2, "c3": c3, "c4": c4, "c5": c5}
DEFAULT_SEEDS = {"c1": 1, "c2": 2, "c3": 3, "c4": 4, "c5": 5}


def build(name: str, seed: int = None, **kw) -> Program:
    if seed is None:
        seed = DEFAULT_SEEDS[name]
    return CONFIGS[name](seed, **kw)
