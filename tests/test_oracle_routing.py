"""Pins of the oracle's topology builder, router and collective
decomposition, and checks of the workload shapes (flow, link and
incidence counts) the configs are defined with."""

import numpy as np
import pytest

from oracle import flows
from oracle.topology import Fabric, ecmp_hash, splitmix
from workloads import configs
from workloads.program import MiB, GiB, Ring, Scenario, Topology
from workloads.rng import mix


def test_splitmix64_reference_values():
    """SplitMix64 started from state 0 yields 0xe220a8397b1dcdaf,
    0x6e789e6aa1b965f4, 0x06c45d188009454f (the published sequence)."""
    g = 0x9E3779B97F4A7C15
    want = [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]
    got = [int(splitmix(np.uint64((i * g) & (2**64 - 1)))) for i in range(3)]
    assert got == want
    assert [mix((i * g) & (2**64 - 1)) for i in range(3)] == want


def _contiguous(fab, fs):
    tail, head = fab.link_ends()
    for f in range(fs.F):
        p = fs.path_link[fs.path_off[f]:fs.path_off[f + 1]]
        if len(p) == 0:
            continue
        assert tail[p[0]] == fs.src[f] and head[p[-1]] == fs.dst[f]
        assert np.all(head[p[:-1]] == tail[p[1:]])
        assert len(set(p.tolist())) == len(p)


@pytest.mark.parametrize("name,kw", [
    ("c1", {}), ("c2", dict(tp_reps=2)), ("c3", dict(groups=2, background=300)),
    ("c4", dict(blocks=1, locals_=2)),
])
def test_routes_are_contiguous(name, kw):
    sc = configs.build(name, **kw).scenarios[0]
    _contiguous(Fabric(sc.topo), flows.expand(sc))


def test_routes_c5_contiguous():
    sc = configs.c5(5, scenarios=1, servers=128, servers_per_leaf=32).scenarios[0]
    _contiguous(Fabric(sc.topo), flows.expand(sc))


def test_route_lengths_and_link_counts():
    """Link counts and hop counts stated for the configs."""
    f1 = Fabric(configs.c1_topology(1))
    assert f1.L == 448 + 128 + 64 and f1.NV == 448
    f3 = Fabric(configs.c3_topology(3))
    assert f3.L == 6144 + 7168 and f3.ncab == 3072
    f4 = Fabric(configs.c4_topology(4))
    assert f4.L == 8192 + 8192 + 4096 + 28672
    # C4: per rank 63 peers = 1 same-edge (2 links) + 30 same-pod (4) + 32 other-pod (6)
    fs = flows.expand(configs.c4(4, blocks=1, locals_=1, phases=1).scenarios[0])
    lens = np.diff(fs.path_off)
    assert fs.F == 64 * 63 and np.sum(lens) == 64 * 314
    assert sorted(np.unique(lens)) == [2, 4, 6]
    # C3 ring hops: 112 intra-pod (4 links) and 16 inter-pod (6 links) per ring step
    fs = flows.expand(configs.c3(3, groups=1, background=0).scenarios[0])
    step0 = np.diff(fs.path_off)[:128]
    assert np.sum(step0 == 4) == 112 and np.sum(step0 == 6) == 16


def test_c1_hand_checked_route():
    """Rank 7 (server 0) -> rank 8 (server 1): NIC up of 7, leaf 0 -> spine h,
    spine h -> leaf 1, NIC down of 8, h = ECMP hash mod 4."""
    topo = configs.c1_topology(1)
    fab = Fabric(topo)
    off, link = fab.route(np.array([7]), np.array([8]))
    h = int(ecmp_hash(topo.ecmp_seed, np.array([7]), np.array([8]))[0]) % 4
    N = 64
    want = [448 + 2 * 7, 448 + 2 * (N + 0 * 4 + h), 448 + 2 * (N + 1 * 4 + h) + 1, 448 + 2 * 8 + 1]
    assert list(link) == want
    off, link = fab.route(np.array([3]), np.array([5]))   # same server: one NVLink
    assert list(link) == [0 * 56 + 3 * 7 + 4]


def test_ecmp_spread():
    """Across-pod C4 traffic spreads over aggregation switches and core
    uplinks about evenly (chi-square well below a loose bound)."""
    topo = configs.c4_topology(4)
    rng = np.random.default_rng(0)
    src = rng.integers(0, 2048, 50000)
    dst = rng.integers(2048, 4096, 50000)
    h = ecmp_hash(topo.ecmp_seed, src, dst)
    a = (h % np.uint64(16)).astype(int)
    u = ((h // np.uint64(16)) % np.uint64(8)).astype(int)
    for x, k in ((a, 16), (u, 8), (a * 8 + u, 128)):
        cnt = np.bincount(x, minlength=k)
        exp = len(x) / k
        chi2 = np.sum((cnt - exp) ** 2 / exp)
        assert chi2 < 3 * k


def test_ring_decomposition_modes():
    """Chained ring: 2(p-1) steps of p flows, step k out of position i waits
    for step k-1 into position i; flat: same flows, no chain; aggregated:
    p flows of 2(p-1)*S/p."""
    topo = Topology(kind="leaf_spine", servers=1, gpus_per_server=5, spines=1)
    ranks = np.array([4, 0, 3, 1, 2], np.int32)
    S = 10 * MiB
    for mode in ("chained", "flat", "aggregated"):
        sc = Scenario(topo)
        sc.add(Ring("allreduce", ranks, S, mode=mode, lag=0.5))
        fs = flows.expand(sc)
        p = 5
        if mode == "aggregated":
            assert fs.F == p and np.all(fs.nbytes == 8 * (S / p))
            assert list(fs.src) == list(ranks) and list(fs.dst) == list(np.roll(ranks, -1))
            continue
        assert fs.F == 8 * p and np.all(fs.nbytes == S / p)
        assert np.all(fs.src.reshape(8, p) == ranks) and np.all(fs.dst.reshape(8, p) == np.roll(ranks, -1))
        if mode == "flat":
            assert fs.dep_off[-1] == 0 and np.all(fs.start == 0.5)
        else:
            assert np.all(fs.start[:p] == 0.5) and np.all(fs.start[p:] == 0)
            for k in range(1, 8):
                for i in range(p):
                    f = k * p + i
                    d = fs.dep_ids[fs.dep_off[f]:fs.dep_off[f + 1]]
                    assert list(d) == [(k - 1) * p + (i - 1) % p]
                    assert fs.dst[d[0]] == fs.src[f]      # the flow into this rank
    sc = Scenario(topo)
    sc.add(Ring("reduce_scatter", ranks, S))
    sc.add(Ring("all_gather", ranks, S, after=(0,)))
    fs = flows.expand(sc)
    assert fs.F == 2 * 4 * 5
    # the all-gather's first step waits for every last-step flow of the reduce-scatter
    for i in range(5):
        d = fs.dep_ids[fs.dep_off[20 + i]:fs.dep_off[21 + i]]
        assert list(d) == list(range(15, 20))


def test_workload_sizes():
    """Flow, barrier and incidence counts the configs are specified with."""
    fs = flows.expand(configs.c1(1).scenarios[0])
    assert fs.F == 8064 and len(fs.path_link) == 11088
    fs = flows.expand(configs.c2(2).scenarios[0])
    assert fs.F == 45312 + 368 and int(np.sum(fs.nbytes == 0)) == 368
    assert len(fs.path_link) == 47616
    fs = flows.expand(configs.c3(3).scenarios[0])
    assert fs.F == 262096
    deg = Topology  # noqa: F841
    assert int(np.sum(fs.cap == 25e9)) == 614
    fs = flows.expand(configs.c4(4).scenarios[0])
    assert fs.F == 1032192 + 192 and len(fs.path_link) == 5144576
    assert len(np.unique(fs.path_link)) == 20480
    nz = fs.nbytes[fs.nbytes > 0]
    assert abs(np.mean(nz) / (4 * MiB) - 1) < 0.02
    assert np.min(nz) > 0.5 * MiB and np.max(nz) < 75 * MiB
    for s in range(3):
        tp, pp, nic, rho = configs.c5_params(5, s)
        fs = flows.expand(configs.c5(5, scenarios=1, first=s).scenarios[0])
        assert fs.F == 16384 + 2 * (pp - 1) * 16384 // pp
        dp = 16384 // (tp * pp)
        assert np.sum(fs.nbytes == 2 * (dp - 1) * (4 * GiB / dp)) == 16384


def test_c4_first_block_is_an_independent_prefix():
    """The full 4096-GPU all-to-all begins with the flows of its first
    64-server block, flow for flow those of the one-block workload (same
    routes, bytes, lags and dependencies), and no later flow shares a link
    with them or depends on them: the complete oracle run of the one-block
    workload is therefore the exact reference for those flows of the full
    run (a stored fixture of the GPU parity tests relies on this)."""
    a = flows.expand(configs.c4(4, blocks=1, locals_=8, phases=4).scenarios[0])
    b = flows.expand(configs.c4(4).scenarios[0])
    F, nnz, nd = a.F, int(a.path_off[-1]), int(a.dep_off[-1])
    assert F == 129048 and b.F == 8 * F
    for k in ("src", "dst", "nbytes", "start"):
        assert np.array_equal(getattr(a, k), getattr(b, k)[:F]), k
    assert np.array_equal(a.cap, b.cap)
    assert np.array_equal(a.path_off, b.path_off[:F + 1])
    assert np.array_equal(a.path_link, b.path_link[:nnz])
    assert np.array_equal(a.dep_off, b.dep_off[:F + 1])
    assert np.array_equal(a.dep_ids, b.dep_ids[:nd])
    used = np.zeros(len(b.cap), bool)
    used[a.path_link] = True
    assert not used[b.path_link[nnz:]].any()
    assert not (b.dep_ids[nd:] < F).any()
