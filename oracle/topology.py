"""Oracle side: cluster links, capacities and ECMP routes.

TEST INFRASTRUCTURE.  Only the tests, the smoke check and the benchmark's
CPU-baseline leg use this package; the simulator library never does.

The paper's simulator takes a topology configuration with port bandwidths,
the interconnect and the multipath routing / load-balancing rule
(Section 4.1, description of netsim).  The paper names no concrete fabric
and no hash, so this module fixes one reading of each, written out here in
plain numpy:

Link numbering (directed links; a cable is two links at full rate):
  * intra-server links first: server s, ordered GPU pair (i -> j), i != j,
    id = s*G*(G-1) + i*(G-1) + (j if j < i else j-1);
  * then cable c gives link NV + 2c (upward: towards the higher tier)
    and NV + 2c + 1 (downward).
Cable order:
  * NIC cables c = h for every GPU h (host <-> its leaf / edge switch);
  * leaf_spine / rail: cable N + leaf*S + spine;
    leaf_spine leaf = server // servers_per_leaf;
    rail leaf = local_gpu * groups + server // servers_per_leaf;
  * fat_tree: edge-agg cable N + (pod*E + e)*A + a, then agg-core cable
    N + P*E*A + (pod*A + a)*U + u (core a*U + u).
Routes (src != dst):
  * same server: the one intra-server link;
  * same leaf / edge switch: NIC up, NIC down;
  * leaf_spine / rail: NIC up, leaf->spine, spine->leaf, NIC down,
    spine = h mod S;
  * fat_tree same pod: NIC up, edge->agg, agg->edge, NIC down, agg = h mod A;
  * fat_tree across pods: NIC up, edge->agg, agg->core, core->agg,
    agg->edge, NIC down, agg = h mod A, core uplink u = (h div A) mod U.
ECMP hash h = mix(mix(seed) XOR (src << 32 | dst)), mix = SplitMix64's
output function (Steele, Lea and Flood, OOPSLA 2014).
"""

from __future__ import annotations

import numpy as np

_GOLDEN = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)


def splitmix(x: np.ndarray) -> np.ndarray:
    with np.errstate(over="ignore"):
        z = np.asarray(x, dtype=np.uint64) + _GOLDEN
        z = (z ^ (z >> np.uint64(30))) * _M1
        z = (z ^ (z >> np.uint64(27))) * _M2
        return z ^ (z >> np.uint64(31))


def ecmp_hash(seed: int, src: np.ndarray, dst: np.ndarray) -> np.ndarray:
    key = splitmix(np.uint64(seed & ((1 << 64) - 1)))
    v = (src.astype(np.uint64) << np.uint64(32)) | dst.astype(np.uint64)
    return splitmix(key ^ v)


class Fabric:
    """Links, capacities and a router for one workloads.Topology."""

    def __init__(self, topo):
        self.t = topo
        self.kind = topo.kind
        if self.kind == "explicit":
            self.cap = np.asarray(topo.capacities, dtype=np.float64).copy()
            self.L = len(self.cap)
            lat = getattr(topo, "latencies", None)
            self.lat = (np.zeros(self.L) if lat is None
                        else np.asarray(lat, dtype=np.float64).copy())
            return
        G, S = topo.gpus_per_server, topo.servers
        self.G, self.S, self.N = G, S, G * S
        self.NV = S * G * (G - 1)
        if self.kind == "leaf_spine":
            self.leaves = S // topo.servers_per_leaf
            self.ncab = self.N + self.leaves * topo.spines
        elif self.kind == "rail":
            self.groups = S // topo.servers_per_leaf
            self.leaves = G * self.groups
            self.ncab = self.N + self.leaves * topo.spines
        elif self.kind == "fat_tree":
            P, E, A, U = topo.pods, topo.edges_per_pod, topo.aggs_per_pod, topo.agg_uplinks
            self.ncab = self.N + P * E * A + P * A * U
        else:
            raise ValueError(f"unknown topology kind {self.kind}")
        self.L = self.NV + 2 * self.ncab
        cap = np.empty(self.L, dtype=np.float64)
        cap[: self.NV] = topo.nvlink_Bps
        cab = np.full(self.ncab, topo.fabric_Bps, dtype=np.float64)
        cab[: self.N] = topo.nic_Bps
        if len(topo.degraded):
            cab[np.asarray(topo.degraded, dtype=np.int64)] = topo.degraded_Bps
        cap[self.NV::2] = cab
        cap[self.NV + 1::2] = cab
        self.cap = cap
        # link latency: NVLink links, then every cable direction
        self.lat = np.empty(self.L, dtype=np.float64)
        self.lat[: self.NV] = getattr(topo, "nvlink_latency_s", 0.0)
        self.lat[self.NV:] = getattr(topo, "fabric_latency_s", 0.0)

    # ---- link end nodes (for checking routes) -----------------------------
    def link_ends(self):
        """(tail, head) node of every link.  Nodes: GPUs 0..N-1, then
        switches (leaf_spine / rail: leaves, spines; fat_tree: edges, aggs,
        cores)."""
        t = self.t
        N, G = self.N, self.G
        tail = np.empty(self.L, np.int64)
        head = np.empty(self.L, np.int64)
        s = np.repeat(np.arange(self.S), G * (G - 1))
        i = np.tile(np.repeat(np.arange(G), G - 1), self.S)
        jj = np.tile(np.tile(np.arange(G - 1), G), self.S)
        j = np.where(jj < i, jj, jj + 1)
        tail[: self.NV] = s * G + i
        head[: self.NV] = s * G + j
        lo = np.empty(self.ncab, np.int64)
        hi = np.empty(self.ncab, np.int64)
        h = np.arange(N)
        lo[:N] = h
        if self.kind in ("leaf_spine", "rail"):
            if self.kind == "leaf_spine":
                leaf = (h // G) // t.servers_per_leaf
            else:
                leaf = (h % G) * self.groups + (h // G) // t.servers_per_leaf
            hi[:N] = N + leaf
            q = np.repeat(np.arange(self.leaves), t.spines)
            p = np.tile(np.arange(t.spines), self.leaves)
            lo[N:] = N + q
            hi[N:] = N + self.leaves + p
        else:
            P, E, A, U = t.pods, t.edges_per_pod, t.aggs_per_pod, t.agg_uplinks
            edge0, agg0, core0 = N, N + P * E, N + P * E + P * A
            hi[:N] = edge0 + (h // G) // t.servers_per_leaf
            pe = np.repeat(np.arange(P * E), A)           # pod*E + e
            a = np.tile(np.arange(A), P * E)
            lo[N:N + P * E * A] = edge0 + pe
            hi[N:N + P * E * A] = agg0 + (pe // E) * A + a
            pa = np.repeat(np.arange(P * A), U)           # pod*A + a
            u = np.tile(np.arange(U), P * A)
            lo[N + P * E * A:] = agg0 + pa
            hi[N + P * E * A:] = core0 + (pa % A) * U + u
        tail[self.NV::2], head[self.NV::2] = lo, hi
        tail[self.NV + 1::2], head[self.NV + 1::2] = hi, lo
        return tail, head

    # ---- link ids -------------------------------------------------------
    def up(self, cable):
        return self.NV + 2 * cable

    def down(self, cable):
        return self.NV + 2 * cable + 1

    def nvlink(self, server, i, j):
        G = self.G
        return server * G * (G - 1) + i * (G - 1) + np.where(j < i, j, j - 1)

    # ---- routing --------------------------------------------------------
    def route(self, src: np.ndarray, dst: np.ndarray):
        """Paths for endpoint pairs (src != dst): (off[F+1] int64, link[] int32)."""
        t = self.t
        src = np.asarray(src, dtype=np.int64)
        dst = np.asarray(dst, dtype=np.int64)
        F = len(src)
        G = self.G
        hops = np.full((F, 6), -1, dtype=np.int64)
        ns = src // G
        nd = dst // G
        same_server = ns == nd
        h = ecmp_hash(t.ecmp_seed, src, dst)
        if self.kind in ("leaf_spine", "rail"):
            spl = t.servers_per_leaf
            if self.kind == "leaf_spine":
                ls, ld = ns // spl, nd // spl
            else:
                ls = (src % G) * self.groups + ns // spl
                ld = (dst % G) * self.groups + nd // spl
            same_leaf = (~same_server) & (ls == ld)
            via = (~same_server) & (~same_leaf)
            sp = (h % np.uint64(t.spines)).astype(np.int64)
            hops[same_leaf, 0] = self.up(src[same_leaf])
            hops[same_leaf, 1] = self.down(dst[same_leaf])
            hops[via, 0] = self.up(src[via])
            hops[via, 1] = self.up(self.N + ls[via] * t.spines + sp[via])
            hops[via, 2] = self.down(self.N + ld[via] * t.spines + sp[via])
            hops[via, 3] = self.down(dst[via])
        else:
            P, E, A, U = t.pods, t.edges_per_pod, t.aggs_per_pod, t.agg_uplinks
            es, ed = ns // t.servers_per_leaf, nd // t.servers_per_leaf
            ps, pd = es // E, ed // E
            same_edge = (~same_server) & (es == ed)
            same_pod = (~same_server) & (~same_edge) & (ps == pd)
            cross = (~same_server) & (~same_edge) & (ps != pd)
            a = (h % np.uint64(A)).astype(np.int64)
            u = ((h // np.uint64(A)) % np.uint64(U)).astype(np.int64)
            ea_s = self.N + es * A + a          # es = pod*E + e already
            ea_d = self.N + ed * A + a
            base_ac = self.N + P * E * A
            ac_s = base_ac + (ps * A + a) * U + u
            ac_d = base_ac + (pd * A + a) * U + u
            m = same_edge
            hops[m, 0] = self.up(src[m])
            hops[m, 1] = self.down(dst[m])
            m = same_pod
            hops[m, 0] = self.up(src[m])
            hops[m, 1] = self.up(ea_s[m])
            hops[m, 2] = self.down(ea_d[m])
            hops[m, 3] = self.down(dst[m])
            m = cross
            hops[m, 0] = self.up(src[m])
            hops[m, 1] = self.up(ea_s[m])
            hops[m, 2] = self.up(ac_s[m])
            hops[m, 3] = self.down(ac_d[m])
            hops[m, 4] = self.down(ea_d[m])
            hops[m, 5] = self.down(dst[m])
        m = same_server
        hops[m, 0] = self.nvlink(ns[m], src[m] % G, dst[m] % G)
        lens = (hops >= 0).sum(axis=1)
        off = np.zeros(F + 1, dtype=np.int64)
        np.cumsum(lens, out=off[1:])
        link = hops[hops >= 0].astype(np.int32)   # row-major keeps hop order
        return off, link
