"""The usage example of README.md, run as written: a ring all-reduce over
64 GPUs on a leaf-spine fabric, then an all-to-all among eight of them that
starts when the ring's last step has finished."""

import numpy as np
import pytest

pytestmark = pytest.mark.gpu


def test_readme_example():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2505_01616_amd import netsim as ns

    MiB = 2**20
    topo = ns.netsim_topology()
    topo.kind = ns.TOPO_LEAF_SPINE
    topo.servers, topo.gpus_per_server, topo.servers_per_leaf, topo.spines = 8, 8, 1, 4
    topo.nvlink_Bps, topo.nic_Bps, topo.fabric_Bps = 900e9, 50e9, 100e9
    topo.ecmp_seed = 1
    h = ns.netsim_create_topology([topo])
    try:
        ring_first, ring_n = ns.netsim_add_ring(h, 0, ns.RING_ALLREDUCE, ns.MODE_CHAINED,
                                                np.arange(64), 256 * MiB)
        ring_exits = ns.netsim_last_exits(h)          # the ring's last step
        a2a_first, a2a_n = ns.netsim_add_all_to_all(h, 0, np.arange(0, 64, 8),
                                                    np.full(64, 4 * MiB), after=ring_exits)
        ns.netsim_run(h)
        finish = ns.netsim_get_finish(h)              # per flow, seconds
        stats = ns.netsim_get_stats(h)
    finally:
        ns.netsim_destroy(h)
    assert ring_n == 2 * 63 * 64 and a2a_n == 8 * 7
    ring_end = finish[ring_first:ring_first + ring_n].max()
    a2a = finish[a2a_first:a2a_first + a2a_n]
    assert np.all(a2a > ring_end)                     # the all-to-all waited for the ring
    assert stats["complete"] == 1 and stats["sim_time"] == finish.max()
