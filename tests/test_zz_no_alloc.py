"""The allocation-free rate solve (netsim_solve_rates_noalloc) against the
entry point it is a variant of, netsim_solve_once in exact mode: two calls in
a row on one device, the second with a smaller input, bit for bit; then a
bad path reported through the device status word, and a good call after it."""

import sys

import numpy as np
import pytest

from workloads import configs

pytestmark = pytest.mark.gpu


def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2505_01616_amd import netsim as ns
    from paper_2505_01616_amd import program as prog
    return torch, ns, prog


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


def _reference(ns, pr, program):
    """Rates of every routed flow of scenario 0 from netsim_solve_once (exact
    mode), with the flows' paths and the scenario's capacities."""
    ld = pr.load_program(program, ns.make_options(exact=1))
    try:
        fl = ns.netsim_export_flows(ld.handle)
        cap = ns.netsim_get_links(ld.handle, 0)
        ids = np.nonzero(fl["nbytes"] > 0)[0]
        rates = ns.netsim_solve_once(ld.handle, 0, ids)
        levels = ns.netsim_get_stats(ld.handle)["rounds"]
    finally:
        ld.close()
    lens = np.diff(fl["path_off"])[ids]
    poff = np.zeros(len(ids) + 1, np.int32)
    np.cumsum(lens, out=poff[1:])
    plink = np.concatenate([fl["path_link"][fl["path_off"][i]:fl["path_off"][i + 1]] for i in ids])
    return cap, poff, plink.astype(np.int32), rates, levels


def _noalloc(torch, ns, cap, poff, plink):
    dev = torch.device("cuda:0")
    d_cap = torch.from_numpy(cap).to(dev)
    d_poff = torch.from_numpy(poff).to(dev)
    d_plink = torch.from_numpy(plink).to(dev)
    F = len(poff) - 1
    d_rates = torch.full((max(F, 1),), -1.0, dtype=torch.float64, device=dev)
    d_status = torch.full((2,), 7, dtype=torch.int64, device=dev)
    torch.cuda.synchronize()
    ns.netsim_solve_rates_noalloc(0, len(cap), d_cap.data_ptr(), F, d_poff.data_ptr(),
                                  d_plink.data_ptr(), d_rates.data_ptr(), d_status.data_ptr(),
                                  torch.cuda.current_stream())
    torch.cuda.synchronize()
    return d_rates.cpu().numpy()[:F], d_status.cpu().numpy()


def test_noalloc_equals_solve_once_twice_then_bad_input():
    torch, ns, pr = _gpu()
    # first call: one all-to-all phase of two 64-rank expert groups on the
    # 4096-GPU fabric (8,064 flows); second: a smaller flat ring (16 ranks of C1, 480 flows)
    big = configs.c4(4, blocks=1, locals_=2, phases=1)
    small = configs.c1(1, mode="flat")
    small.scenarios[0].ops[0].ranks = small.scenarios[0].ops[0].ranks[:16]
    for name, program in (("c4-two-groups", big), ("c1-sixteen-ranks", small)):
        cap, poff, plink, want, levels = _reference(ns, pr, program)
        _say(f"noalloc {name}: {len(poff) - 1} flows, {len(cap)} links")
        got, status = _noalloc(torch, ns, cap, poff, plink)
        assert status[0] == ns.OK, status
        assert status[1] == levels
        assert np.array_equal(got, want)
    # a link id out of range in flow 3: reported, nothing solved
    bad = plink.copy()
    bad[poff[3]] = len(cap)
    _, status = _noalloc(torch, ns, cap, poff, bad)
    assert status[0] == ns.E_INVALID and status[1] == 3
    # the shared scratch holds the last call's contents: a good call after
    # the failed one is still exact
    got, status = _noalloc(torch, ns, cap, poff, plink)
    assert status[0] == ns.OK and np.array_equal(got, want)


def test_noalloc_host_checks():
    torch, ns, pr = _gpu()
    with pytest.raises(ns.NetsimError) as ei:
        ns.netsim_solve_rates_noalloc(0, 1 << 17, 1, 1, 1, 1, 1, 1)
    assert ei.value.status == ns.E_LIMIT
    with pytest.raises(ns.NetsimError) as ei:
        ns.netsim_solve_rates_noalloc(0, 4, 1, 1, 0, 1, 1, 1)
    assert ei.value.status == ns.E_INVALID
