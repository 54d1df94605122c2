"""Benchmark: max-min rate solves/s and events/s of the flow-level simulator
on the 4096-GPU expert-parallel all-to-all workload (C4), on one MI355X.

A step is one event of the simulator's event loop: find the next
completion or release, settle completions and releases, and re-solve the
max-min rates of all active flows.  The timed region is one device-resident
run of exactly K events from t = 0 (one kernel launch); W warm-up events
run first in a separate launch.  Inputs (flows, routes, capacities) are
resident in HBM before timing starts.

Prints one JSON line.  Also reports the roofline of the event-loop kernel
(algorithmic bytes per launch / launch duration, against 8 TB/s) and the
CPU oracle's rate on a bounded sample of the same workload.
"""

from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0

# Algorithmic bytes ("Roofline"): what each unit of work must
# move at least once per visit.
BYTES_PER_FLOW_ROUND = 28      # list entry 4 + path offsets 8 + min-share write 8 + read 8
BYTES_PER_INCIDENCE_ROUND = 21  # link id 4+4 + residual capacity 8 + count 4 + flag 1
BYTES_PER_ACTIVE_EVENT = 48    # rem, rate read twice (32) + rem write 8 + list in/out 8
BYTES_PER_PENDING_EVENT = 28   # list in 4 + release time 8, twice, + list out 4


def algorithmic_bytes(st: dict) -> float:
    return (BYTES_PER_FLOW_ROUND * st["flows_swept"] + BYTES_PER_INCIDENCE_ROUND * st["incidences_swept"]
            + BYTES_PER_ACTIVE_EVENT * st["active_swept"] + BYTES_PER_PENDING_EVENT * st["pending_swept"])


# The first 64 events of C4 are the arrivals of the 64 groups (small active
# sets); from then on every solve covers all ~258k flows of a phase.  Both the
# GPU and the oracle are also timed on events 65..128 alone (by differencing
# two runs) so that their rates are compared on the same steady-state window.
STEADY = (64, 128)


def cpu_baseline():
    """The fp64 oracle (single thread, as it stands) on events 65..128 of C4."""
    from oracle import flows as oflows
    from oracle import sim as osim
    from workloads import configs
    fs = oflows.expand(configs.c4(4).scenarios[0])
    t = []
    for e in STEADY:
        t0 = time.perf_counter()
        r = osim.run_flowset(fs, max_events=e)
        t.append((time.perf_counter() - t0, r.solves, r.events))
    dt = t[1][0] - t[0][0]
    return {"value": (t[1][1] - t[0][1]) / dt, "unit": "solves/s", "cores": 1, "kind": "oracle",
            "events_per_s": (t[1][2] - t[0][2]) / dt, "seconds": t[0][0] + t[1][0],
            "sample": f"events {STEADY[0] + 1}..{STEADY[1]} of the 4096-GPU all-to-all workload "
                      f"(every group active, ~258k flows per solve), timed as the difference "
                      f"of runs to {STEADY[0]} and {STEADY[1]} events; fp64 oracle, one thread"}


def traffic_from_profile(steps: int, exec_: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if
    it was taken on the current kernel source with the same launch."""
    import hashlib
    try:
        with open(os.path.join(ROOT, "profiles", "netsim_grid_kernel_c4_traffic.json")) as fh:
            prof = json.load(fh)
        with open(os.path.join(ROOT, "paper_2505_01616_amd", "csrc", "kernels.hip"), "rb") as fh:
            sha = hashlib.sha256(fh.read()).hexdigest()[:16]
    except OSError:
        return None
    if prof.get("kernels_hip_sha256_16") != sha or prof.get("steps") != steps or exec_ != "grid":
        return None
    return prof["traffic_bytes"]


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2000)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--exec", choices=["grid", "block", "auto"], default="grid")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run only a 1 GiB device copy (for scaling HBM counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build runs the whole simulated cluster "
              "on a single MI355X (no multi-GPU path); use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    if args.copy_calibration:
        a = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_each_way": 1 << 30, "launches": 3}))
        return

    from paper_2505_01616_amd import netsim as ns
    from paper_2505_01616_amd import program as prog
    from workloads import configs

    stream = torch.cuda.current_stream()
    program = configs.c4(4)
    ex = {"grid": ns.EXEC_GRID, "block": ns.EXEC_BLOCK, "auto": ns.EXEC_AUTO}[args.exec]
    ld = prog.load_program(program, ns.make_options(exec=ex))
    h = ld.handle
    try:
        nflows, nnz, ndeps = ns.netsim_counts(h)
        # warm-up (also uploads the static data once)
        ns.netsim_set_limits(h, max_events=max(args.warmup, 1))
        ns.netsim_run(h, stream)
        # timed: exactly K events, one launch
        ns.netsim_set_limits(h, max_events=args.steps)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ns.netsim_run(h, stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        st = ns.netsim_get_stats(h)
        # steady-state window (same events as the CPU baseline)
        steady_dev = []
        for e in STEADY:
            ns.netsim_set_limits(h, max_events=e)
            ns.netsim_run(h, stream)
            s2 = ns.netsim_get_stats(h)
            steady_dev.append((s2["device_seconds"], s2["solves"]))
    finally:
        ld.close()
    gpu_steady = (steady_dev[1][1] - steady_dev[0][1]) / (steady_dev[1][0] - steady_dev[0][0])
    dev = st["device_seconds"]
    assert st["events"] == args.steps, st
    solves_per_s = st["solves"] / dev
    events_per_s = st["events"] / dev
    abytes = algorithmic_bytes(st)
    achieved = abytes / dev / 1e9
    traffic = traffic_from_profile(args.steps, args.exec)
    line = {
        "metric": "max-min rate solves/sec + events/sec (4096-GPU all-to-all); achieved HBM GB/s",
        "value": solves_per_s,
        "unit": "solves/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": dev * 1e3 / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {"workload": "c4: 4096 GPUs, 3-tier fat-tree 2:1 at the core, 64 EP groups x 64 "
                               "ranks, 4 all-to-all phases, Zipf(1.2) bytes mean 4 MiB, seed 4",
                   "flows": nflows, "incidences": nnz, "exec": args.exec},
        "events_per_s": events_per_s,
        "steady_state_solves_per_s": gpu_steady,
        "solves": st["solves"],
        "rounds_per_solve": st["rounds"] / max(st["solves"], 1),
        "wall_s_incl_state_reset": wall,
        "sim_time_s": st["sim_time"],
        "phase_seconds": dict(zip(["next_event", "settle", "solve_setup", "sweep_b", "wait_b",
                                   "sweep_c", "wait_c"], [round(x, 6) for x in st["phase_seconds"][:7]])),
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS, "traffic": traffic,
                     "kernel": "netsim_grid_kernel" if args.exec == "grid" else "netsim_block_kernel",
                     "algorithmic_bytes": abytes, "launch_seconds": dev},
    }
    if not args.no_cpu_baseline and int(os.environ.get("RANK", "0")) == 0:
        line["cpu_baseline"] = cpu_baseline()
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
