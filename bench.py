"""Benchmark: max-min rate solves/s and events/s of the flow-level simulator
on the 4096-GPU expert-parallel all-to-all workload (C4), on one MI355X.

A step is one complete simulation of the workload: every flow of the four
back-to-back all-to-all phases from release to completion (about 0.9 M
events, each ending in a max-min rate solve).  The simulator splits the
workload into its independent parts (the eight groups of expert-parallel
ranks that share fabric links) and runs each with its own clock; by default
(AUTO) each part gets the workgroups of one XCD: a leader running its event
loop and 15 helpers solving its large re-solves (--exec block: one workgroup
per part).  Events and solves are counted per part.  Each step is one kernel
launch, timed with HIP events on the launch stream; W warm-up steps run
first.  Inputs (flows, routes, capacities) are resident in HBM
before timing starts; the per-run state reset is outside the kernel time.

Prints one JSON line, with the roofline of the event-loop kernel
(algorithmic bytes per launch / launch duration, against 8 TB/s), the
cold-cache measurement of the wide exact solve's sweeps at the shape of one
all-to-all phase (roofline_sweep), and the CPU oracle's rate on a bounded
sample of the same workload (one independent block, on its own clock).
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

# Algorithmic bytes of the max-min path: what progressive filling must move
# per unit of work, whatever the layout (link state in shared memory counts
# like link state in HBM).
#   per round:   4 B link id + 8 B gathered share per unfrozen incidence;
#                8 B path offsets + 1 B frozen flag per unfrozen flow;
#                36 B per link whose share the round computes (R, n, k read;
#                R, n, s written);
#   per freeze:  9 B (rate + flag written) per flow frozen;
#   per event:   24 B (remaining bytes, rate, predicted completion) per active
#                flow; 12 B (id + release time) per pending flow looked at.
B_INCIDENCE_ROUND = 12
B_FLOW_ROUND = 9
B_LINK_ROUND = 36
B_FROZEN = 9
B_ACTIVE_EVENT = 24
B_PENDING_EVENT = 12


def algorithmic_bytes(st: dict, frozen: int) -> float:
    return (B_INCIDENCE_ROUND * st["incidences_swept"] + B_FLOW_ROUND * st["flows_swept"]
            + B_LINK_ROUND * st["links_swept"] + B_FROZEN * frozen
            + B_ACTIVE_EVENT * st["active_swept"] + B_PENDING_EVENT * st["pending_swept"])


# The oracle as it stands, on a bounded sample of the same work: one of the
# eight independent 64-server blocks of the workload (the unit one part of
# the GPU simulation runs, on its own clock as the part does), events 65 ..
# 65 + SAMPLE_EVENTS of that block (the first 64 events are the arrivals of
# its groups), timed as the difference of runs to 64 and to 64 +
# SAMPLE_EVENTS events (about 15 s on one core).
SAMPLE_EVENTS = 1000
C4_BLOCK_FLOWS = 129048


def cpu_baseline(total_events: int):
    """The fp64 oracle (single thread) on events 65..1064 of one C4 block."""
    import platform
    from oracle import flows as oflows
    from oracle import sim as osim
    from workloads import configs
    fs = oflows.expand(configs.c4(4, blocks=1).scenarios[0])
    assert fs.F == C4_BLOCK_FLOWS
    t = []
    for e in (64, 64 + SAMPLE_EVENTS):
        t0 = time.perf_counter()
        r = osim.run_flowset(fs, max_events=e)
        t.append((time.perf_counter() - t0, r.solves, r.events))
    dt = t[1][0] - t[0][0]
    solves_per_s = (t[1][1] - t[0][1]) / dt
    events_per_s = (t[1][2] - t[0][2]) / dt
    cpu = platform.processor() or ""
    try:
        with open("/proc/cpuinfo") as fh:
            for ln in fh:
                if ln.startswith("model name"):
                    cpu = ln.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"value": solves_per_s, "unit": "solves/s", "cores": 1, "kind": "oracle",
            "events_per_s": events_per_s, "seconds": t[0][0] + t[1][0], "cpu_model": cpu,
            "host_threads": os.cpu_count(),
            "projected_complete_s_at_sample_rate": total_events / events_per_s,
            "sample": f"events 65..{64 + SAMPLE_EVENTS} of one 64-server block of the 4096-GPU "
                      f"all-to-all (129,048 flows, the unit one GPU part simulates, on its own "
                      f"clock), timed as the difference of runs to 64 and {64 + SAMPLE_EVENTS} "
                      f"events; fp64 oracle, one thread; solves and events are per part as on "
                      f"the GPU; the sample is the densest stretch of the run (the first "
                      f"phase, every group active at full width), so the projection of the "
                      f"workload's {total_events} part events at its rate is an upper bound"}


def sweep_bench(ns, prog, stream, reps=20, flush=1 << 30):
    """Cold-cache timing of the two sweeps of a wide exact solve at the shape
    of the 4096-GPU workload at its start: the full workload loaded (one part
    in exact mode: 1,032,384 flows, 5,144,576 incidences, 20,480 links), every
    flow of the first all-to-all phase active (258,048 flows, 1,286,144
    incidences).  The per-link count sweeps the part's whole link-major
    incidence (flows of later phases count as inactive), the freezing sweep
    the 258,048 unfrozen flows of the first level.  Before each sweep a 1 GiB
    streaming write evicts the L2s and the Infinity Cache.  Then the complete
    wide solve of that set (all its progressive-filling levels)."""
    import numpy as np
    from workloads import configs
    program = configs.c4(4)
    ld = prog.load_program(program, ns.make_options(exact=1))
    h = ld.handle
    try:
        ex = ns.netsim_export_flows(h)
        act = np.nonzero((ex["nbytes"] > 0) & (np.diff(ex["dep_off"]) == 0))[0]
        nnz_all = int(len(ex["path_link"]))
        nnz = int(np.diff(ex["path_off"])[act].sum())
        links = int(len(np.unique(ex["path_link"])))
        t = ns.netsim_bench_sweeps(h, 0, act, reps, flush, stream)
        ns.netsim_solve_once(h, 0, act)
        st = ns.netsim_get_stats(h)
    finally:
        ld.close()
    F = len(act)
    # freezing sweep of the first level (every flow unfrozen): the per-round
    # terms of the byte model
    frz_bytes = B_INCIDENCE_ROUND * nnz + B_FLOW_ROUND * F
    # per-link count over the whole link-major incidence: flow id 4 B + its
    # flag 1 B per entry; per link the offsets 4 B and the count 4 B
    cnt_bytes = 5 * nnz_all + 8 * links
    # work-efficient lower bound of one solve: every incidence and flow
    # touched a constant number of times
    we_bytes = 16 * nnz + 24 * F

    def leg(kernel, ab, ev, kern):
        e, k = float(np.median(ev)) * 1e-3, float(np.median(kern)) * 1e-3
        return {"kernel": kernel, "algorithmic_bytes": ab,
                "kernel_s": k, "achieved": ab / k / 1e9, "frac": ab / k / 1e9 / HBM_PEAK_GBPS,
                "event_s": e, "achieved_incl_dispatch": ab / e / 1e9, "unit": "GB/s",
                "kernel_s_min": float(np.min(kern)) * 1e-3}

    sol = st["device_seconds"]
    return {
        "shape": {"flows_active": F, "incidences_active": nnz, "incidences_part": nnz_all,
                  "links": links},
        "flush_bytes": flush, "reps": reps,
        "timing": "kernel_s: first workgroup start to last workgroup end on the device wall "
                  "clock (median over reps); event_s: HIP events around the launch",
        "freeze_sweep": leg("exact_freeze_kernel", frz_bytes, t["freeze_ms"], t["freeze_kernel_ms"]),
        "link_count": leg("exact_count_kernel", cnt_bytes, t["count_ms"], t["count_kernel_ms"]),
        "full_solve": {"device_s": sol, "levels": st["rounds"], "flows_swept": st["flows_swept"],
                       "incidences_swept": st["incidences_swept"], "links_swept": st["links_swept"],
                       "algorithmic_bytes": B_INCIDENCE_ROUND * st["incidences_swept"]
                       + B_FLOW_ROUND * st["flows_swept"] + B_LINK_ROUND * st["links_swept"]
                       + B_FROZEN * F,
                       "work_efficient_bytes": we_bytes,
                       "work_efficient_GBps": we_bytes / sol / 1e9},
    }


def traffic_from_profile(kernel: str, steps: int):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if
    it was taken on the current kernel source for the same kernel."""
    import hashlib
    try:
        with open(os.path.join(ROOT, "profiles", f"{kernel}_c4_traffic.json")) as fh:
            prof = json.load(fh)
        with open(os.path.join(ROOT, "paper_2505_01616_amd", "csrc", "kernels.hip"), "rb") as fh:
            sha = hashlib.sha256(fh.read()).hexdigest()[:16]
    except OSError:
        return None
    if prof.get("kernels_hip_sha256_16") != sha or prof.get("kernel") != kernel:
        return None
    return prof["traffic_bytes_per_launch"]


def sweep_traffic_from_profile():
    """HBM bytes of the count and freezing sweeps (cold repetitions) from the
    committed rocprofv3 counter summary, if taken on the current sweep.hip."""
    import hashlib
    try:
        with open(os.path.join(ROOT, "profiles", "exact_sweeps_c4_traffic.json")) as fh:
            prof = json.load(fh)
        with open(os.path.join(ROOT, "paper_2505_01616_amd", "csrc", "sweep.hip"), "rb") as fh:
            sha = hashlib.sha256(fh.read()).hexdigest()[:16]
    except OSError:
        return None
    if prof.get("sweep_hip_sha256_16") != sha:
        return None
    return prof["freeze_traffic_bytes"] + prof["count_traffic_bytes"]


def rollback_bench(ns, prog, program, stream, pieces=10, history_mb=72000):
    """Time rollback on C4: the complete simulation as one launch; the same
    simulation advanced in `pieces` checkpointed launches, with checkpoints
    only (AUTO's cluster layout, and the block layout) and also keeping the
    rollback history (`history_mb` MiB: every undo record of the complete
    run fits; the block layout, as the cluster kernel keeps none); then a
    start moved for a flow that finished at about 55% of the horizon.  With
    checkpoints only its part goes back to the last checkpoint before the
    flow's release, with the history to its last event before it; either
    way the part is re-simulated to the end while the other parts stay
    finished, and both give the same finish times bit for bit."""
    import numpy as np
    out = {"metric": "time rollback on the 4096-GPU all-to-all workload", "pieces": pieces}
    ld = prog.load_program(program)
    try:
        ns.netsim_run(ld.handle, stream)
        out["one_run_device_s"] = ns.netsim_get_stats(ld.handle)["device_seconds"]
        ref = ns.netsim_get_finish(ld.handle)
    finally:
        ld.close()
    T = float(np.nanmax(ref))
    results = {}
    legs = (("checkpoints", 0, ns.EXEC_AUTO), ("checkpoints_block", 0, ns.EXEC_BLOCK),
            ("history", history_mb, ns.EXEC_AUTO))
    for name, mb, ex in legs:
        ld = prog.load_program(program, ns.make_options(history_mb=mb, exec=ex))
        h = ld.handle
        r = {"history_mb": mb}
        try:
            dev, wall = 0.0, time.perf_counter()
            for k in range(1, pieces + 1):
                ns.netsim_advance(h, until=T * k / pieces if k < pieces else math.inf, stream=stream)
                dev += ns.netsim_get_stats(h)["device_seconds"]
            print(f"{name}: {pieces} advances done", file=sys.stderr, flush=True)
            r["pieces_device_s"] = dev
            r["pieces_wall_s_incl_checkpoints"] = time.perf_counter() - wall
            r["pieces_equal_one_run_bitwise"] = bool(np.array_equal(ns.netsim_get_finish(h), ref))
            r["checkpoints"] = ns.netsim_num_checkpoints(h)
            ex = ns.netsim_export_flows(h)
            cand = np.nonzero((ex["nbytes"] > 0) & (ref > 0.55 * T) & (ref < 0.6 * T))[0]
            x = int(cand[len(cand) // 2])
            t0 = time.perf_counter()
            ns.netsim_update_start(h, x, float(ex["start"][x]) + 20e-6)
            r["rollback_update_wall_s"] = time.perf_counter() - t0
            ns.netsim_advance(h, stream=stream)
            st = ns.netsim_get_stats(h)
            r["layout"] = {ns.EXEC_GRID: "grid", ns.EXEC_BLOCK: "block",
                           ns.EXEC_CLUSTER: "cluster"}.get(st["layout"], st["layout"])
            r["resimulate_device_s"] = st["device_seconds"]
            r["resimulated_events"] = st["launch_events"]
            got = ns.netsim_get_finish(h)
            r["moved_flows"] = int(np.sum(got != ref))
            results[name] = (r, got)
            print(f"{name}: rollback and re-simulation done", file=sys.stderr, flush=True)
        finally:
            ld.close()
        out[name] = r
    out["history_equals_checkpoints_bitwise"] = bool(
        np.array_equal(results["history"][1], results["checkpoints"][1]) and
        np.array_equal(results["history"][1], results["checkpoints_block"][1]))
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1, help="timed complete simulations")
    ap.add_argument("--warmup", type=int, default=1, help="untimed complete simulations first")
    ap.add_argument("--exec", choices=["grid", "block", "cluster", "auto"], default="auto")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-sweep", action="store_true",
                    help="skip the cold-cache sweep measurement of the wide exact solve")
    ap.add_argument("--sweep-only", action="store_true",
                    help="run only the cold-cache sweep measurement (one JSON line)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run only a 1 GiB device copy (for scaling HBM counters)")
    ap.add_argument("--rollback", action="store_true",
                    help="measure time rollback on the same workload instead (one JSON line)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the simulator runs the whole simulated cluster "
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
    if args.rollback:
        print(json.dumps(rollback_bench(ns, prog, program, stream)), flush=True)
        return
    if args.sweep_only:
        print(json.dumps(sweep_bench(ns, prog, stream)), flush=True)
        return
    ex = {"grid": ns.EXEC_GRID, "block": ns.EXEC_BLOCK, "cluster": ns.EXEC_CLUSTER,
          "auto": ns.EXEC_AUTO}[args.exec]
    ld = prog.load_program(program, ns.make_options(exec=ex))
    h = ld.handle
    keys = ("events", "solves", "rounds", "flows_swept", "incidences_swept", "active_swept",
            "pending_swept", "reselected", "wide_solves", "links_swept")
    tot = {k: 0 for k in keys}
    tot["device_seconds"] = 0.0
    phases = [0.0] * 8
    try:
        nflows, nnz, ndeps = ns.netsim_counts(h)
        for i in range(args.warmup):
            ns.netsim_run(h, stream)
            print(f"warm-up step {i + 1}/{args.warmup} done", file=sys.stderr, flush=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(args.steps):
            ns.netsim_run(h, stream)
            st = ns.netsim_get_stats(h)
            assert st["complete"] == 1, st
            for k in keys:
                tot[k] += st[k]
            tot["device_seconds"] += st["device_seconds"]
            phases = [a + b for a, b in zip(phases, st["phase_seconds"])]
            print(f"step {i + 1}/{args.steps}: {st['device_seconds']:.3f} s device, "
                  f"{st['solves']} solves", file=sys.stderr, flush=True)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        parts = st["parts"]
        sim_time = st["sim_time"]
        layout = st["layout"]
        assisted = st["assisted_solves"]
    finally:
        ld.close()
    dev = tot["device_seconds"]
    solves_per_s = tot["solves"] / dev
    events_per_s = tot["events"] / dev
    # every re-solved flow is frozen once in its solve
    abytes = algorithmic_bytes(tot, tot["reselected"])
    achieved = abytes / dev / 1e9
    kernel = {ns.EXEC_GRID: "netsim_grid_kernel", ns.EXEC_BLOCK: "netsim_block_kernel",
              ns.EXEC_CLUSTER: "netsim_cluster_kernel"}[layout]
    traffic = traffic_from_profile(kernel, args.steps)
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
                               "ranks, 4 all-to-all phases, Zipf(1.2) bytes mean 4 MiB, seed 4; "
                               "one step = the complete simulation",
                   "flows": nflows, "incidences": nnz, "exec": args.exec, "parts": parts,
                   "layout": kernel},
        "events_per_s": events_per_s,
        "events_per_step": tot["events"] / args.steps,
        "solves_per_step": tot["solves"] / args.steps,
        "rounds_per_solve": tot["rounds"] / max(tot["solves"], 1),
        "reselected_per_solve": tot["reselected"] / max(tot["solves"], 1),
        "wide_solves": tot["wide_solves"],
        "assisted_solves_per_step": assisted,
        "wall_s_incl_state_reset": wall,
        "sim_time_s": sim_time,
        "phase_seconds_summed_over_parts": dict(zip(
            ["next_event", "settle", "solve_setup", "sweep_b", "wait_b", "sweep_c", "wait_c",
             "reselect"], [round(x, 4) for x in phases])),
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS, "traffic": traffic, "kernel": kernel,
                     "algorithmic_bytes_per_launch": abytes / args.steps,
                     "launch_seconds": dev / args.steps,
                     "links_swept_per_launch": tot["links_swept"] / args.steps},
    }
    if not args.no_sweep:
        sw = sweep_bench(ns, prog, stream)
        fz, ct = sw["freeze_sweep"], sw["link_count"]
        ab = fz["algorithmic_bytes"] + ct["algorithmic_bytes"]
        ks = fz["kernel_s"] + ct["kernel_s"]
        line["roofline_sweep"] = {"bound": "hbm", "achieved": ab / ks / 1e9, "peak": HBM_PEAK_GBPS,
                                  "unit": "GB/s", "frac": ab / ks / 1e9 / HBM_PEAK_GBPS,
                                  "kernel": "exact_count_kernel + exact_freeze_kernel",
                                  "traffic": sweep_traffic_from_profile(), "detail": sw}
        print(f"sweeps: freeze {fz['kernel_s'] * 1e6:.1f} us ({fz['achieved']:.0f} GB/s), count "
              f"{ct['kernel_s'] * 1e6:.1f} us ({ct['achieved']:.0f} GB/s), full solve "
              f"{sw['full_solve']['device_s']:.3f} s", file=sys.stderr, flush=True)
    if not args.no_cpu_baseline and int(os.environ.get("RANK", "0")) == 0:
        line["cpu_baseline"] = cpu_baseline(tot["events"] // args.steps)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
