"""Writes the stored oracle values used by the full-size GPU parity tests.

Calls only the oracle (``oracle/``) and the seeded workload generator.  Run
from the repository root:
  python tests/golden/make_golden.py [c3] [c5] [c4part] [c3full] [c4blocks]

c5_makespans.json   per-scenario makespan of all 256 C5 scenarios (fp64 oracle)
c4_part_summary.json  one part of the 4096-GPU expert-parallel all-to-all at
                    full width (the eight expert groups of one 64-server block,
                    one dispatch phase, ~32k flows): makespan, event and solve
                    counts and a seeded sample of per-flow finish times of the
                    complete run
c3_summary.json     C3 (full size): makespan, a seeded sample of per-flow
                    finish times, and the oracle's own spread under changes
                    of every capacity by k ulps, k in -5..-1 and 1..6 (C3 is
                    ill-conditioned in fp64; eleven perturbations, run in
                    parallel processes)
c3_finish.npz       C3 (full size): the complete per-flow finish times of the
                    unperturbed oracle run (f64store format), with
c3_full.json        its event, solve and progressive-filling iteration counts
c4_blocks_finish.npz  the 4096-GPU all-to-all at full size (four phases):
                    complete per-flow finish times of each of its eight
                    independent 64-server blocks (flows b*129048 ..
                    (b+1)*129048-1 of the full workload; a block shares no
                    link and no dependency with another), each run by the
                    oracle on its own clock, in parallel processes
c4_blocks.json      per block: event, solve and iteration counts, makespan
"""

from __future__ import annotations

import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

from oracle import flows as oflows  # noqa: E402
from oracle import sim as osim  # noqa: E402
from workloads import configs  # noqa: E402

sys.path.insert(0, HERE)
import f64store  # noqa: E402


def c5():
    prog = configs.c5(5)
    out = []
    t0 = time.time()
    for s, sc in enumerate(prog.scenarios):
        r = osim.run_scenario(sc)
        out.append({"scenario": s, "makespan": r.makespan, "events": r.events,
                    "solves": r.solves, "flows": int(len(r.finish))})
    with open(os.path.join(HERE, "c5_makespans.json"), "w") as fh:
        json.dump({"config": "c5 seed 5 (256 scenarios)", "writer": "tests/golden/make_golden.py",
                   "scenarios": out}, fh, indent=0)
    print(f"c5: {len(out)} scenarios in {time.time() - t0:.0f} s", flush=True)


def _perturbed(fs, k):
    cap = fs.cap.copy()
    for _ in range(abs(k)):
        cap = np.nextafter(cap, np.inf if k > 0 else 0.0)
    return oflows.FlowSet(cap, fs.src, fs.dst, fs.nbytes, fs.start, fs.path_off, fs.path_link,
                          fs.dep_off, fs.dep_ids)


C3_ULPS = (-5, -4, -3, -2, -1, 1, 2, 3, 4, 5, 6)


def _c3_run(k):
    fs = oflows.expand(configs.c3(3).scenarios[0])
    return osim.run_flowset(_perturbed(fs, k) if k else fs)


def c3():
    from multiprocessing import Pool
    t0 = time.time()
    fs = oflows.expand(configs.c3(3).scenarios[0])
    with Pool(min(6, len(C3_ULPS) + 1)) as pool:
        res = pool.map(_c3_run, (0,) + C3_ULPS)
    ref = res[0]
    runs = [r.finish for r in res[1:]]
    dev = np.max([np.abs(r - ref.finish) / ref.finish for r in runs], axis=0)
    order = np.argsort(ref.finish)
    bad = order[dev[order] > 1e-9]
    horizon = float(ref.finish[bad[0]]) if len(bad) else float("inf")
    rng = np.random.default_rng(33)
    sample = np.sort(rng.choice(fs.F, size=4000, replace=False))
    early = np.nonzero(ref.finish < horizon)[0]
    early_sample = np.sort(rng.choice(early, size=min(2000, len(early)), replace=False))
    data = {
        "config": "c3 seed 3 (full size)", "writer": "tests/golden/make_golden.py",
        "ulp_perturbations": list(C3_ULPS),
        "flows": int(fs.F), "events": ref.events, "solves": ref.solves,
        "makespan": ref.makespan,
        "ulp_spread_makespan": max(abs(float(np.max(r)) - ref.makespan) for r in runs) / ref.makespan,
        "ulp_spread_q99": float(np.quantile(dev, 0.99)),
        "horizon": horizon,
        "sample_ids": sample.tolist(), "sample_finish": ref.finish[sample].tolist(),
        "early_ids": early_sample.tolist(), "early_finish": ref.finish[early_sample].tolist(),
    }
    with open(os.path.join(HERE, "c3_summary.json"), "w") as fh:
        json.dump(data, fh)
    print(f"c3: {time.time() - t0:.0f} s, horizon {horizon:.4g}", flush=True)


def c4part(phases=1):
    t0 = time.time()
    prog = configs.c4(4, blocks=1, locals_=8, phases=phases)
    fs = oflows.expand(prog.scenarios[0])
    ref = osim.run_flowset(fs)
    rng = np.random.default_rng(44)
    sample = np.sort(rng.choice(fs.F, size=3000, replace=False))
    data = {
        "config": f"c4 seed 4, blocks=1, locals_=8, phases={phases} (one 64-server block, 8 expert groups)",
        "writer": "tests/golden/make_golden.py",
        "flows": int(fs.F), "events": ref.events, "solves": ref.solves, "makespan": ref.makespan,
        "finished": int(np.isfinite(ref.finish).sum()),
        "sample_ids": sample.tolist(), "sample_finish": ref.finish[sample].tolist(),
    }
    name = "c4_part_summary.json" if phases == 1 else f"c4_part{phases}_summary.json"
    with open(os.path.join(HERE, name), "w") as fh:
        json.dump(data, fh)
    print(f"c4part phases={phases}: {time.time() - t0:.0f} s, {ref.events} events", flush=True)


def c3full():
    t0 = time.time()
    fs = oflows.expand(configs.c3(3).scenarios[0])
    ref = osim.run_flowset(fs)
    assert ref.complete and np.all(np.isfinite(ref.finish))
    f64store.save(os.path.join(HERE, "c3_finish.npz"), finish=ref.finish)
    with open(os.path.join(HERE, "c3_full.json"), "w") as fh:
        json.dump({"config": "c3 seed 3 (full size)", "writer": "tests/golden/make_golden.py",
                   "flows": int(fs.F), "events": ref.events, "solves": ref.solves,
                   "iterations": ref.iterations, "flows_swept": ref.flows_swept,
                   "incidences_swept": ref.incidences_swept, "makespan": ref.makespan,
                   "oracle_seconds": time.time() - t0}, fh, indent=1)
    print(f"c3full: {time.time() - t0:.0f} s, {ref.events} events, "
          f"{ref.iterations} iterations", flush=True)


C4_BLOCK_FLOWS = 129048


def c4_block_flowset(fs, b):
    """Flows b*129048 .. (b+1)*129048-1 of the full 4096-GPU all-to-all as a
    flow set of their own (dependency ids shifted; links unchanged)."""
    f0, f1 = b * C4_BLOCK_FLOWS, (b + 1) * C4_BLOCK_FLOWS
    p0, p1 = fs.path_off[f0], fs.path_off[f1]
    d0, d1 = fs.dep_off[f0], fs.dep_off[f1]
    dids = fs.dep_ids[d0:d1] - f0
    assert dids.size == 0 or (dids.min() >= 0 and dids.max() < f1 - f0)
    return oflows.FlowSet(fs.cap, fs.src[f0:f1], fs.dst[f0:f1], fs.nbytes[f0:f1],
                          fs.start[f0:f1], fs.path_off[f0:f1 + 1] - p0,
                          fs.path_link[p0:p1], fs.dep_off[f0:f1 + 1] - d0, dids)


def _c4_block_run(b):
    t0 = time.time()
    fs = oflows.expand(configs.c4(4).scenarios[0])
    assert fs.F == 8 * C4_BLOCK_FLOWS
    sub = c4_block_flowset(fs, b)
    del fs
    r = osim.run_flowset(sub)
    assert r.complete and np.all(np.isfinite(r.finish))
    print(f"c4 block {b}: {time.time() - t0:.0f} s, {r.events} events", flush=True)
    return b, r.finish, {"block": b, "events": r.events, "solves": r.solves,
                         "iterations": r.iterations, "makespan": r.makespan,
                         "oracle_seconds": time.time() - t0}


def c4blocks():
    from multiprocessing import Pool
    t0 = time.time()
    with Pool(8) as pool:
        res = sorted(pool.map(_c4_block_run, range(8)))
    f64store.save(os.path.join(HERE, "c4_blocks_finish.npz"),
                  **{f"block{b}": fin for b, fin, _ in res})
    with open(os.path.join(HERE, "c4_blocks.json"), "w") as fh:
        json.dump({"config": "c4 seed 4 (full size, four phases)",
                   "writer": "tests/golden/make_golden.py",
                   "block_flows": C4_BLOCK_FLOWS, "blocks": [m for _, _, m in res]}, fh, indent=1)
    print(f"c4blocks: {time.time() - t0:.0f} s", flush=True)


if __name__ == "__main__":
    which = sys.argv[1:] or ["c5", "c3", "c4part", "c3full", "c4blocks"]
    if "c5" in which:
        c5()
    if "c3" in which:
        c3()
    if "c4part" in which:
        c4part()
    if "c3full" in which:
        c3full()
    if "c4blocks" in which:
        c4blocks()
