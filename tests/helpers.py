"""Small builders shared by the tests (no simulator arithmetic here)."""

from __future__ import annotations

import numpy as np

from workloads.program import Barrier, PathFlow, Program, Scenario, Topology


def explicit(caps, flows):
    """flows: list of dicts with keys path, nbytes, lag=0, after=() or
    {"barrier": True, ...}."""
    sc = Scenario(Topology(kind="explicit", capacities=np.asarray(caps, np.float64)))
    for f in flows:
        if f.get("barrier"):
            sc.add(Barrier(lag=f.get("lag", 0.0), after=tuple(f.get("after", ()))))
        else:
            sc.add(PathFlow(list(f["path"]), float(f["nbytes"]), lag=f.get("lag", 0.0),
                            after=tuple(f.get("after", ()))))
    return sc


def rel_err(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    den = np.maximum(np.abs(b), 1e-300)
    return np.max(np.abs(a - b) / den) if a.size else 0.0
