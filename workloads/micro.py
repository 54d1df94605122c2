"""Small seeded cases on explicit topologies (random links and paths)."""

from __future__ import annotations

import numpy as np

from .program import Barrier, PathFlow, Program, Scenario, Topology
from .rng import Stream


class _Draws:
    """Successive uniform draws of one stream, fetched in blocks."""

    def __init__(self, stream: Stream):
        self.st = stream
        self.i = 0
        self.buf = stream.u01(256)

    def __call__(self) -> float:
        if self.i >= len(self.buf):
            self.buf = np.concatenate([self.buf, self.st.u01(256, len(self.buf))])
        self.i += 1
        return float(self.buf[self.i - 1])


def random_static(seed: int, max_links: int = 8, max_flows: int = 10,
                  integer_caps: bool = True) -> Program:
    """All flows released at t=0, no dependencies (a single rate solve)."""
    nxt = _Draws(Stream(seed, "micro-static"))

    L = 1 + int(nxt() * max_links)
    F = 1 + int(nxt() * max_flows)
    if integer_caps:
        caps = np.array([1 + int(nxt() * 9) for _ in range(L)], dtype=np.float64)
    else:
        caps = np.array([0.5 + 9.5 * nxt() for _ in range(L)], dtype=np.float64)
    sc = Scenario(Topology(kind="explicit", capacities=caps))
    for _ in range(F):
        path = [l for l in range(L) if nxt() < 0.4]
        if not path:
            path = [min(int(nxt() * L), L - 1)]
        sc.add(PathFlow(path, float(1 + int(nxt() * 100))))
    return Program(f"micro-static-{seed}", [sc])


def random_dynamic(seed: int, max_links: int = 6, max_flows: int = 12,
                   barriers: bool = True, integer_caps: bool = True) -> Program:
    """Random releases and dependencies on a random explicit topology."""
    nxt = _Draws(Stream(seed, "micro-dynamic"))

    L = 1 + int(nxt() * max_links)
    F = 2 + int(nxt() * (max_flows - 1))
    if integer_caps:
        caps = np.array([1 + int(nxt() * 9) for _ in range(L)], dtype=np.float64)
    else:
        caps = np.array([0.5 + 9.5 * nxt() for _ in range(L)], dtype=np.float64)
    sc = Scenario(Topology(kind="explicit", capacities=caps))
    for i in range(F):
        after = tuple(j for j in range(i) if nxt() < 0.2)
        lag = float(int(nxt() * 8)) if nxt() < 0.6 else 0.0
        if barriers and nxt() < 0.1:
            sc.add(Barrier(lag=lag, after=after))
            continue
        path = [l for l in range(L) if nxt() < 0.45]
        if not path:
            path = [min(int(nxt() * L), L - 1)]
        sc.add(PathFlow(path, float(1 + int(nxt() * 40)), lag=lag, after=after))
    return Program(f"micro-dynamic-{seed}", [sc])
