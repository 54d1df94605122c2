"""Seeded synthetic workloads: topology parameters plus communication
operations.  Input generation only: routing, collective decomposition and
simulation are done separately by each consumer."""

from .program import (GiB, MiB, AllToAll, Barrier, PathFlow, Program, Ring,
                      Scenario, Send, Topology, gbit)
from .configs import CONFIGS, DEFAULT_SEEDS, build

__all__ = ["GiB", "MiB", "AllToAll", "Barrier", "PathFlow", "Program", "Ring",
           "Scenario", "Send", "Topology", "gbit", "CONFIGS", "DEFAULT_SEEDS",
           "build"]
