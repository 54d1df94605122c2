"""Oracle for the flow-level max-min network simulator.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py`` import, call or load anything in
this package.  The simulator library (``paper_2505_01616_amd``) never
does, and the two share no code: this package builds its own links,
routes and flows from the seeded workload description and runs its own
simulation.

Contents:
  topology.py       links, capacities, ECMP routes (numpy)
  flows.py          communication operations -> flows (numpy)
  netsim_oracle.c   fp64 single-threaded event loop + progressive filling
  sim.py            ctypes entry points of the C oracle
  plain.py          pure-Python exact (Fraction) and fp64 forms, and the
                    brute-force max-min check, for small cases
Every function in this package is pinned by tests under ``tests/``
(closed forms, textbook examples, brute force, invariants, metamorphic
relations); none is "parity unpinned".
"""
