"""MI355X flow-level network simulator (max-min fair bandwidth sharing).

The C ABI is ``include/netsim.h``; ``netsim`` is its ctypes binding and
``program`` loads workload descriptions into a handle.  Build the library
with ``python -m paper_2505_01616_amd.build``.
"""

__all__ = ["netsim", "program"]
