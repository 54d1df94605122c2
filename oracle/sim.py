"""Python entry points of the fp64 C oracle.

TEST INFRASTRUCTURE (see ``oracle/__init__.py``).
"""

from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

from .build import LIB, SRC, build
from .flows import FlowSet, expand

_lib = None

_P = ctypes.c_void_p
_I64 = ctypes.c_int64


def _load():
    global _lib
    if _lib is None:
        # NETSIM_ORACLE_LIB: another build of netsim_oracle.c (the sanitizer
        # build of tests/test_native_checks.py)
        path = os.environ.get("NETSIM_ORACLE_LIB")
        if not path:
            path = LIB
            if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
                build()
        lib = ctypes.CDLL(path)
        lib.oracle_run.restype = ctypes.c_int
        lib.oracle_run.argtypes = [_I64, _P, _I64, _P, _P, _P, _P, _P, _P, _P, _I64,
                                   ctypes.c_double, _I64, _P, _P, _P, _P]
        lib.oracle_solve.restype = ctypes.c_int
        lib.oracle_solve.argtypes = [_I64, _P, _I64, _P, _P, _I64, _P, _P, _P]
        _lib = lib
    return _lib


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


@dataclass
class OracleResult:
    finish: np.ndarray
    events: int
    solves: int
    iterations: int
    flows_swept: int
    incidences_swept: int
    snap_rates: np.ndarray = None
    snap_time: float = None
    complete: bool = True

    @property
    def makespan(self) -> float:
        return float(np.max(self.finish)) if len(self.finish) else 0.0


class OracleError(RuntimeError):
    pass


def run_flowset(fs: FlowSet, max_events: int = 0, snap_solve: int = 0,
                until: float = float("inf")) -> OracleResult:
    """Runs the fp64 oracle on one scenario.  ``max_events`` > 0 stops after
    that many events; ``until`` stops before the first event later than it.
    Either way ``complete`` is False and unfinished flows have finish NaN."""
    lib = _load()
    F = fs.F
    cap = np.ascontiguousarray(fs.cap, np.float64)
    nb = np.ascontiguousarray(fs.nbytes, np.float64)
    st = np.ascontiguousarray(fs.start, np.float64)
    poff = np.ascontiguousarray(fs.path_off, np.int64)
    plink = np.ascontiguousarray(fs.path_link, np.int32)
    doff = np.ascontiguousarray(fs.dep_off, np.int64)
    dids = np.ascontiguousarray(fs.dep_ids, np.int64)
    if len(plink) == 0:
        plink = np.zeros(1, np.int32)
    if len(dids) == 0:
        dids = np.zeros(1, np.int64)
    finish = np.full(max(F, 1), np.nan)
    counts = np.zeros(5, np.int64)
    snap = np.zeros(max(F, 1)) if snap_solve else None
    stime = np.zeros(1)
    lat = (np.ascontiguousarray(fs.lat, np.float64)
           if getattr(fs, "lat", None) is not None and F > 0 else None)
    rc = lib.oracle_run(fs.L, _ptr(cap), F, _ptr(nb), _ptr(st),
                        _ptr(lat) if lat is not None else None, _ptr(poff), _ptr(plink),
                        _ptr(doff), _ptr(dids), int(max_events), float(until),
                        int(snap_solve),
                        _ptr(snap) if snap is not None else None, _ptr(stime),
                        _ptr(finish), _ptr(counts))
    if rc not in (0, 1) and not (rc == -5 and max_events > 0):
        raise OracleError(f"oracle_run failed with status {rc}")
    return OracleResult(finish[:F].copy(), *[int(c) for c in counts],
                        snap_rates=None if snap is None else snap[:F].copy(),
                        snap_time=float(stime[0]) if snap_solve else None,
                        complete=(rc == 0))


def run_scenario(scenario, **kw) -> OracleResult:
    return run_flowset(expand(scenario), **kw)


def run_program(program, **kw):
    return [run_scenario(sc, **kw) for sc in program.scenarios]


def solve_rates(cap, path_off, path_link, active) -> np.ndarray:
    """Rates of one max-min solve over the flows listed in ``active``."""
    lib = _load()
    cap = np.ascontiguousarray(cap, np.float64)
    poff = np.ascontiguousarray(path_off, np.int64)
    plink = np.ascontiguousarray(path_link, np.int32)
    act = np.ascontiguousarray(active, np.int64)
    out = np.zeros(max(len(act), 1))
    it = np.zeros(1, np.int64)
    rc = lib.oracle_solve(len(cap), _ptr(cap), len(poff) - 1, _ptr(poff),
                          _ptr(plink if len(plink) else np.zeros(1, np.int32)),
                          len(act), _ptr(act), _ptr(out), _ptr(it))
    if rc != 0:
        raise OracleError(f"oracle_solve failed with status {rc}")
    return out[: len(act)].copy()
