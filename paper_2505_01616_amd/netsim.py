"""Thin ctypes binding of libnetsim (include/netsim.h).

Argument marshalling only: every step of the simulation runs in the
library's HIP kernels.  Functions keep the C names; arrays are numpy arrays
(converted to the C types) and failures raise ``NetsimError`` with the
library's message.  The library must be built first
(``python -m paper_2505_01616_amd.build``); importing this module without
it raises an error instead of falling back to anything else.
"""

from __future__ import annotations

import ctypes
import math
import os
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
# NETSIM_LIB: another build of the library (the sanitizer build of the host
# code made by tests/test_native_checks.py)
LIB_PATH = os.environ.get("NETSIM_LIB") or os.path.join(HERE, "libnetsim.so")

OK, E_INVALID, E_NOMEM, E_DEVICE, E_STATE, E_LIMIT = 0, -1, -2, -3, -4, -5
TOPO_LEAF_SPINE, TOPO_RAIL, TOPO_FAT_TREE = 1, 2, 3
RING_ALLREDUCE, RING_REDUCE_SCATTER, RING_ALL_GATHER = 0, 1, 2
MODE_CHAINED, MODE_FLAT, MODE_AGGREGATED = 0, 1, 2
EXEC_AUTO, EXEC_GRID, EXEC_BLOCK, EXEC_CLUSTER, EXEC_EXACT = 0, 1, 2, 3, 4

STATUS_NAMES = {OK: "NETSIM_OK", E_INVALID: "NETSIM_E_INVALID", E_NOMEM: "NETSIM_E_NOMEM",
                E_DEVICE: "NETSIM_E_DEVICE", E_STATE: "NETSIM_E_STATE", E_LIMIT: "NETSIM_E_LIMIT"}


class netsim_options(ctypes.Structure):
    _fields_ = [("device", ctypes.c_int32), ("exec", ctypes.c_int32),
                ("max_events", ctypes.c_int64), ("until", ctypes.c_double),
                ("max_rounds", ctypes.c_int32), ("block_threads", ctypes.c_int32),
                ("debug", ctypes.c_int32), ("single_clock", ctypes.c_int32),
                ("assist_min_flows", ctypes.c_int32), ("assist_helpers", ctypes.c_int32),
                ("exact", ctypes.c_int32), ("history_mb", ctypes.c_int32)]


class netsim_topology(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("servers", ctypes.c_int32),
                ("gpus_per_server", ctypes.c_int32), ("servers_per_leaf", ctypes.c_int32),
                ("spines", ctypes.c_int32), ("pods", ctypes.c_int32),
                ("edges_per_pod", ctypes.c_int32), ("aggs_per_pod", ctypes.c_int32),
                ("agg_uplinks", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("nvlink_Bps", ctypes.c_double), ("nic_Bps", ctypes.c_double),
                ("fabric_Bps", ctypes.c_double), ("ecmp_seed", ctypes.c_uint64),
                ("num_degraded", ctypes.c_int64),
                ("degraded_cables", ctypes.POINTER(ctypes.c_int64)),
                ("degraded_Bps", ctypes.c_double),
                ("fabric_latency_s", ctypes.c_double), ("nvlink_latency_s", ctypes.c_double)]


class netsim_stats(ctypes.Structure):
    _fields_ = [("events", ctypes.c_int64), ("solves", ctypes.c_int64),
                ("rounds", ctypes.c_int64), ("flows_swept", ctypes.c_int64),
                ("incidences_swept", ctypes.c_int64), ("active_swept", ctypes.c_int64),
                ("pending_swept", ctypes.c_int64), ("completed_flows", ctypes.c_int64),
                ("reselected", ctypes.c_int64), ("wide_solves", ctypes.c_int64),
                ("complete", ctypes.c_int32), ("parts", ctypes.c_int32),
                ("sim_time", ctypes.c_double), ("device_seconds", ctypes.c_double),
                ("upload_seconds", ctypes.c_double), ("phase_seconds", ctypes.c_double * 8),
                ("assisted_solves", ctypes.c_int64), ("layout", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("links_swept", ctypes.c_int64),
                ("launch_events", ctypes.c_int64)]

    def as_dict(self):
        d = {k: getattr(self, k) for k, _ in self._fields_ if k != "reserved"}
        d["phase_seconds"] = list(self.phase_seconds)
        return d


class NetsimError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


_P = ctypes.c_void_p
_H = ctypes.c_void_p
_I32, _I64, _D = ctypes.c_int32, ctypes.c_int64, ctypes.c_double

# name -> (restype, argtypes)
_SIGS = {
    "netsim_default_options": (None, [ctypes.POINTER(netsim_options)]),
    "netsim_create": (_I32, [ctypes.POINTER(_H), _I32, _P, _P, ctypes.POINTER(netsim_options)]),
    "netsim_create_topology": (_I32, [ctypes.POINTER(_H), _I32, ctypes.POINTER(netsim_topology),
                                      ctypes.POINTER(netsim_options)]),
    "netsim_get_links": (_I32, [_H, _I32, ctypes.POINTER(_I64), _P]),
    "netsim_add_flows": (_I32, [_H, _I32, _I64, _P, _P, _P, _P, _P, _P, _P, _P,
                                ctypes.POINTER(_I64)]),
    "netsim_add_ring": (_I32, [_H, _I32, _I32, _I32, _I32, _P, _D, _D, _I64, _P,
                               ctypes.POINTER(_I64), ctypes.POINTER(_I64)]),
    "netsim_add_all_to_all": (_I32, [_H, _I32, _I32, _P, _P, _D, _I64, _P,
                                     ctypes.POINTER(_I64), ctypes.POINTER(_I64)]),
    "netsim_add_tree_allreduce": (_I32, [_H, _I32, _I32, _P, _D, _D, _I64, _P,
                                         ctypes.POINTER(_I64), ctypes.POINTER(_I64)]),
    "netsim_add_hier_allreduce": (_I32, [_H, _I32, _I32, _I32, _P, _D, _D, _I64, _P,
                                         ctypes.POINTER(_I64), ctypes.POINTER(_I64)]),
    "netsim_set_link_latency": (_I32, [_H, _I32, _I64, _P]),
    "netsim_stream_tree_allreduce": (_I32, [_H, _I32, _I32, _P, _P, _D, _P]),
    "netsim_stream_hier_allreduce": (_I32, [_H, _I32, _I32, _I32, _P, _P, _D, _P]),
    "netsim_counts": (_I32, [_H, ctypes.POINTER(_I64), ctypes.POINTER(_I64), ctypes.POINTER(_I64)]),
    "netsim_last_exits": (_I32, [_H, ctypes.POINTER(_I64), _P]),
    "netsim_export_flows": (_I32, [_H, _P, _P, _P, _P, _P, _P, _P, _P, _P]),
    "netsim_set_limits": (_I32, [_H, _I64, _D]),
    "netsim_run": (_I32, [_H, _P]),
    "netsim_get_finish": (_I32, [_H, _P, _P]),
    "netsim_get_finish_device": (_I32, [_H, _P]),
    "netsim_get_stats": (_I32, [_H, ctypes.POINTER(netsim_stats)]),
    "netsim_solve_once": (_I32, [_H, _I32, _I64, _P, _P]),
    "netsim_advance": (_I32, [_H, _D, _I64, _P]),
    "netsim_stream_compute": (_I32, [_H, _I32, _I64, _D, _I64, _P, ctypes.POINTER(_I64)]),
    "netsim_stream_wait": (_I32, [_H, _I32, _I64, _I64, _P]),
    "netsim_stream_tail": (_I32, [_H, _I32, _I64, ctypes.POINTER(_I64)]),
    "netsim_stream_ring": (_I32, [_H, _I32, _I32, _I32, _I32, _P, _P, _D, _P]),
    "netsim_stream_all_to_all": (_I32, [_H, _I32, _I32, _P, _P, _P, _P]),
    "netsim_stream_send": (_I32, [_H, _I32, _I32, _I64, _I32, _I64, _D, ctypes.POINTER(_I64)]),
    "netsim_update_start": (_I32, [_H, _I64, _D]),
    "netsim_gc": (_I32, [_H, _D]),
    "netsim_num_checkpoints": (_I32, [_H, ctypes.POINTER(_I64)]),
    "netsim_solve_rates_noalloc": (_I32, [_I32, _I32, _P, _I32, _P, _P, _P, _P, _P]),
    "netsim_bench_sweeps": (_I32, [_H, _I32, _I64, _P, _I32, _I64, _P, _P, _P, _P, _P]),
    "netsim_last_error": (ctypes.c_char_p, [_H]),
    "netsim_destroy": (None, [_H]),
}

_lib = None


def load_library(path: str = LIB_PATH):
    """Loads libnetsim.so and declares every exported entry point."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"libnetsim is not built ({path} missing); run "
                          "`python -m paper_2505_01616_amd.build`")
    lib = ctypes.CDLL(path)
    for name, (res, args) in _SIGS.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _arr(x, dtype):
    return None if x is None else np.ascontiguousarray(x, dtype=dtype)


def _check(h, rc):
    if rc != OK:
        msg = _lib.netsim_last_error(h)
        raise NetsimError(rc, msg.decode() if msg else "")


def netsim_default_options() -> netsim_options:
    o = netsim_options()
    load_library().netsim_default_options(ctypes.byref(o))
    return o


def make_options(device=0, exec=EXEC_AUTO, max_events=0, until=math.inf, max_rounds=0,
                 block_threads=0, debug=0, single_clock=0, assist_min_flows=0,
                 assist_helpers=0, exact=0, history_mb=0) -> netsim_options:
    o = netsim_default_options()
    o.device, o.exec, o.max_events, o.until = device, exec, max_events, until
    o.max_rounds, o.block_threads, o.debug = max_rounds, block_threads, debug
    o.single_clock, o.assist_min_flows, o.assist_helpers = single_clock, assist_min_flows, assist_helpers
    o.exact, o.history_mb = exact, history_mb
    return o


def netsim_create(link_off, capacity_Bps, opt: Optional[netsim_options] = None) -> int:
    lib = load_library()
    lo = _arr(link_off, np.int64)
    cap = _arr(capacity_Bps, np.float64)
    h = _H()
    rc = lib.netsim_create(ctypes.byref(h), len(lo) - 1, _ptr(lo), _ptr(cap),
                           ctypes.byref(opt) if opt is not None else None)
    _check(None, rc)
    return h.value


def netsim_create_topology(topos, opt: Optional[netsim_options] = None) -> int:
    """topos: list of netsim_topology (keep referenced arrays alive)."""
    lib = load_library()
    arr = (netsim_topology * len(topos))(*topos)
    h = _H()
    rc = lib.netsim_create_topology(ctypes.byref(h), len(topos), arr,
                                    ctypes.byref(opt) if opt is not None else None)
    _check(None, rc)
    return h.value


def netsim_get_links(h, scen):
    lib = load_library()
    n = _I64()
    _check(h, lib.netsim_get_links(h, scen, ctypes.byref(n), None))
    cap = np.zeros(n.value)
    _check(h, lib.netsim_get_links(h, scen, ctypes.byref(n), _ptr(cap)))
    return cap


def netsim_add_flows(h, scen, nbytes, start, src=None, dst=None, path_off=None, path_link=None,
                     dep_off=None, dep_ids=None) -> int:
    lib = load_library()
    nb = _arr(nbytes, np.float64)
    st = _arr(start, np.float64)
    s, d = _arr(src, np.int32), _arr(dst, np.int32)
    po, pl = _arr(path_off, np.int64), _arr(path_link, np.int32)
    do, di = _arr(dep_off, np.int64), _arr(dep_ids, np.int64)
    first = _I64(-1)
    rc = lib.netsim_add_flows(h, scen, len(nb), _ptr(s), _ptr(d), _ptr(nb), _ptr(st), _ptr(po),
                              _ptr(pl), _ptr(do), _ptr(di), ctypes.byref(first))
    _check(h, rc)
    return first.value


def netsim_add_ring(h, scen, kind, mode, ranks, nbytes, lag=0.0, after=()):
    lib = load_library()
    r = _arr(ranks, np.int32)
    a = _arr(np.asarray(after, dtype=np.int64), np.int64)
    first, count = _I64(-1), _I64(0)
    rc = lib.netsim_add_ring(h, scen, kind, mode, len(r), _ptr(r), float(nbytes), float(lag),
                             len(a), _ptr(a) if len(a) else None, ctypes.byref(first),
                             ctypes.byref(count))
    _check(h, rc)
    return first.value, count.value


def netsim_add_tree_allreduce(h, scen, ranks, nbytes, lag=0.0, after=()):
    lib = load_library()
    r = _arr(ranks, np.int32)
    a = _arr(np.asarray(after, dtype=np.int64), np.int64)
    first, count = _I64(-1), _I64(0)
    _check(h, lib.netsim_add_tree_allreduce(h, scen, len(r), _ptr(r), float(nbytes), float(lag),
                                            len(a), _ptr(a) if len(a) else None,
                                            ctypes.byref(first), ctypes.byref(count)))
    return first.value, count.value


def netsim_add_hier_allreduce(h, scen, ranks, nbytes, lag=0.0, after=()):
    """ranks: an m x g array (row = server)."""
    lib = load_library()
    r2 = np.asarray(ranks)
    m, g = r2.shape
    r = _arr(r2.reshape(-1), np.int32)
    a = _arr(np.asarray(after, dtype=np.int64), np.int64)
    first, count = _I64(-1), _I64(0)
    _check(h, lib.netsim_add_hier_allreduce(h, scen, m, g, _ptr(r), float(nbytes), float(lag),
                                            len(a), _ptr(a) if len(a) else None,
                                            ctypes.byref(first), ctypes.byref(count)))
    return first.value, count.value


def netsim_set_link_latency(h, scen, latency_s):
    lat = _arr(latency_s, np.float64)
    _check(h, load_library().netsim_set_link_latency(h, scen, len(lat), _ptr(lat) if len(lat) else None))


def netsim_add_all_to_all(h, scen, ranks, nbytes, lag=0.0, after=()):
    lib = load_library()
    r = _arr(ranks, np.int32)
    m = _arr(nbytes, np.float64)
    a = _arr(np.asarray(after, dtype=np.int64), np.int64)
    first, count = _I64(-1), _I64(0)
    rc = lib.netsim_add_all_to_all(h, scen, len(r), _ptr(r), _ptr(m), float(lag), len(a),
                                   _ptr(a) if len(a) else None, ctypes.byref(first),
                                   ctypes.byref(count))
    _check(h, rc)
    return first.value, count.value


def netsim_counts(h):
    lib = load_library()
    f, z, d = _I64(), _I64(), _I64()
    _check(h, lib.netsim_counts(h, ctypes.byref(f), ctypes.byref(z), ctypes.byref(d)))
    return f.value, z.value, d.value


def netsim_last_exits(h) -> np.ndarray:
    lib = load_library()
    n = _I64()
    _check(h, lib.netsim_last_exits(h, ctypes.byref(n), None))
    ids = np.zeros(max(n.value, 1), np.int64)
    _check(h, lib.netsim_last_exits(h, ctypes.byref(n), _ptr(ids)))
    return ids[: n.value]


def netsim_export_flows(h) -> dict:
    lib = load_library()
    F, nnz, nd = netsim_counts(h)
    out = dict(scen=np.zeros(F, np.int32), src=np.zeros(F, np.int32), dst=np.zeros(F, np.int32),
               nbytes=np.zeros(F), start=np.zeros(F), path_off=np.zeros(F + 1, np.int64),
               path_link=np.zeros(max(nnz, 1), np.int32), dep_off=np.zeros(F + 1, np.int64),
               dep_ids=np.zeros(max(nd, 1), np.int64))
    _check(h, lib.netsim_export_flows(h, *[_ptr(out[k]) for k in
                                           ("scen", "src", "dst", "nbytes", "start", "path_off",
                                            "path_link", "dep_off", "dep_ids")]))
    out["path_link"] = out["path_link"][:nnz]
    out["dep_ids"] = out["dep_ids"][:nd]
    return out


def netsim_set_limits(h, max_events=0, until=math.inf):
    _check(h, load_library().netsim_set_limits(h, int(max_events), float(until)))


def _stream(stream):
    """None, an int handle, or an object with a ``cuda_stream`` attribute
    (a torch.cuda.Stream)."""
    if stream is not None and not isinstance(stream, int):
        stream = stream.cuda_stream
    return stream


def netsim_run(h, stream=None):
    _check(h, load_library().netsim_run(h, _stream(stream)))


def netsim_get_finish(h):
    lib = load_library()
    F = netsim_counts(h)[0]
    fin = np.zeros(max(F, 1))
    _check(h, lib.netsim_get_finish(h, _ptr(fin), None))
    return fin[:F]


def netsim_get_makespan(h, num_scenarios):
    lib = load_library()
    F = netsim_counts(h)[0]
    fin = np.zeros(max(F, 1))
    ms = np.zeros(num_scenarios)
    _check(h, lib.netsim_get_finish(h, _ptr(fin), _ptr(ms)))
    return ms


def netsim_get_finish_device(h, d_ptr: int):
    _check(h, load_library().netsim_get_finish_device(h, ctypes.c_void_p(d_ptr)))


def netsim_get_stats(h) -> dict:
    s = netsim_stats()
    _check(h, load_library().netsim_get_stats(h, ctypes.byref(s)))
    return s.as_dict()


def netsim_solve_once(h, scen, active_ids):
    ids = _arr(active_ids, np.int64)
    rates = np.zeros(max(len(ids), 1))
    _check(h, load_library().netsim_solve_once(h, scen, len(ids), _ptr(ids), _ptr(rates)))
    return rates[: len(ids)]


def netsim_stream_compute(h, scen, stream, duration, wait=()) -> int:
    w = _arr(list(wait), np.int64)
    out = _I64()
    _check(h, load_library().netsim_stream_compute(h, scen, int(stream), float(duration), len(w),
                                                   _ptr(w) if len(w) else None, ctypes.byref(out)))
    return out.value


def netsim_stream_wait(h, scen, stream, wait):
    w = _arr(list(wait), np.int64)
    _check(h, load_library().netsim_stream_wait(h, scen, int(stream), len(w), _ptr(w) if len(w) else None))


def netsim_stream_tail(h, scen, stream) -> int:
    out = _I64()
    _check(h, load_library().netsim_stream_tail(h, scen, int(stream), ctypes.byref(out)))
    return out.value


def netsim_stream_ring(h, scen, kind, mode, ranks, streams, nbytes) -> np.ndarray:
    r = _arr(ranks, np.int32)
    st = _arr(streams, np.int64)
    done = np.zeros(len(r), np.int64)
    _check(h, load_library().netsim_stream_ring(h, scen, kind, mode, len(r), _ptr(r), _ptr(st),
                                                float(nbytes), _ptr(done)))
    return done


def netsim_stream_all_to_all(h, scen, ranks, streams, nbytes) -> np.ndarray:
    r = _arr(ranks, np.int32)
    st = _arr(streams, np.int64)
    b = _arr(nbytes, np.float64).reshape(-1)
    done = np.zeros(len(r), np.int64)
    _check(h, load_library().netsim_stream_all_to_all(h, scen, len(r), _ptr(r), _ptr(st), _ptr(b),
                                                      _ptr(done)))
    return done


def netsim_stream_tree_allreduce(h, scen, ranks, streams, nbytes) -> np.ndarray:
    r = _arr(ranks, np.int32)
    st = _arr(streams, np.int64)
    done = np.zeros(len(r), np.int64)
    _check(h, load_library().netsim_stream_tree_allreduce(h, scen, len(r), _ptr(r), _ptr(st),
                                                          float(nbytes), _ptr(done)))
    return done


def netsim_stream_hier_allreduce(h, scen, ranks, streams, nbytes) -> np.ndarray:
    """ranks: m x g (row = server); streams in the same row-major order."""
    r2 = np.asarray(ranks)
    m, g = r2.shape
    r = _arr(r2.reshape(-1), np.int32)
    st = _arr(np.asarray(streams).reshape(-1), np.int64)
    done = np.zeros(len(r), np.int64)
    _check(h, load_library().netsim_stream_hier_allreduce(h, scen, m, g, _ptr(r), _ptr(st),
                                                          float(nbytes), _ptr(done)))
    return done


def netsim_stream_send(h, scen, src, src_stream, dst, dst_stream, nbytes) -> int:
    out = _I64()
    _check(h, load_library().netsim_stream_send(h, scen, int(src), int(src_stream), int(dst),
                                                int(dst_stream), float(nbytes), ctypes.byref(out)))
    return out.value


def netsim_advance(h, until=math.inf, max_events=0, stream=None):
    _check(h, load_library().netsim_advance(h, float(until), int(max_events), _stream(stream)))


def netsim_update_start(h, flow_id, start):
    _check(h, load_library().netsim_update_start(h, int(flow_id), float(start)))


def netsim_gc(h, t_min):
    _check(h, load_library().netsim_gc(h, float(t_min)))


def netsim_num_checkpoints(h) -> int:
    n = _I64()
    _check(h, load_library().netsim_num_checkpoints(h, ctypes.byref(n)))
    return n.value


def netsim_bench_sweeps(h, scen, active_ids, reps, flush_bytes, stream=None):
    """Per-repetition times (ms) of the count and freezing sweeps: with HIP
    events (dispatch included) and inside the kernels."""
    ids = _arr(active_ids, np.int64)
    a, b, c, d = (np.zeros(int(reps)) for _ in range(4))
    _check(h, load_library().netsim_bench_sweeps(h, scen, len(ids), _ptr(ids), int(reps),
                                                 int(flush_bytes), _stream(stream), _ptr(a), _ptr(b),
                                                 _ptr(c), _ptr(d)))
    return {"count_ms": a, "freeze_ms": b, "count_kernel_ms": c, "freeze_kernel_ms": d}


def netsim_solve_rates_noalloc(device, num_links, d_cap, num_flows, d_path_off, d_path_link,
                               d_rates, d_status, stream=None):
    """Arguments are device addresses (ints, e.g. torch tensors' data_ptr());
    enqueues the solve and returns; d_status[0] holds the solve's status."""
    _check(None, load_library().netsim_solve_rates_noalloc(
        int(device), int(num_links), _P(d_cap), int(num_flows), _P(d_path_off), _P(d_path_link),
        _P(d_rates), _P(d_status), _stream(stream)))


def netsim_last_error(h=None) -> str:
    msg = load_library().netsim_last_error(h)
    return msg.decode() if msg else ""


def netsim_destroy(h):
    if h:
        load_library().netsim_destroy(h)
