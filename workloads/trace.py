"""Traces of stream operations: the input of the event-queue front end.

A trace is what the simulator's tracer and intercepted CUDA/NCCL calls
deliver (paper Section 4.1): per rank, operations issued on CUDA streams --
computations of known duration, waits on events recorded on other streams,
NCCL collectives and point-to-point transfers issued by every rank of a
communicator on its own stream.  A trace is plain data: each side of a
parity check (the library's front end, the oracle's) turns it into flows
with its own code.

References: ``Ref = (op_index, position)`` names the completion of an earlier
operation on one of its streams -- position 0 for ``Compute`` and
``StreamWait``, the rank's position for ``Collective``, 0 (sender) or 1
(receiver) for ``SendRecv``.  A reference is what a CUDA event recorded
right after that operation would complete with.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Sequence, Tuple, Union

import numpy as np

from .program import MiB, Topology, gbit
from .rng import Stream

Ref = Tuple[int, int]


@dataclass
class Compute:
    stream: int
    duration: float
    wait: Sequence[Ref] = ()


@dataclass
class StreamWait:
    stream: int
    wait: Sequence[Ref]


@dataclass
class Collective:
    # "allreduce" | "reduce_scatter" | "all_gather" (rings), "all_to_all",
    # "tree_allreduce" (double binary tree), "hier_allreduce" (ranks and
    # streams m x g, row = server)
    kind: str
    ranks: np.ndarray
    streams: np.ndarray             # the stream each rank issues it on (same shape)
    nbytes: Union[float, np.ndarray]  # total bytes; p x p matrix for all_to_all
    mode: str = "chained"           # rings only


@dataclass
class SendRecv:
    src: int
    src_stream: int
    dst: int
    dst_stream: int
    nbytes: float


TraceOp = Union[Compute, StreamWait, Collective, SendRecv]


@dataclass
class Trace:
    name: str
    topo: Topology
    ops: List[TraceOp] = field(default_factory=list)

    def add(self, op: TraceOp) -> int:
        for k, j in getattr(op, "wait", ()):
            if not (0 <= k < len(self.ops)) or not (0 <= j < positions(self.ops[k])):
                raise ValueError("a wait must name an earlier operation and one of its streams")
        if isinstance(op, Collective):
            n = np.size(op.ranks)
            if n < 2 or np.shape(op.streams) != np.shape(op.ranks) \
                    or len(set(int(x) for x in np.ravel(op.streams))) != n:
                raise ValueError("a collective needs p >= 2 ranks on p distinct streams")
        if isinstance(op, SendRecv) and (op.src == op.dst or op.src_stream == op.dst_stream):
            raise ValueError("a send/recv joins two ranks on two streams")
        self.ops.append(op)
        return len(self.ops) - 1


def positions(op: TraceOp) -> int:
    """Number of streams an operation completes on."""
    if isinstance(op, Collective):
        return int(np.size(op.ranks))
    return 2 if isinstance(op, SendRecv) else 1


def training_step(seed: int = 6, tp: int = 8, pp: int = 4, dp: int = 4, microbatches: int = 8,
                  layers: int = 4, fwd_s: float = 1.2e-3, bwd_s: float = 2.4e-3,
                  tp_bytes: float = 16 * MiB, act_bytes: float = 32 * MiB,
                  grad_bytes: float = 512 * MiB, optim_s: float = 0.5e-3,
                  jitter: float = 0.1, allreduce: str = "ring", fabric_latency_s: float = 0.0,
                  nvlink_latency_s: float = 0.0) -> Trace:
    """One 3D-parallel (TP x PP x DP) training step with a GPipe schedule.

    Rank ``t + tp*(d + dp*s)`` is tensor position t of data-parallel replica
    d in pipeline stage s; eight ranks per server, so with tp = 8 tensor
    parallelism stays inside a server and the pipeline and data-parallel
    peers of a rank share its rail.  Every rank has a compute stream
    (2*rank) and a communication stream (2*rank + 1).

    Forward, per micro-batch, replica and stage: ``layers`` computations,
    each followed (tp > 1) by a tensor-parallel ring all-reduce of
    ``tp_bytes`` on the compute streams; then the activations go to the
    next stage as a send/recv of ``act_bytes`` on the communication streams
    (the send waits for the forward through an event; the next stage's
    compute stream waits for the receive).  The backward pass mirrors this
    in reverse stage order after every forward has been issued.  Finally,
    per (stage, tensor position), a data-parallel ring all-reduce of
    ``grad_bytes`` on the communication streams after each rank's last
    backward, and an optimizer computation on the compute stream after it.
    Computation times are the per-layer times with a seeded multiplicative
    jitter uniform in [1 - jitter, 1 + jitter].  Fabric: rail-optimised,
    one leaf per rail, 400 Gb/s NICs and switch cables, eight spines, with
    the given link latencies.  ``allreduce`` picks the algorithm of every
    all-reduce: "ring" (chained) or "tree" (double binary tree).
    """
    nranks = tp * pp * dp
    servers = max(1, -(-nranks // 8))
    topo = Topology(kind="rail", servers=servers, gpus_per_server=8, servers_per_leaf=servers,
                    spines=8, nvlink_Bps=900e9, nic_Bps=gbit(400), fabric_Bps=gbit(400),
                    ecmp_seed=int(Stream(seed, "trace-ecmp").u64(1)[0]),
                    fabric_latency_s=fabric_latency_s, nvlink_latency_s=nvlink_latency_s)
    ar = "allreduce" if allreduce == "ring" else "tree_allreduce"
    tr = Trace(f"training step tp{tp} pp{pp} dp{dp} mb{microbatches}", topo)
    draws = Stream(seed, "trace-jitter")
    nd = [0]

    def jittered(base):
        u = float(draws.u01(1, nd[0])[0])
        nd[0] += 1
        return base * (1.0 + jitter * (2.0 * u - 1.0))

    def rank(t, d, s):
        return t + tp * (d + dp * s)

    def comp(r):
        return 2 * r

    def comm(r):
        return 2 * r + 1

    last = {}       # rank -> reference to the last operation on its compute stream

    def stage_pass(d, s, m, per_layer, recv):
        ranks = np.array([rank(t, d, s) for t in range(tp)], np.int32)
        if recv is not None:
            for t, r in enumerate(ranks):
                last[int(r)] = (tr.add(StreamWait(comp(r), [recv[t]])), 0)
        for _ in range(layers):
            for r in ranks:
                last[int(r)] = (tr.add(Compute(comp(r), jittered(per_layer))), 0)
            if tp > 1:
                k = tr.add(Collective(ar, ranks, np.array([comp(r) for r in ranks]), tp_bytes))
                for t, r in enumerate(ranks):
                    last[int(r)] = (k, t)
        return ranks

    def send_to(ranks, d, s_to):
        recv = []
        for t, a in enumerate(ranks):
            b = rank(t, d, s_to)
            tr.add(StreamWait(comm(a), [last[int(a)]]))
            recv.append((tr.add(SendRecv(int(a), comm(a), b, comm(b), act_bytes)), 1))
        return recv

    fwd_recv, bwd_recv = {}, {}
    for m in range(microbatches):
        for d in range(dp):
            for s in range(pp):
                ranks = stage_pass(d, s, m, fwd_s / layers, fwd_recv.get((d, s, m)))
                if s + 1 < pp:
                    fwd_recv[(d, s + 1, m)] = send_to(ranks, d, s + 1)
    for m in range(microbatches):
        for d in range(dp):
            for s in reversed(range(pp)):
                ranks = stage_pass(d, s, m, bwd_s / layers, bwd_recv.get((d, s, m)))
                if s > 0:
                    bwd_recv[(d, s - 1, m)] = send_to(ranks, d, s - 1)
    for s in range(pp):
        for t in range(tp):
            ranks = np.array([rank(t, d, s) for d in range(dp)], np.int32)
            if dp > 1:
                for r in ranks:
                    tr.add(StreamWait(comm(r), [last[int(r)]]))
                k = tr.add(Collective(ar, ranks, np.array([comm(r) for r in ranks]), grad_bytes))
                for i, r in enumerate(ranks):
                    last[int(r)] = (tr.add(Compute(comp(r), jittered(optim_s), wait=[(k, i)])), 0)
            else:
                r = int(ranks[0])
                last[r] = (tr.add(Compute(comp(r), jittered(optim_s))), 0)
    return tr
