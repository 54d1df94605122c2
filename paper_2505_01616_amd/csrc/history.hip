// Time rollback to an earlier event from the rollback history (paper
// Section 4.2: the throughput history of every flow lets the simulator
// return to the state it had at any earlier event, then re-simulate from
// there).
//
// The event loop records, per part, an undo record for every flow it takes
// back for a re-solve (the flow's remaining bytes, their time and its rate
// from before that event) and a record of every event (its time, the undo
// records written up to its end, the part's statistics at its end), and it
// notes per flow the events at which the flow's last predecessor finished
// (evr), at which it became active (eva) and at which it finished (evd).
// Going back to the end of event es:
//   1. flows finished after es lose their finish time; flows that became
//      active after es are waiting or pending again; flows whose last
//      predecessor finished after es are waiting, with their initial count,
//      release time and base;
//   2. every flow finished by es counts down its waiting successors (and,
//      with link latency, raises their base to its arrival, as the event
//      loop does);
//   3. each flow's first undo record after es gives back its remaining
//      bytes, their time and its rate at es (a flow with none kept them);
//   4. the active flows fill the slots again (predicted completion
//      tref + rem / rate, the same operations as the event loop's) and the
//      pending ones the pending list of event es + 1;
//   5. the part's control block resumes at event es + 1.
// The slot order differs from the original run's; nothing the event loop
// computes depends on it (minima, integer sums, per-flow updates).
#include "device.h"

namespace netsim_dev {

namespace {

__global__ void hist_flows_kernel(Params P, int f0, int f1, int32_t es, const int32_t* cnt0,
                                  const double* rel0, int32_t* first) {
  const int f = f0 + (int)(blockIdx.x * blockDim.x + threadIdx.x);
  if (f >= f1) return;
  const int i = f - f0;
  const bool done = P.evd[f] <= es;
  const bool act = !done && P.eva[f] <= es;
  const bool ready = cnt0[i] == 0 || P.evr[f] <= es;
  if (!done) {
    P.finish[f] = __longlong_as_double(0x7FF8000000000000ll);  // NaN: not finished
    P.evd[f] = EV_NEVER;
  }
  if (!done && !act) P.eva[f] = EV_NEVER;
  if (!ready) {
    P.evr[f] = EV_NEVER;
    P.cnt[f] = cnt0[i];
    P.base[f] = 0.0;
    P.rel[f] = rel0[i];
  } else {
    P.cnt[f] = 0;
  }
  first[i] = 0x7FFFFFFF;
}

__global__ void hist_succ_kernel(Params P, int f0, int f1) {
  const int f = f0 + (int)(blockIdx.x * blockDim.x + threadIdx.x);
  if (f >= f1 || P.evd[f] == EV_NEVER) return;
  for (int k = P.soff[f]; k < P.soff[f + 1]; ++k) {
    const int s = P.succ[k];
    if (P.evr[s] != EV_NEVER) continue;  // released by es: its count is zero
    if (P.lat)
      __hip_atomic_fetch_max(reinterpret_cast<unsigned long long*>(&P.base[s]),
                             (unsigned long long)__double_as_longlong(P.finish[f]), __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_fetch_add(&P.cnt[s], -1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// first[f - f0]: offset from p0 of the flow's first undo record in [p0, p1)
__global__ void hist_first_kernel(Params P, int f0, int f1, int64_t hbase, int64_t hcap, int64_t p0,
                                  int64_t n, int32_t* first) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int f = P.hist[hbase + (p0 + i) % hcap].f;
    if (f >= f0 && f < f1)
      __hip_atomic_fetch_min(&first[f - f0], (int32_t)i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

__global__ void hist_apply_kernel(Params P, int f0, int f1, int64_t hbase, int64_t hcap, int64_t p0,
                                  const int32_t* first) {
  const int f = f0 + (int)(blockIdx.x * blockDim.x + threadIdx.x);
  if (f >= f1) return;
  const int32_t k = first[f - f0];
  if (k == 0x7FFFFFFF) return;
  const HistUndo u = P.hist[hbase + (p0 + k) % hcap];
  P.rem[f] = u.rem;
  P.tref[f] = u.tref;
  P.rate[f] = u.rate;
}

// counters[0]: slots filled, counters[1]: pending flows listed
__global__ void hist_lists_kernel(Params P, int f0, int f1, int32_t es, uint32_t* counters) {
  const int f = f0 + (int)(blockIdx.x * blockDim.x + threadIdx.x);
  if (f >= f1) return;
  if (P.evd[f] != EV_NEVER) return;  // finished by es
  if (P.eva[f] != EV_NEVER) {
    const uint32_t s = atomicAdd(&counters[0], 1u);
    const double r = P.rate[f];
    P.act0[f0 + s] = f;
    P.srate0[f0 + s] = r;
    P.tau0[f0 + s] = P.tref[f] + P.rem[f] / r;
  } else if (P.evr[f] != EV_NEVER || P.cnt[f] == 0) {
    const uint32_t s = atomicAdd(&counters[1], 1u);
    int32_t* pend = ((es + 1) & 1) ? P.pend1 : P.pend0;
    pend[f0 + s] = f;
  }
}

__global__ void hist_ctl_kernel(Params P, int p, int32_t es, HistEv rec, const uint32_t* counters) {
  ScenCtl* C = &P.ctl[p];
  C->started = 1;
  C->e = es + 1;
  C->q = 0;
  C->ab = 0;
  C->nslots = (int32_t)counters[0];
  C->holes = 0;
  C->npend = (int32_t)counters[1];
  C->t = rec.t;
  C->events = es + 1;
  C->solves = rec.solves;
  C->rounds = rec.rounds;
  C->flows_swept = rec.flows_swept;
  C->active_swept = rec.active_swept;
  C->pending_swept = rec.pending_swept;
  C->reselected = rec.reselected;
  C->wide_solves = rec.wide_solves;
  C->assisted = rec.assisted;
  C->hpos = rec.hpos;
  C->status = ST_STOPPED;
  C->k = Lists{};
}

}  // namespace

hipError_t history_restore(const Params& P, int p, int f0, int f1, int64_t hbase, int64_t hcap, int32_t es,
                           const HistEv& rec, int64_t hpos_now, const int32_t* cnt0, const double* rel0,
                           int32_t* first, uint32_t* counters, hipStream_t st) {
  const int n = f1 - f0;
  const int T = 256;
  const int B = (n + T - 1) / T;
  hipError_t e = hipMemsetAsync(counters, 0, 2 * sizeof(uint32_t), st);
  if (e != hipSuccess) return e;
  if (n > 0) {
    hipLaunchKernelGGL(hist_flows_kernel, dim3(B), dim3(T), 0, st, P, f0, f1, es, cnt0, rel0, first);
    hipLaunchKernelGGL(hist_succ_kernel, dim3(B), dim3(T), 0, st, P, f0, f1);
    const int64_t nu = hpos_now - rec.hpos;
    if (nu > 0) {
      const int64_t want = (nu + T - 1) / T;
      const int blocks = (int)(want < 65536 ? want : 65536);
      hipLaunchKernelGGL(hist_first_kernel, dim3(blocks), dim3(T), 0, st, P, f0, f1, hbase, hcap, rec.hpos,
                         nu, first);
    }
    hipLaunchKernelGGL(hist_apply_kernel, dim3(B), dim3(T), 0, st, P, f0, f1, hbase, hcap, rec.hpos, first);
    hipLaunchKernelGGL(hist_lists_kernel, dim3(B), dim3(T), 0, st, P, f0, f1, es, counters);
  }
  hipLaunchKernelGGL(hist_ctl_kernel, dim3(1), dim3(1), 0, st, P, p, es, rec, counters);
  return hipGetLastError();
}

}  // namespace netsim_dev
