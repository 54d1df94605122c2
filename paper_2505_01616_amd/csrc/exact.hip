// Exact progressive filling on gfx950: the event loop and rate solve of the
// fluid model carried out with the arithmetic of a sequential fp64 program,
// one workgroup per scenario (batched scenarios run side by side).
//
// Model (Section 4.1, netsim; Section 4.2, the network simulator with time
// rollback): active flows share link bandwidth max-min fairly (per-flow
// fairness), rates stay constant between consecutive events, the loop jumps
// to the next release or completion and solves the rates again.
//
// Rate solve: progressive filling, one bottleneck level per iteration (the
// water-filling of Section 4.2: find the bottleneck link, give its flows
// their share, repeat).  Every link crossed by an active flow starts with
// residual capacity R_l = c_l and unfrozen count n_l; per level
//   s_l = R_l / n_l for every link with n_l > 0, s* = min_l s_l
//     (LDS-staged block minimum: wave shuffles, then one value per wave);
//   the links with s_l <= s* * THR (THR = 1 + 1e-12) are the bottlenecks;
//     every unfrozen flow crossing one gets rate s* (a sweep over the
//     unfrozen list: each flow looks up its links' shares);
//   k_l = flows frozen on l (integer atomics); R_l = R_l - k_l * s* (the
//     product rounded, then the difference), n_l -= k_l.
// Event loop: t_next = min(earliest pending release, min over active flows
// of t + rem/r); active flows with t + rem/r <= t_next * THR send their last
// byte at t_next (finish = t_next + path latency), the others lose
// r * (t_next - t) bytes; dependants whose predecessors have all finished
// are released at start + latest predecessor finish; pending flows released
// at or before t arrive (zero-byte flows finish at once and release their
// dependants in turn, to a fixpoint); if the active set changed it is solved
// again.
//
// Every value is rounded as a sequential program rounds it: no contraction
// of products into sums, IEEE division, minima (exact in any order) and
// integer counts.  Nothing depends on the order in which threads run, so the
// finish times are the same bit for bit for any workgroup size.
#include "device.h"
#include "netsim.h"

#include <math.h>

#include <mutex>
#include <string>

#pragma clang fp contract(off)

namespace netsim_dev {

namespace {

constexpr double XTHR = 1.000000000001;
constexpr int DEBUG_EXACT_GLOBAL_LINKS = 16;  // options.debug bit 4
constexpr double XINF = __builtin_huge_val();

// Work-list counters of the part a workgroup runs (shared memory).
struct XShared {
  double red[2][16];  // block minimum: one value per wave, two buffers
  int32_t nact[2];    // active lists
  int32_t npend[2];   // pending lists
  int32_t ndone[2];   // flows finished in the current wave of releases
  int32_t nunf[2];    // unfrozen flows of the current solve
  int32_t nlive[2];   // links with unfrozen flows
  int32_t changed;    // the active set changed in this event
  int32_t fault;      // a work list held an id outside the part
  int64_t fsw, isw;   // flows / incidences swept (summed over waves)
  int64_t lsw;        // links with unfrozen flows, summed over levels
};

__device__ __forceinline__ double xwave_min(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const double w = __shfl_xor(v, o, 64);
    v = w < v ? w : v;
  }
  return v;
}

// Minimum over the workgroup.  Every thread reads the per-wave values after
// one barrier; the two buffers alternate, so a fast thread's next call never
// overwrites values a slow thread still reads (it passes a barrier first).
__device__ __forceinline__ double xblock_min(double v, XShared& sh, int& rb) {
  v = xwave_min(v);
  if ((threadIdx.x & 63) == 0) sh.red[rb][threadIdx.x >> 6] = v;
  __syncthreads();
  const int nw = blockDim.x >> 6;
  double m = XINF;
  for (int j = 0; j < nw; ++j) {
    const double x = sh.red[rb][j];
    m = x < m ? x : m;
  }
  rb ^= 1;
  return m;
}

// Appends the lanes with `pred` to a list counted in shared memory: one
// atomic per wave.  Every lane of the wave must call it.
__device__ __forceinline__ int xappend(int32_t* counter, bool pred) {
  const uint64_t mask = __ballot(pred);
  if (mask == 0) return -1;
  const int lane = threadIdx.x & 63;
  const int leader = __ffsll((unsigned long long)mask) - 1;
  int base = 0;
  if (lane == leader) base = atomicAdd(counter, (int)__popcll(mask));
  base = __shfl(base, leader, 64);
  return pred ? base + (int)__popcll(mask & ((1ull << lane) - 1ull)) : -1;
}

__device__ __forceinline__ int64_t xwave_sum(int64_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Link state of one part, by device link id: residual capacity R, share s,
// unfrozen count n, frozen-this-level count k.  In shared memory (the part's
// links fit the dynamic pool; ids offset by the part's first link) or in
// global memory (the part's slice of the handle's arrays).
template <bool LDS>
struct XLinks {
  double* R;
  double* s;
  int32_t* n;
  int32_t* k;
  int off;
  __device__ __forceinline__ int ix(int l) const { return l - off; }
  __device__ __forceinline__ int add_n(int l, int v) {
    if constexpr (LDS) return atomicAdd(&n[ix(l)], v);
    else return __hip_atomic_fetch_add(&n[ix(l)], v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  }
  __device__ __forceinline__ void add_k(int l, int v) {
    if constexpr (LDS) atomicAdd(&k[ix(l)], v);
    else __hip_atomic_fetch_add(&k[ix(l)], v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  }
  __device__ __forceinline__ int get_n(int l) const {
    if constexpr (LDS) return n[ix(l)];
    else return __hip_atomic_load(&n[ix(l)], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  }
  __device__ __forceinline__ int get_k(int l) const {
    if constexpr (LDS) return k[ix(l)];
    else return __hip_atomic_load(&k[ix(l)], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  }
  __device__ __forceinline__ void set_nk(int l, int nv, int kv) {
    if constexpr (LDS) {
      n[ix(l)] = nv;
      k[ix(l)] = kv;
    } else {
      __hip_atomic_store(&n[ix(l)], nv, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      __hip_atomic_store(&k[ix(l)], kv, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    }
  }
};

constexpr int XLINK_BYTES = 24;  // R, s (f64), n, k (i32)

template <bool LDS>
__device__ __forceinline__ XLinks<LDS> xlinks(const Params& P, const ScenCtl* C, unsigned char* pool) {
  if constexpr (LDS) {
    const int nl = C->l1 - C->l0;
    double* R = reinterpret_cast<double*>(pool);
    double* s = R + nl;
    int32_t* n = reinterpret_cast<int32_t*>(s + nl);
    int32_t* k = n + nl;
    return XLinks<true>{R, s, n, k, C->l0};
  } else {
    return XLinks<false>{P.xR, P.xs, P.xn, P.xk, 0};
  }
}

// Max-min rates of the nu flows listed in U (all of the part), written to
// P.rate.  Work lists: unf0/unf1 (flows), xlive0/xlive1 (links), each used on
// the part's slice.  Returns a status (ST_DONE, ST_BAD_SHARE, ST_ROUNDS).
template <bool LDS>
__device__ int exact_solve(const Params& P, const ScenCtl* C, XLinks<LDS>& lk, XShared& sh, int& rb,
                           const int32_t* U, int nu, int64_t& rounds) {
  const int T = blockDim.x, tid = threadIdx.x;
  const int f0 = C->f0, l0 = C->l0;
  int32_t* unf[2] = {P.unf0 + f0, P.unf1 + f0};
  int32_t* live[2] = {P.xlive0 + l0, P.xlive1 + l0};
  // every link of the part starts the solve with no flow
  for (int l = l0 + tid; l < C->l1; l += T) lk.set_nk(l, 0, 0);
  if (tid == 0) {
    sh.nlive[0] = 0;
    sh.nlive[1] = 0;
    sh.nunf[0] = 0;
    sh.nunf[1] = 0;
  }
  __syncthreads();
  // unfrozen counts; the first flow on a link lists it as live
  for (int b = 0; b < nu; b += T) {
    const int i = b + tid;
    const int f = i < nu ? U[i] : -1;
    const int e0 = f >= 0 ? P.poff[f] : 0, e1 = f >= 0 ? P.poff[f + 1] : 0;
    for (int e = e0; e < e1; ++e) {
      const int l = P.plink[e];
      if (lk.add_n(l, 1) == 0) live[0][atomicAdd(&sh.nlive[0], 1)] = l;
    }
  }
  __syncthreads();
  int nl = sh.nlive[0];
  int lb = 0, ub = 0;
  const int32_t* cur = U;
  double sprev = 0.0;
  bool first = true;
  int status = ST_DONE;
  int64_t fsw = 0, isw = 0;
  int levels = 0;
  while (nu > 0) {
    // every level freezes at least one flow: more levels than the watchdog
    // allows (default: flows + 1) means a fault
    if (levels >= P.max_rounds) {
      status = ST_ROUNDS;
      break;
    }
    ++levels;
    // link pass: apply the last level's freezes, new shares, level minimum
    int32_t* lin = live[lb];
    int32_t* lout = live[lb ^ 1];
    double loc = XINF;
    for (int b = 0; b < nl; b += T) {
      const int i = b + tid;
      bool keep = false;
      int l = 0;
      double sv = XINF;
      if (i < nl) {
        l = lin[i];
        int n = lk.get_n(l);
        double R;
        if (first) {
          R = P.capf[l];
          lk.R[lk.ix(l)] = R;
        } else {
          const int k = lk.get_k(l);
          R = lk.R[lk.ix(l)];
          if (k != 0) {
            const double dec = (double)k * sprev;
            R = R - dec;
            n -= k;
            lk.R[lk.ix(l)] = R;
            lk.set_nk(l, n, 0);
          }
        }
        keep = n > 0;
        if (keep) {
          sv = R / (double)n;
          lk.s[lk.ix(l)] = sv;
        }
      }
      const int slot = xappend(&sh.nlive[lb ^ 1], keep);
      if (keep) lout[slot] = l;
      loc = sv < loc ? sv : loc;
    }
    const double sstar = xblock_min(loc, sh, rb);
    nl = sh.nlive[lb ^ 1];
    if (tid == 0) sh.lsw += nl;  // links whose share this level computed
    if (!(sstar > 0.0) || !(sstar < XINF)) {
      status = ST_BAD_SHARE;
      break;
    }
    first = false;
    rounds += 1;
    const double thr = sstar * XTHR;
    // freezing sweep over the unfrozen flows
    int32_t* uout = unf[ub];
    if (tid == 0) sh.nlive[lb] = 0;  // the next link pass appends there
    for (int b = 0; b < nu; b += T) {
      const int i = b + tid;
      bool keep = false;
      int f = -1;
      if (i < nu) {
        f = cur[i];
        const int e0 = P.poff[f], e1 = P.poff[f + 1];
        bool fz = false;
        for (int e = e0; e < e1; ++e) fz |= lk.s[lk.ix(P.plink[e])] <= thr;
        fsw += 1;
        isw += e1 - e0;
        if (fz) {
          P.rate[f] = sstar;
          for (int e = e0; e < e1; ++e) lk.add_k(P.plink[e], 1);
        } else {
          keep = true;
        }
      }
      const int slot = xappend(&sh.nunf[ub], keep);
      if (keep) uout[slot] = f;
    }
    __syncthreads();
    nu = sh.nunf[ub];
    cur = uout;
    if (tid == 0) sh.nunf[ub ^ 1] = 0;  // the next sweep appends there
    ub ^= 1;
    lb ^= 1;
    sprev = sstar;
  }
  fsw = xwave_sum(fsw);
  isw = xwave_sum(isw);
  if ((tid & 63) == 0) {
    atomicAdd((unsigned long long*)&sh.fsw, (unsigned long long)fsw);
    atomicAdd((unsigned long long*)&sh.isw, (unsigned long long)isw);
  }
  __syncthreads();
  return status;
}

// The event loop of part sc from t = 0, or (P.resume) from where the last
// launch stopped it.  State between launches: the control block (time,
// counts, list sizes, buffer indices) and the per-flow arrays (remaining
// bytes at the part's current time, rate, finish, release, release base,
// predecessor count; active and pending lists).
template <bool LDS>
__device__ void exact_loop(const Params& P, int sc, XShared& sh, unsigned char* pool) {
  ScenCtl* C = &P.ctl[sc];
  XLinks<LDS> lk = xlinks<LDS>(P, C, pool);
  const int T = blockDim.x, tid = threadIdx.x;
  const int f0 = C->f0, cap = C->f1 - C->f0;
  int32_t* act[2] = {P.act0 + f0, P.act1 + f0};
  int32_t* pend[2] = {P.pend0 + f0, P.pend1 + f0};
  int32_t* done[2] = {P.comp0 + f0, P.comp1 + f0};
  double* tau = P.tau0 + f0;
  const bool resume = P.resume && C->started;
  double t = resume ? C->t : 0.0;
  int ab = resume ? C->ab : 0;
  int pb = resume ? C->e : 0;
  int na = resume ? C->nslots : 0;
  int np = resume ? C->npend : C->n_pend0;
  int64_t events = resume ? C->events : 0;
  int64_t solves = resume ? C->solves : 0;
  int64_t rounds = resume ? C->rounds : 0;
  int64_t asw = resume ? C->active_swept : 0;
  int64_t psw = resume ? C->pending_swept : 0;
  const int64_t events0 = events;
  int rb = 0;
  int status = ST_DONE;
  if (tid == 0) {
    sh.fsw = resume ? C->flows_swept : 0;
    sh.isw = resume ? C->incidences_swept : 0;
    sh.lsw = resume ? C->links_swept : 0;
    sh.fault = 0;
    sh.npend[pb] = np;  // releases append after the pending flows
  }
  __syncthreads();
  auto bad = [&](int f) { return (unsigned)(f - f0) >= (unsigned)cap; };
  for (;;) {
    if (na == 0 && np == 0) break;
    if (P.max_events > 0 && events - events0 >= P.max_events) {
      status = ST_STOPPED;
      break;
    }
    // next event: earliest predicted completion or release
    if (tid == 0) {
      sh.nact[ab ^ 1] = 0;
      sh.ndone[0] = 0;
      sh.ndone[1] = 0;
      sh.changed = 0;
    }
    const int32_t* A = act[ab];
    const int32_t* Pd = pend[pb];
    double loc = XINF;
    for (int i = tid; i < na; i += T) {
      const int f = A[i];
      if (bad(f)) { sh.fault = 1; continue; }
      const double tv = t + P.rem[f] / P.rate[f];
      tau[i] = tv;
      loc = tv < loc ? tv : loc;
    }
    for (int i = tid; i < np; i += T) {
      const int f = Pd[i];
      if (bad(f)) { sh.fault = 1; continue; }
      const double rv = P.rel[f];
      loc = rv < loc ? rv : loc;
    }
    const double tn = xblock_min(loc, sh, rb);
    asw += na;
    psw += np;
    if (sh.fault) {
      status = ST_OVERFLOW;
      break;
    }
    if (tn > P.until) {
      status = ST_STOPPED;
      break;
    }
    events += 1;
    const double thr = tn * XTHR;
    const double step = tn - t;
    // completions (finish at tn, plus the path latency) and advance
    int db = 0;
    for (int b = 0; b < na; b += T) {
      const int i = b + tid;
      const bool in = i < na;
      const int f = in ? A[i] : -1;
      bool fin = false;
      if (in) {
        if (tau[i] <= thr) {
          fin = true;
          P.finish[f] = P.lat ? tn + P.lat[f] : tn;
        } else {
          const double moved = P.rate[f] * step;
          P.rem[f] = P.rem[f] - moved;
        }
      }
      const int s1 = xappend(&sh.ndone[db], fin);
      if (fin) done[db][s1] = f;
      const int s2 = xappend(&sh.nact[ab ^ 1], in && !fin);
      if (in && !fin) act[ab ^ 1][s2] = f;
    }
    __syncthreads();
    int nd = sh.ndone[db];
    bool changed = nd > 0;
    na = sh.nact[ab ^ 1];
    ab ^= 1;
    t = tn;
    // releases and arrivals, to a fixpoint
    for (;;) {
      const int32_t* D = done[db];
      // every finished flow raises its dependants' release base ...
      for (int i = tid; i < nd; i += T) {
        const int f = D[i];
        const uint64_t fb = (uint64_t)__double_as_longlong(P.finish[f]);
        for (int e = P.soff[f]; e < P.soff[f + 1]; ++e)
          __hip_atomic_fetch_max((unsigned long long*)&P.base[P.succ[e]], (unsigned long long)fb,
                                 __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      }
      if (tid == 0) sh.npend[pb ^ 1] = 0;
      __syncthreads();
      // ... then counts down their predecessors; the last one releases
      for (int i = tid; i < nd; i += T) {
        const int f = D[i];
        for (int e = P.soff[f]; e < P.soff[f + 1]; ++e) {
          const int g = P.succ[e];
          if (__hip_atomic_fetch_add(&P.cnt[g], -1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) == 1) {
            const double bv = __longlong_as_double((long long)__hip_atomic_load(
                (unsigned long long*)&P.base[g], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP));
            P.rel[g] = P.start[g] + bv;
            pend[pb][atomicAdd(&sh.npend[pb], 1)] = g;
          }
        }
      }
      if (tid == 0) sh.ndone[db ^ 1] = 0;
      __syncthreads();
      np = sh.npend[pb];
      // arrivals at or before t
      const int32_t* Pi = pend[pb];
      int32_t* Po = pend[pb ^ 1];
      for (int b = 0; b < np; b += T) {
        const int i = b + tid;
        const int f = i < np ? Pi[i] : -1;
        bool arrive = false, zero = false;
        double rv = 0.0;
        if (f >= 0) {
          rv = P.rel[f];
          arrive = rv <= t;
          zero = arrive && P.nbytes[f] == 0.0;
        }
        const int s1 = xappend(&sh.npend[pb ^ 1], f >= 0 && !arrive);
        if (f >= 0 && !arrive) Po[s1] = f;
        const int s2 = xappend(&sh.ndone[db ^ 1], zero);
        if (zero) {
          P.finish[f] = rv;
          done[db ^ 1][s2] = f;
        }
        const int s3 = xappend(&sh.nact[ab], arrive && !zero);
        if (arrive && !zero) {
          P.rem[f] = P.nbytes[f];
          act[ab][s3] = f;
          sh.changed = 1;
        }
      }
      __syncthreads();
      np = sh.npend[pb ^ 1];
      pb ^= 1;
      na = sh.nact[ab];
      nd = sh.ndone[db ^ 1];
      db ^= 1;
      changed = changed || sh.changed;
      if (nd == 0) break;
      if (tid == 0) sh.npend[pb] = np;  // the next wave's releases append after the survivors
      __syncthreads();
    }
    // a changed active set is solved again
    if (changed && na > 0) {
      const int rc = exact_solve<LDS>(P, C, lk, sh, rb, act[ab], na, rounds);
      solves += 1;
      if (rc != ST_DONE) {
        status = rc;
        break;
      }
    } else {
      // the counters read above are reset at the top of the next event
      __syncthreads();
    }
  }
  __syncthreads();
  if (tid == 0) {
    C->started = 1;
    C->t = t;
    C->ab = ab;
    C->e = pb;
    C->nslots = na;
    C->npend = np;
    C->holes = 0;
    C->events = events;
    C->launch_events = events - events0;
    C->solves = solves;
    C->rounds = rounds;
    C->flows_swept = sh.fsw;
    C->incidences_swept = sh.isw;
    C->links_swept = sh.lsw;
    C->active_swept = asw;
    C->pending_swept = psw;
    C->status = status;
  }
}

// One rate solve of the C->n_solve flows listed in act0 of part sc.
template <bool LDS>
__device__ void exact_solve_only(const Params& P, int sc, XShared& sh, unsigned char* pool) {
  ScenCtl* C = &P.ctl[sc];
  XLinks<LDS> lk = xlinks<LDS>(P, C, pool);
  if (threadIdx.x == 0) {
    sh.fsw = 0;
    sh.isw = 0;
    sh.lsw = 0;
  }
  __syncthreads();
  int rb = 0;
  int64_t rounds = 0;
  int rc = ST_DONE;
  if (C->n_solve > 0) rc = exact_solve<LDS>(P, C, lk, sh, rb, P.act0 + C->f0, C->n_solve, rounds);
  __syncthreads();
  if (threadIdx.x == 0) {
    C->solves = C->n_solve > 0 ? 1 : 0;
    C->rounds = rounds;
    C->flows_swept = sh.fsw;
    C->incidences_swept = sh.isw;
    C->links_swept = sh.lsw;
    C->status = rc;
  }
}

}  // namespace

// One workgroup per part (a scenario: exact mode keeps one clock per
// scenario).  A part whose link state fits the dynamic shared-memory pool
// keeps it there; the others use their slice of the global link arrays.
__global__ __launch_bounds__(1024) void netsim_exact_kernel(Params P) {
  __shared__ XShared sh;
  extern __shared__ __align__(16) unsigned char xpool[];
  for (int sc = blockIdx.x; sc < P.num_scen; sc += gridDim.x) {
    const ScenCtl* C = &P.ctl[sc];
    const bool lds = (P.debug & DEBUG_EXACT_GLOBAL_LINKS) == 0 &&
                     (int64_t)(C->l1 - C->l0) * XLINK_BYTES <= (int64_t)P.exact_lds_bytes;
    if (P.mode == 0) {
      if (lds) exact_loop<true>(P, sc, sh, xpool);
      else exact_loop<false>(P, sc, sh, xpool);
    } else {
      if (lds) exact_solve_only<true>(P, sc, sh, xpool);
      else exact_solve_only<false>(P, sc, sh, xpool);
    }
    __syncthreads();
  }
}

int exact_link_bytes() { return XLINK_BYTES; }

// ------------------------------------------- allocation-free rate solve
// Scratch of netsim_solve_rates_noalloc: per link R, s (f64), n, k and two
// live lists (i32); per flow the solve list and two unfrozen lists (i32);
// a status block.  The array lives in device memory for the whole process
// (one copy per device); host code reaches it only through the address
// hipGetSymbolAddress returns for the current device.
constexpr int NA_MAX_LINKS = 1 << 16;
constexpr int NA_MAX_FLOWS = 1 << 18;
constexpr size_t NA_LINK_BYTES = (size_t)NA_MAX_LINKS * (8 + 8 + 4 + 4 + 4 + 4);
constexpr size_t NA_FLOW_BYTES = (size_t)NA_MAX_FLOWS * (4 + 4 + 4);
constexpr size_t NA_HEAD_BYTES = 256;  // kept free (alignment of what follows)
constexpr int ST_BAD_INPUT = -100;
constexpr size_t NA_SCRATCH_BYTES = NA_HEAD_BYTES + NA_LINK_BYTES + NA_FLOW_BYTES;

// One workgroup: validates the caller's CSR (offsets from 0, non-decreasing;
// every path non-empty, its link ids in range and distinct; capacities
// finite and > 0), then runs the exact solve over all F flows with link
// state in the scratch array.
__global__ __launch_bounds__(1024) void netsim_noalloc_solve_kernel(const double* cap, int L,
                                                                    const int32_t* poff,
                                                                    const int32_t* plink, int F,
                                                                    double* rates, int64_t* status_out,
                                                                    unsigned char* ws, int max_rounds) {
  __shared__ XShared sh;
  __shared__ int bad;
  double* R = reinterpret_cast<double*>(ws + NA_HEAD_BYTES);
  double* S = R + NA_MAX_LINKS;
  int32_t* n = reinterpret_cast<int32_t*>(S + NA_MAX_LINKS);
  int32_t* k = n + NA_MAX_LINKS;
  int32_t* live0 = k + NA_MAX_LINKS;
  int32_t* live1 = live0 + NA_MAX_LINKS;
  int32_t* U = live1 + NA_MAX_LINKS;
  int32_t* unf0 = U + NA_MAX_FLOWS;
  int32_t* unf1 = unf0 + NA_MAX_FLOWS;
  const int T = blockDim.x, tid = threadIdx.x;
  if (tid == 0) bad = INT32_MAX;
  __syncthreads();
  if (tid == 0 && F > 0 && poff[0] != 0) atomicMin(&bad, 0);
  for (int f = tid; f < F; f += T) {
    const int e0 = poff[f], e1 = poff[f + 1];
    bool ok = e1 > e0;
    for (int e = e0; ok && e < e1; ++e) {
      const int l = plink[e];
      ok = l >= 0 && l < L;
      for (int q = e0; ok && q < e; ++q) ok = plink[q] != l;
    }
    if (!ok) atomicMin(&bad, f);
    U[f] = f;
  }
  for (int l = tid; l < L; l += T) {
    const double c = cap[l];
    if (!(c > 0.0) || !(c < XINF)) atomicMin(&bad, F + l);
  }
  __syncthreads();
  int status = ST_BAD_INPUT;
  int64_t levels = 0;
  if (bad == INT32_MAX) {
    Params P{};
    P.poff = poff;
    P.plink = plink;
    P.capf = cap;
    P.rate = rates;
    P.xR = R;
    P.xs = S;
    P.xn = n;
    P.xk = k;
    P.xlive0 = live0;
    P.xlive1 = live1;
    P.unf0 = unf0;
    P.unf1 = unf1;
    P.max_rounds = max_rounds;
    ScenCtl C{};
    C.f0 = 0;
    C.f1 = F;
    C.l0 = 0;
    C.l1 = L;
    XLinks<false> lk{R, S, n, k, 0};
    if (tid == 0) {
      sh.fsw = 0;
      sh.isw = 0;
      sh.lsw = 0;
    }
    __syncthreads();
    int rb = 0;
    status = F > 0 ? exact_solve<false>(P, &C, lk, sh, rb, U, F, levels) : ST_DONE;
  }
  if (tid == 0) {
    // the C status codes of include/netsim.h
    status_out[0] = status == ST_DONE ? 0 : status == ST_BAD_INPUT ? -1 : status == ST_ROUNDS ? -5 : -3;
    status_out[1] = status == ST_BAD_INPUT ? (int64_t)bad : levels;
  }
}

// The scratch array's device address on each device, found once per device.
unsigned char* g_scratch_ptr[64];
std::mutex g_scratch_mu;

hipError_t launch_exact(const Params& p, int blocks, int threads, hipStream_t s) {
  if (p.exact_lds_bytes > 0) {
    hipError_t e = hipFuncSetAttribute((const void*)netsim_exact_kernel,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, p.exact_lds_bytes);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(netsim_exact_kernel, dim3(blocks), dim3(threads), (size_t)p.exact_lds_bytes, s, p);
  return hipGetLastError();
}

}  // namespace netsim_dev

// Scratch of the allocation-free entry point (see NA_* above).
static __device__ __align__(256) unsigned char scratch[netsim_dev::NA_SCRATCH_BYTES];

extern "C" netsim_status netsim_solve_rates_noalloc(int32_t device, int32_t num_links,
                                                    const double* d_capacity_Bps, int32_t num_flows,
                                                    const int32_t* d_path_off,
                                                    const int32_t* d_path_link, double* d_rates,
                                                    int64_t* d_status, void* hip_stream) {
  using namespace netsim_dev;
  auto fail = [](netsim_status code, const std::string& m) {
    netsim_host::set_thread_error(m.c_str());
    return code;
  };
  if (device < 0 || device >= 64) return fail(NETSIM_E_INVALID, "solve_rates_noalloc: bad device");
  if (num_links < 0 || num_flows < 0) return fail(NETSIM_E_INVALID, "solve_rates_noalloc: negative size");
  if (num_links > NA_MAX_LINKS || num_flows > NA_MAX_FLOWS)
    return fail(NETSIM_E_LIMIT, "solve_rates_noalloc: more than " + std::to_string(NA_MAX_LINKS) +
                                    " links or " + std::to_string(NA_MAX_FLOWS) + " flows");
  if (!d_status || !d_path_off || (num_links > 0 && !d_capacity_Bps) ||
      (num_flows > 0 && (!d_path_link || !d_rates)))
    return fail(NETSIM_E_INVALID, "solve_rates_noalloc: NULL array");
  hipError_t he = hipSetDevice(device);
  if (he != hipSuccess) return fail(NETSIM_E_DEVICE, std::string("hipSetDevice: ") + hipGetErrorString(he));
  unsigned char* ws = nullptr;
  {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[device]) {
      void* p = nullptr;
      he = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (he != hipSuccess || !p)
        return fail(NETSIM_E_DEVICE, std::string("hipGetSymbolAddress: ") + hipGetErrorString(he));
      g_scratch_ptr[device] = static_cast<unsigned char*>(p);
    }
    ws = g_scratch_ptr[device];
  }
  hipLaunchKernelGGL(netsim_noalloc_solve_kernel, dim3(1), dim3(1024), 0,
                     static_cast<hipStream_t>(hip_stream), d_capacity_Bps, num_links, d_path_off,
                     d_path_link, num_flows, d_rates, d_status, ws, num_flows + 1);
  he = hipGetLastError();
  if (he != hipSuccess) return fail(NETSIM_E_DEVICE, std::string("solve_rates_noalloc: ") + hipGetErrorString(he));
  return NETSIM_OK;
}
