// Device-resident event loop and max-min rate solver for gfx950.
//
// Model (paper Section 4.1, netsim; Section 4.2, time rollback and the
// iterative water-filling solve): the active flows share link bandwidth
// max-min fairly; rates are constant between events; the loop jumps to the
// next completion or release, settles completions, releases dependants and
// re-solves.
//
// The rate solve finds the max-min allocation by rounds of "local minimum"
// freezing instead of one bottleneck per iteration.  With residual capacity
// R_l, unfrozen count n_l and share s_l = R_l / n_l:
//   phase B: every unfrozen flow f computes m_f = min over its path of s_l,
//            and marks each link of its path whose share exceeds m_f*THR
//            (THR = 1 + 1e-12) as blocked for this round;
//   phase C: a flow crossing at least one unblocked link is frozen at
//            r_f = m_f and its links lose r_f and one flow.
// An unblocked link's share is within THR of the smallest share seen by
// every flow through it, i.e. it is a bottleneck of its neighbourhood.
// Shares never decrease during progressive filling, so such a link is
// frozen at its current share by the one-bottleneck-at-a-time procedure
// too: both give the same (unique) max-min allocation in exact arithmetic,
// but this one needs as many rounds as the longest chain of bottleneck
// dependencies rather than one iteration per distinct share level.
// Residual capacities are kept in 64-bit fixed point (a power-of-two
// scale), so the per-link sums are order independent and every run is
// deterministic.
//
// The same code runs over a "group" of threads: one workgroup per scenario
// (BlockG, workgroup barriers) or the whole grid on one scenario at a time
// (GridG, an atomic grid barrier with a time-out).  Every loop exit depends
// only on values read after a group barrier, so all waves leave together.
#include "device.h"

#include <math.h>

namespace netsim_dev {

namespace {

constexpr double THR = 1.000000000001;
constexpr double INF = __builtin_huge_val();
constexpr int FAST_DEG = 8;
constexpr uint64_t BARRIER_TIMEOUT_TICKS = 1000000000ull;  // 10 s at 100 MHz

__device__ __forceinline__ double wave_min(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    double w = __shfl_xor(v, o, 64);
    v = w < v ? w : v;
  }
  return v;
}

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }

// ------------------------------------------------------------------ groups
struct BlockG {
  double* lds;
  __device__ int tid() const { return threadIdx.x; }
  __device__ int nthr() const { return blockDim.x; }
  __device__ bool aborted() const { return false; }
  __device__ void sync() { __syncthreads(); }
  __device__ double min_all(double v) {
    v = wave_min(v);
    const int w = threadIdx.x >> 6;
    if (lane_id() == 0) lds[w] = v;
    __syncthreads();
    if (threadIdx.x < 64) {
      double x = threadIdx.x < (blockDim.x >> 6) ? lds[threadIdx.x] : INF;
      x = wave_min(x);
      if (threadIdx.x == 0) lds[16] = x;
    }
    __syncthreads();
    return lds[16];
  }
  template <class T>
  __device__ T add(T* p, T v) {
    return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  }
  template <class T>
  __device__ T load(const T* p) {
    return __hip_atomic_load(const_cast<T*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  }
  template <class T>
  __device__ void store(T* p, T v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  }
};

struct GridG {
  double* lds;
  int* flag;      // shared: abort state as seen by this block's thread 0
  uint32_t* bar;
  uint64_t* slots;
  uint32_t gen;
  uint32_t nred;
  bool ab;        // block-uniform copy of *flag, refreshed at every barrier
  __device__ int tid() const { return blockIdx.x * blockDim.x + threadIdx.x; }
  __device__ int nthr() const { return gridDim.x * blockDim.x; }
  __device__ bool aborted() const { return ab; }
  // Generation barrier.  The last block to arrive resets the arrival count
  // and publishes the next generation (release); the others wait for it
  // (acquire).  A block waiting longer than BARRIER_TIMEOUT_TICKS raises the
  // abort flag; a waiting block that sees the flag stops waiting.  Thread 0
  // passes the flag to its block through shared memory, so every decision
  // taken on it is uniform inside the block and all blocks leave their loops.
  __device__ void sync() {
    __syncthreads();
    if (threadIdx.x == 0) {
      uint32_t a = __hip_atomic_load(&bar[2], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (a == 0) {
        const uint32_t g = gen;
        const uint32_t prev =
            __hip_atomic_fetch_add(&bar[0], 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
        if (prev == gridDim.x - 1) {
          __hip_atomic_store(&bar[0], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          __hip_atomic_store(&bar[1], g + 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
        } else {
          const uint64_t t0 = wall_clock64();
          while (__hip_atomic_load(&bar[1], __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) == g) {
            __builtin_amdgcn_s_sleep(1);
            if (__hip_atomic_load(&bar[2], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0) break;
            if (wall_clock64() - t0 > BARRIER_TIMEOUT_TICKS) {
              __hip_atomic_store(&bar[2], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
              break;
            }
          }
        }
        a = __hip_atomic_load(&bar[2], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      *flag = (int)a;
    }
    gen += 1;
    __syncthreads();
    ab = *flag != 0;
  }
  // Grid-wide minimum of non-negative doubles: block minimum, then an
  // atomic min on the bit pattern (ordered like the values) in one of four
  // rotating slots; block 0 resets the slot used three reductions later.
  __device__ double min_all(double v) {
    v = wave_min(v);
    const int w = threadIdx.x >> 6;
    if (lane_id() == 0) lds[w] = v;
    __syncthreads();
    const uint32_t k = nred++;
    if (threadIdx.x < 64) {
      double x = threadIdx.x < (blockDim.x >> 6) ? lds[threadIdx.x] : INF;
      x = wave_min(x);
      if (threadIdx.x == 0) {
        __hip_atomic_fetch_min(&slots[k & 3], (uint64_t)__double_as_longlong(x), __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
        if (blockIdx.x == 0)
          __hip_atomic_store(&slots[(k + 1) & 3], (uint64_t)__double_as_longlong(INF),
                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    sync();
    return __longlong_as_double(
        (long long)__hip_atomic_load(&slots[k & 3], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
  }
  template <class T>
  __device__ T add(T* p, T v) {
    return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  template <class T>
  __device__ T load(const T* p) {
    return __hip_atomic_load(const_cast<T*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  template <class T>
  __device__ void store(T* p, T v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
};

// Appends the lanes with `pred` to a list: one atomic per wave.  Must be
// reached by every lane of the wave.  Returns the slot (or -1 without pred).
template <class G>
__device__ __forceinline__ int wave_append(G& g, int32_t* counter, bool pred) {
  const uint64_t mask = __ballot(pred);
  if (mask == 0) return -1;
  const int lane = lane_id();
  const int leader = __ffsll((unsigned long long)mask) - 1;
  int base = 0;
  if (lane == leader) base = g.add(counter, (int32_t)__popcll(mask));
  base = __shfl(base, leader, 64);
  return pred ? base + (int)__popcll(mask & ((1ull << lane) - 1ull)) : -1;
}

__device__ __forceinline__ double share(const Params& P, int l) {
  return ((double)P.Rres[l] / (double)P.nres[l]) * P.inv_scale;
}

// ------------------------------------------------------------- rate solve
// Max-min rates of the n0 flows listed in list0 (all active).  Link state is
// initialised from nact.  Returns 0 or a negative status.
template <class G>
__device__ int solve(G& g, const Params& P, ScenCtl* C, const int32_t* list0, int n0,
                     int32_t* unf_a, int32_t* unf_b, int cap, int64_t& rounds, int64_t& fsw,
                     int64_t& isw) {
  const int T = g.nthr();
  const int tid = g.tid();
  const int w0 = tid - lane_id();
  for (int l = C->l0 + tid; l < C->l1; l += T) {
    P.Rres[l] = P.R0[l];
    P.nres[l] = P.nact[l];
    P.blocked0[l] = 0;
    P.blocked1[l] = 0;
  }
  if (tid == 0) {
    g.store(&C->cnt_unf[0], 0);
    g.store(&C->cnt_unf[1], 0);
  }
  g.sync();
  const int32_t* in = list0;
  int n = n0;
  int r = 0;
  int bad = 0;
  for (;;) {
    uint8_t* bl = (r & 1) ? P.blocked1 : P.blocked0;
    uint8_t* bl_next = (r & 1) ? P.blocked0 : P.blocked1;
    int32_t* out = (r & 1) ? unf_b : unf_a;
    int32_t* out_cnt = &C->cnt_unf[r & 1];
    if (tid == 0 && r > 0) g.store(out_cnt, 0);
    // phase B: smallest share on each path; block links above it
    for (int i0 = w0; i0 < n; i0 += T) {
      const int i = i0 + lane_id();
      if (i < n) {
        const int f = in[i];
        const int e0 = P.poff[f], e1 = P.poff[f + 1];
        const int deg = e1 - e0;
        isw += deg;
        double m = INF;
        if (deg <= FAST_DEG) {
          double sv[FAST_DEG];
          int lv[FAST_DEG];
#pragma unroll
          for (int k = 0; k < FAST_DEG; ++k) {
            if (k < deg) {
              lv[k] = P.plink[e0 + k];
              sv[k] = share(P, lv[k]);
              m = sv[k] < m ? sv[k] : m;
            }
          }
          const double thr = m * THR;
#pragma unroll
          for (int k = 0; k < FAST_DEG; ++k)
            if (k < deg && sv[k] > thr) bl[lv[k]] = 1;
        } else {
          for (int e = e0; e < e1; ++e) {
            const double s = share(P, P.plink[e]);
            m = s < m ? s : m;
          }
          const double thr = m * THR;
          for (int e = e0; e < e1; ++e)
            if (share(P, P.plink[e]) > thr) bl[P.plink[e]] = 1;
        }
        if (!(m > 0.0) || !(m < INF)) bad = 1;
        P.mf[f] = m;
      }
    }
    g.sync();
    // phase C: freeze flows that cross an unblocked link
    for (int i0 = w0; i0 < n; i0 += T) {
      const int i = i0 + lane_id();
      bool keep = false;
      int f = -1;
      if (i < n) {
        f = in[i];
        const int e0 = P.poff[f], e1 = P.poff[f + 1];
        bool frozen = false;
        for (int e = e0; e < e1; ++e) frozen |= (bl[P.plink[e]] == 0);
        if (frozen) {
          const double m = P.mf[f];
          P.rate[f] = m;
          const int64_t q = (int64_t)__builtin_rint(m * P.scale);
          for (int e = e0; e < e1; ++e) {
            const int l = P.plink[e];
            g.add(&P.Rres[l], -q);
            g.add(&P.nres[l], -1);
          }
        } else {
          keep = true;
        }
      }
      const int slot = wave_append(g, out_cnt, keep);
      if (keep) {
        if (slot < cap) out[slot] = f;
        else bad = 2;
      }
    }
    for (int l = C->l0 + tid; l < C->l1; l += T) bl_next[l] = 0;
    if (bad) g.store(&C->fault_info, bad);
    g.sync();
    rounds += 1;
    fsw += n;
    if (g.aborted()) return ST_BARRIER;
    const int nout = g.load(out_cnt);
    if (g.load(&C->fault_info) != 0) return g.load(&C->fault_info) == 2 ? ST_OVERFLOW : ST_BAD_SHARE;
    if (nout == 0) return 0;
    if (nout >= n) return ST_BAD_SHARE;  // a round must freeze something
    if (++r > P.max_rounds) return ST_ROUNDS;
    in = out;
    n = nout;
  }
}

// ------------------------------------------------------------- event loop
template <class G>
__device__ void event_loop(G& g, const Params& P, const int sc) {
  ScenCtl* C = &P.ctl[sc];
  const int f0 = C->f0;
  const int cap = C->f1 - C->f0;
  int32_t* act[2] = {P.act0 + f0, P.act1 + f0};
  int32_t* pend[2] = {P.pend0 + f0, P.pend1 + f0};
  int32_t* comp[3] = {P.comp0 + f0, P.comp1 + f0, P.comp2 + f0};
  int32_t* unf_a = P.unf0 + f0;
  int32_t* unf_b = P.unf1 + f0;
  const int T = g.nthr();
  const int tid = g.tid();
  const int w0 = tid - lane_id();
  double t = 0.0;
  int64_t events = 0, solves = 0, rounds = 0, fsw = 0, isw = 0, asw = 0, psw = 0;
  int nAct = 0;
  int nPend = C->n_pend0;
  int e = 0;  // event index: lists act[e&1], pend[e&1] are this event's input
  int q = 0;  // completion-list phase index (three rotating lists)
  int status = ST_DONE;
  for (;;) {
    const int ib = e & 1, ob = ib ^ 1;
    const int32_t* actIn = act[ib];
    int32_t* actOut = act[ob];
    const int32_t* pendIn = pend[ib];
    int32_t* pendOut = pend[ob];
    if (tid == 0) {
      g.store(&C->cnt_act[ob], 0);
      g.store(&C->cnt_pend[ob], 0);
      g.store(&C->changed[ib], 0);
    }
    // next event time: earliest completion or release
    double loc = INF;
    for (int i = tid; i < nAct; i += T) {
      const int f = actIn[i];
      const double dt = P.rem[f] / P.rate[f];
      const double tau = t + dt;
      loc = tau < loc ? tau : loc;
    }
    for (int i = tid; i < nPend; i += T) {
      const double rl = P.rel[pendIn[i]];
      loc = rl < loc ? rl : loc;
    }
    asw += nAct;
    psw += nPend;
    const double tn = g.min_all(loc);
    if (g.aborted()) { status = ST_BARRIER; break; }
    if (!(tn < INF)) break;
    if ((P.max_events > 0 && events >= P.max_events) || tn > P.until) {
      status = ST_STOPPED;
      break;
    }
    events += 1;
    const double thr = tn * THR;
    const double step = tn - t;
    int32_t* compOut = comp[q % 3];
    int32_t* compCnt = &C->cnt_comp[q % 3];
    if (tid == 0) g.store(&C->cnt_comp[(q + 1) % 3], 0);
    int err = 0;
    // completions and advance
    for (int i0 = w0; i0 < nAct; i0 += T) {
      const int i = i0 + lane_id();
      bool done = false, keep = false;
      int f = -1;
      if (i < nAct) {
        f = actIn[i];
        const double dt = P.rem[f] / P.rate[f];
        const double tau = t + dt;
        if (tau <= thr) {
          done = true;
          P.finish[f] = tn;
          for (int k = P.poff[f]; k < P.poff[f + 1]; ++k) g.add(&P.nact[P.plink[k]], -1);
        } else {
          keep = true;
          const double moved = P.rate[f] * step;
          P.rem[f] = P.rem[f] - moved;
        }
      }
      const int sd = wave_append(g, compCnt, done);
      const int sk = wave_append(g, &C->cnt_act[ob], keep);
      if (done) { if (sd < cap) compOut[sd] = f; else err = 1; }
      if (keep) { if (sk < cap) actOut[sk] = f; else err = 1; }
      if (done) g.store(&C->changed[ib], 1);
    }
    // releases due now
    for (int i0 = w0; i0 < nPend; i0 += T) {
      const int i = i0 + lane_id();
      bool zero = false, start = false, keep = false;
      int f = -1;
      if (i < nPend) {
        f = pendIn[i];
        const double rl = P.rel[f];
        if (rl <= tn) {
          if (P.nbytes[f] == 0.0) {
            zero = true;
            P.finish[f] = rl;
          } else {
            start = true;
            P.rem[f] = P.nbytes[f];
            for (int k = P.poff[f]; k < P.poff[f + 1]; ++k) g.add(&P.nact[P.plink[k]], 1);
          }
        } else {
          keep = true;
        }
      }
      const int sz = wave_append(g, compCnt, zero);
      const int ss = wave_append(g, &C->cnt_act[ob], start);
      const int sk = wave_append(g, &C->cnt_pend[ob], keep);
      if (zero) { if (sz < cap) compOut[sz] = f; else err = 1; }
      if (start) { if (ss < cap) actOut[ss] = f; else err = 1; g.store(&C->changed[ib], 1); }
      if (keep) { if (sk < cap) pendOut[sk] = f; else err = 1; }
    }
    if (err) g.store(&C->fault_info, 2);
    g.sync();
    t = tn;
    q += 1;
    // dependants of finished flows, to a fixpoint through zero-byte flows
    int nc = g.load(&C->cnt_comp[(q - 1) % 3]);
    while (nc > 0) {
      const int32_t* cin = comp[(q - 1) % 3];
      int32_t* cout = comp[q % 3];
      int32_t* coutCnt = &C->cnt_comp[q % 3];
      if (tid == 0) g.store(&C->cnt_comp[(q + 1) % 3], 0);
      for (int i = tid; i < nc; i += T) {
        const int f = cin[i];
        for (int k = P.soff[f]; k < P.soff[f + 1]; ++k) {
          const int h = P.succ[k];
          if (g.add(&P.cnt[h], -1) != 1) continue;
          const double rl = P.start[h] + t;
          if (rl <= t) {
            if (P.nbytes[h] == 0.0) {
              P.finish[h] = rl;
              const int s = g.add(coutCnt, 1);
              if (s < cap) cout[s] = h; else err = 1;
            } else {
              P.rem[h] = P.nbytes[h];
              for (int j = P.poff[h]; j < P.poff[h + 1]; ++j) g.add(&P.nact[P.plink[j]], 1);
              const int s = g.add(&C->cnt_act[ob], 1);
              if (s < cap) actOut[s] = h; else err = 1;
              g.store(&C->changed[ib], 1);
            }
          } else {
            P.rel[h] = rl;
            const int s = g.add(&C->cnt_pend[ob], 1);
            if (s < cap) pendOut[s] = h; else err = 1;
          }
        }
      }
      if (err) g.store(&C->fault_info, 2);
      g.sync();
      q += 1;
      nc = g.load(&C->cnt_comp[(q - 1) % 3]);
    }
    if (g.aborted()) { status = ST_BARRIER; break; }
    if (g.load(&C->fault_info) != 0) { status = ST_OVERFLOW; break; }
    const int nNew = g.load(&C->cnt_act[ob]);
    const int pNew = g.load(&C->cnt_pend[ob]);
    if (g.load(&C->changed[ib]) && nNew > 0) {
      const int rc = solve(g, P, C, actOut, nNew, unf_a, unf_b, cap, rounds, fsw, isw);
      solves += 1;
      if (rc != 0) { status = rc; break; }
    }
    nAct = nNew;
    nPend = pNew;
    e += 1;
  }
  g.add(&C->incidences_swept, isw);
  if (tid == 0) {
    C->t = t;
    C->events = events;
    C->solves = solves;
    C->rounds = rounds;
    C->flows_swept = fsw;
    C->active_swept = asw;
    C->pending_swept = psw;
    C->status = status;
  }
}

template <class G>
__device__ void solve_only(G& g, const Params& P, const int sc) {
  ScenCtl* C = &P.ctl[sc];
  const int f0 = C->f0;
  int64_t rounds = 0, fsw = 0, isw = 0;
  int rc = 0;
  if (C->n_solve > 0)
    rc = solve(g, P, C, P.act0 + f0, C->n_solve, P.unf0 + f0, P.unf1 + f0, C->f1 - f0, rounds,
               fsw, isw);
  g.add(&C->incidences_swept, isw);
  if (g.tid() == 0) {
    C->solves = C->n_solve > 0 ? 1 : 0;
    C->rounds = rounds;
    C->flows_swept = fsw;
    C->status = rc;
  }
}

}  // namespace

__global__ __launch_bounds__(1024) void netsim_block_kernel(Params P) {
  __shared__ double lds[32];
  BlockG g{lds};
  for (int sc = blockIdx.x; sc < P.num_scen; sc += gridDim.x) {
    if (P.mode == 0) event_loop(g, P, sc);
    else solve_only(g, P, sc);
    __syncthreads();
  }
}

__global__ __launch_bounds__(1024) void netsim_grid_kernel(Params P) {
  __shared__ double lds[32];
  __shared__ int flag;
  GridG g{lds, &flag, P.bar, P.slots, 0u, 0u, false};
  for (int sc = 0; sc < P.num_scen; ++sc) {
    if (P.mode == 0) event_loop(g, P, sc);
    else solve_only(g, P, sc);
    g.sync();
  }
}

hipError_t launch_block(const Params& p, int blocks, int threads, hipStream_t s) {
  hipLaunchKernelGGL(netsim_block_kernel, dim3(blocks), dim3(threads), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_grid(const Params& p, int blocks, int threads, hipStream_t s) {
  Params copy = p;
  void* args[] = {&copy};
  return hipLaunchCooperativeKernel((const void*)netsim_grid_kernel, dim3(blocks), dim3(threads),
                                    args, 0, s);
}

hipError_t grid_capacity(int device, int threads, int* blocks) {
  int per_cu = 0;
  hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, netsim_grid_kernel, threads, 0);
  if (e != hipSuccess) return e;
  hipDeviceProp_t prop;
  e = hipGetDeviceProperties(&prop, device);
  if (e != hipSuccess) return e;
  *blocks = per_cu * prop.multiProcessorCount;
  return hipSuccess;
}

}  // namespace netsim_dev
