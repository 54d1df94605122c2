// Device-resident event loop and max-min rate solver for gfx950.
//
// Model (paper Section 4.1, netsim; Section 4.2, time rollback and the
// water-filling rate solve): the active flows share link bandwidth
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
constexpr int FAST_DEG = 6;
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
  int* ldsi;
  __device__ int tid() const { return threadIdx.x; }
  __device__ int block_base() const { return 0; }
  __device__ int nblocks() const { return 1; }
  __device__ int block_id() const { return 0; }
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
  __device__ void amin(uint64_t* p, uint64_t v) {
    __hip_atomic_fetch_min(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  }
};

// Barrier words (uint32 indices into Params::bar, 64-byte lines apart):
constexpr int BAR_COUNT = 0, BAR_GEN = 1, BAR_ABORT = 16, BAR_REG = 32, BAR_REG_GEN = 33;
constexpr int BAR_XCD = 64;        // XCD x: arrivals at 64 + 32x, generation at 64 + 32x + 16
constexpr int BAR_XCD_BLOCKS = 640;  // blocks resident on XCD x
constexpr int BAR_WORDS = 1024;

__device__ __forceinline__ unsigned xcc_id() {
  return __builtin_amdgcn_s_getreg(6164) & 15u;  // hwreg(HW_REG_XCC_ID, 0, 4)
}

struct GridG {
  double* lds;
  int* ldsi;
  int* flag;      // shared: abort state as seen by this block's thread 0
  uint32_t* bar;
  uint64_t* slots;
  uint32_t gen;
  uint32_t nred;
  bool ab;        // block-uniform copy of *flag, refreshed at every barrier
  uint32_t xcc, mine, nx;  // this block's XCD, blocks on it, XCDs in use
  __device__ int tid() const { return blockIdx.x * blockDim.x + threadIdx.x; }
  __device__ int block_base() const { return blockIdx.x * blockDim.x; }
  __device__ int nblocks() const { return gridDim.x; }
  __device__ int block_id() const { return blockIdx.x; }
  __device__ int nthr() const { return gridDim.x * blockDim.x; }
  __device__ bool aborted() const { return ab; }

  // Waits (thread 0 only) until *p != g; gives up on the abort flag or after
  // BARRIER_TIMEOUT_TICKS, raising the flag.  Returns false if it gave up.
  __device__ __forceinline__ bool wait_change(uint32_t* p, uint32_t g) {
    const uint64_t t0 = wall_clock64();
    while (__hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == g) {
      __builtin_amdgcn_s_sleep(1);
      if (__hip_atomic_load(&bar[BAR_ABORT], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0)
        return false;
      if (wall_clock64() - t0 > BARRIER_TIMEOUT_TICKS) {
        __hip_atomic_store(&bar[BAR_ABORT], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return false;
      }
    }
    return true;
  }

  // Once per launch: every block counts itself on its XCD, then one flat
  // barrier, after which each block knows how many blocks share its XCD.
  __device__ __forceinline__ void init() {
    __shared__ uint32_t s_mine, s_nx;
    if (threadIdx.x == 0) {
      const uint32_t x = xcc_id();
      __hip_atomic_fetch_add(&bar[BAR_XCD_BLOCKS + x], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const uint32_t prev =
          __hip_atomic_fetch_add(&bar[BAR_REG], 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
      if (prev == gridDim.x - 1) {
        __hip_atomic_store(&bar[BAR_REG_GEN], 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
      } else {
        wait_change(&bar[BAR_REG_GEN], 0u);
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
      }
      uint32_t n = 0;
      for (int k = 0; k < 16; ++k)
        n += __hip_atomic_load(&bar[BAR_XCD_BLOCKS + k], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) > 0;
      s_mine = __hip_atomic_load(&bar[BAR_XCD_BLOCKS + x], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      s_nx = n;
      *flag = (int)__hip_atomic_load(&bar[BAR_ABORT], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
    xcc = xcc_id();
    mine = s_mine;
    nx = s_nx;
    ab = *flag != 0;
    __syncthreads();
  }

  // Two-level barrier.  The blocks of one XCD share its L2: the last of them
  // to arrive writes that L2 back once (release) and arrives at the global
  // count; the last XCD to arrive publishes the next generation.  Every block
  // then acquires (invalidating its L1 and the XCD's L2) before going on.
  // Writing an L2 back once per XCD instead of once per block is what makes
  // this cheaper than a flat barrier.  A block waiting longer than
  // BARRIER_TIMEOUT_TICKS raises the abort flag; thread 0 passes the flag to
  // its block through shared memory, so decisions on it are block-uniform.
  __device__ __forceinline__ void sync() {
    __syncthreads();
    if (threadIdx.x == 0) {
      uint32_t a = __hip_atomic_load(&bar[BAR_ABORT], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (a == 0) {
        uint32_t* xc = &bar[BAR_XCD + 32 * xcc];
        uint32_t* xg = &bar[BAR_XCD + 32 * xcc + 16];
        const uint32_t g = gen;
        const uint32_t prev = __hip_atomic_fetch_add(xc, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (prev == mine - 1) {
          __hip_atomic_store(xc, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
          const uint32_t gp =
              __hip_atomic_fetch_add(&bar[BAR_COUNT], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          if (gp == nx - 1) {
            __hip_atomic_store(&bar[BAR_COUNT], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(&bar[BAR_GEN], g + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          } else {
            wait_change(&bar[BAR_GEN], g);
          }
          __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
          __hip_atomic_store(xg, g + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        } else {
          wait_change(xg, g);
          __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        }
        a = __hip_atomic_load(&bar[BAR_ABORT], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
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
  __device__ __forceinline__ double min_all(double v) {
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
  __device__ void amin(uint64_t* p, uint64_t v) {
    __hip_atomic_fetch_min(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
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

// Appends to K lists at once with one atomic per list per workgroup: wave
// ballots, per-wave counts in shared memory, a prefix over the waves and a
// single fetch-add on each list counter.  Every thread of the workgroup must
// call it (loops that use it run the same trip count in the whole block).
template <int K, class G>
__device__ __forceinline__ void block_append(G& g, int32_t* const* counters, const bool* pred,
                                             int* slot) {
  int* sh = g.ldsi;  // [K*16] per-wave counts (K <= 4), [96 + k] list bases
  const int lane = lane_id(), w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  uint64_t mask[K];
#pragma unroll
  for (int k = 0; k < K; ++k) {
    mask[k] = __ballot(pred[k]);
    if (lane == 0) sh[k * 16 + w] = (int)__popcll(mask[k]);
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < K; ++k) {
    if ((int)threadIdx.x == k) {
      int total = 0;
      for (int j = 0; j < nw; ++j) {
        const int c = sh[k * 16 + j];
        sh[k * 16 + j] = total;
        total += c;
      }
      sh[96 + k] = total ? g.add(counters[k], (int32_t)total) : 0;
    }
  }
  __syncthreads();
  const uint64_t below = (1ull << lane) - 1ull;
#pragma unroll
  for (int k = 0; k < K; ++k)
    slot[k] = pred[k] ? sh[96 + k] + sh[k * 16 + w] + (int)__popcll(mask[k] & below) : -1;
  __syncthreads();
}

// Per-phase wall-clock accounting by the group's first thread, kept in
// shared memory (acc[0..8) and the last reading in acc[8]).
struct Clock {
  bool on;
  uint64_t* acc;
  __device__ Clock(bool o, uint64_t* a) : on(o), acc(a) {
    if (on) {
      for (int k = 0; k < 8; ++k) acc[k] = 0;
      acc[8] = wall_clock64();
    }
  }
  __device__ __forceinline__ void lap(int k) {
    if (on) {
      const uint64_t now = wall_clock64();
      acc[k] += now - acc[8];
      acc[8] = now;
    }
  }
};

// A flow id read from a work list must lie in the scenario's range.
__device__ __forceinline__ bool in_range(int f, int f0, int cap) {
  return (unsigned)(f - f0) < (unsigned)cap;
}

// ------------------------------------------------------------ link state
// Per link: residual capacity R (fixed point), unfrozen flows n, active
// flows nact and two alternating "blocked" flags.  Two homes for it, with
// one interface taking device link ids:
//   LinksGlobal - global memory; any group (the whole grid, or a workgroup
//                 on a part too large for shared memory);
//   LinksShared - the shared memory of the one workgroup running a part
//                 whose links fit there; atomics stay inside the CU.
// Blocked flags of one round, indexed by device link id.
struct Flags {
  uint8_t* p;
  int off;
  __device__ uint8_t& operator[](int l) const { return p[l - off]; }
};

struct LinksGlobal {
  int64_t* lst;      // [2L] (R, n) pairs: one 16-byte load per link
  int32_t* nact;
  uint8_t* bl0;
  uint8_t* bl1;
  double inv;
  __device__ double share(int l) const {
    const longlong2 v = *reinterpret_cast<const longlong2*>(lst + 2 * l);
    return ((double)v.x / (double)v.y) * inv;
  }
  __device__ void set(int l, int64_t R, int64_t n) {
    lst[2 * l] = R;
    lst[2 * l + 1] = n;
  }
  __device__ int nactv(int l) const { return nact[l]; }
  __device__ void clear_flags(int l) {
    bl0[l] = 0;
    bl1[l] = 0;
  }
  // link at rest: full capacity, no flow (active counts are cleared by the host)
  __device__ void reset(int l, int64_t R) {
    set(l, R, 0);
    clear_flags(l);
  }
  __device__ Flags flags(int r) const { return Flags{(r & 1) ? bl1 : bl0, 0}; }
  template <class G> __device__ void addR(G& g, int l, int64_t v) { g.add(&lst[2 * l], v); }
  template <class G> __device__ void addN(G& g, int l, int64_t v) { g.add(&lst[2 * l + 1], v); }
  template <class G> __device__ void addNact(G& g, int l, int32_t v) { g.add(&nact[l], v); }
};

constexpr int LDS_LINKS = 2816;

struct LinkLds {
  int64_t R[LDS_LINKS];
  int32_t n[LDS_LINKS];
  int32_t nact[LDS_LINKS];
  uint8_t bl[2][LDS_LINKS];
};

struct LinksShared {
  LinkLds* s;
  int l0;
  double inv;
  __device__ double share(int l) const {
    const int i = l - l0;
    return ((double)s->R[i] / (double)s->n[i]) * inv;
  }
  __device__ void set(int l, int64_t R, int64_t n) {
    s->R[l - l0] = R;
    s->n[l - l0] = (int32_t)n;
  }
  __device__ int nactv(int l) const { return s->nact[l - l0]; }
  __device__ void clear_flags(int l) {
    s->bl[0][l - l0] = 0;
    s->bl[1][l - l0] = 0;
  }
  __device__ void reset(int l, int64_t R) {
    set(l, R, 0);
    s->nact[l - l0] = 0;
    clear_flags(l);
  }
  __device__ Flags flags(int r) const { return Flags{s->bl[r & 1], l0}; }
  template <class G> __device__ void addR(G&, int l, int64_t v) {
    __hip_atomic_fetch_add(&s->R[l - l0], v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  }
  template <class G> __device__ void addN(G&, int l, int64_t v) {
    __hip_atomic_fetch_add(&s->n[l - l0], (int32_t)v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  }
  template <class G> __device__ void addNact(G&, int l, int32_t v) {
    __hip_atomic_fetch_add(&s->nact[l - l0], v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  }
};

// ------------------------------------------------------------- rate solve
// Max-min rates of the n0 flows listed in list0 (all active), with work
// lists in global memory.  Cold (warm = false): link state starts from the
// capacities and the active counts; warm: from the residual state the event
// loop prepared.  Returns 0 or a negative status.
template <class G, class LK>
__device__ __forceinline__ int solve(G& g, const Params& P, LK& lk, ScenCtl* C, const int32_t* list0,
                                     int n0, int32_t* unf_a, int32_t* unf_b, int cap, int64_t& rounds,
                                     int64_t& fsw, int64_t& isw, Clock& clk, bool warm) {
  const int T = g.nthr();
  const int tid = g.tid();
  const int b0 = g.block_base();
  const bool one = g.nblocks() == 1;
  if (!warm) {
    for (int l = C->l0 + tid; l < C->l1; l += T) {
      lk.set(l, P.R0[l], lk.nactv(l));
      lk.clear_flags(l);
    }
  }
  if (tid == 0) {
    g.store(&C->cnt_unf[0], 0);
    g.store(&C->cnt_unf[1], 0);
  }
  g.sync();
  clk.lap(2);
  const int32_t* in = list0;
  int n = n0;
  int r = 0;
  int bad = 0;
  for (;;) {
    const Flags bl = lk.flags(r);
    const Flags bl_next = lk.flags(r + 1);
    int32_t* out = (r & 1) ? unf_b : unf_a;
    int32_t* out_cnt = &C->cnt_unf[r & 1];
    if (tid == 0 && r > 0) g.store(out_cnt, 0);
    // phase B: smallest share on each path; block links above it
    for (int i = tid; i < n; i += T) {
      const int f = in[i];
      if (!in_range(f, C->f0, cap)) { bad = 2; continue; }
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
            sv[k] = lk.share(lv[k]);
            m = sv[k] < m ? sv[k] : m;
          }
        }
        const double thr = m * THR;
#pragma unroll
        for (int k = 0; k < FAST_DEG; ++k)
          if (k < deg && sv[k] > thr) bl[lv[k]] = 1;
      } else {
        for (int e = e0; e < e1; ++e) {
          const double sh = lk.share(P.plink[e]);
          m = sh < m ? sh : m;
        }
        const double thr = m * THR;
        for (int e = e0; e < e1; ++e)
          if (lk.share(P.plink[e]) > thr) bl[P.plink[e]] = 1;
      }
      if (!(m > 0.0) || !(m < INF)) bad = 1;
      P.mf[f] = m;
    }
    clk.lap(3);
    g.sync();
    clk.lap(4);
    // phase C: freeze flows that cross an unblocked link
    for (int base = b0; base < n; base += T) {
      const int i = base + (int)threadIdx.x;
      bool keep = false;
      int f = -1;
      if (i < n) f = in[i];
      if (i < n && !in_range(f, C->f0, cap)) bad = 2;
      if (i < n && in_range(f, C->f0, cap)) {
        const int e0 = P.poff[f], e1 = P.poff[f + 1];
        bool frozen = false;
        for (int e = e0; e < e1; ++e) frozen |= (bl[P.plink[e]] == 0);
        if (frozen) {
          const double m = P.mf[f];
          P.rate[f] = m;
          const int64_t q = (int64_t)__builtin_rint(m * P.scale);
          for (int e = e0; e < e1; ++e) {
            const int l = P.plink[e];
            lk.addR(g, l, -q);
            lk.addN(g, l, (int64_t)-1);
          }
        } else {
          keep = true;
        }
      }
      int32_t* const cnts[1] = {out_cnt};
      const bool pr[1] = {keep};
      int slot[1];
      block_append<1>(g, cnts, pr, slot);
      if (keep) {
        if (slot[0] < cap) out[slot[0]] = f;
        else bad = 2;
      }
    }
    // Blocked flags are clean outside solves.  Several workgroups: clear the
    // next round's array now (its last readers passed a barrier) and this
    // round's after the final barrier.  One workgroup: clear exactly the
    // links this round may have flagged, once every thread has read them.
    if (!one) {
      for (int l = C->l0 + tid; l < C->l1; l += T) bl_next[l] = 0;
    } else {
      __syncthreads();
      for (int i = tid; i < n; i += T) {
        const int f = in[i];
        if (in_range(f, C->f0, cap))
          for (int e = P.poff[f]; e < P.poff[f + 1]; ++e) bl[P.plink[e]] = 0;
      }
    }
    if (bad) g.store(&C->fault_info, bad);
    clk.lap(5);
    g.sync();
    clk.lap(6);
    rounds += 1;
    fsw += n;
    if (g.aborted()) return ST_BARRIER;
    const int nout = g.load(out_cnt);
    if (g.load(&C->fault_info) != 0) return g.load(&C->fault_info) == 2 ? ST_OVERFLOW : ST_BAD_SHARE;
    if (nout == 0) {
      if (!one)
        for (int l = C->l0 + tid; l < C->l1; l += T) bl[l] = 0;
      return 0;
    }
    if (nout >= n) return ST_BAD_SHARE;  // a round must freeze something
    if (++r > P.max_rounds) return ST_ROUNDS;
    in = out;
    n = nout;
  }
}

// ---------------------------------------------- shared-memory-resident solve
// Each workgroup takes a contiguous slice of the active list (at most
// LDS_FLOWS flows), copies the flow ids and their padded paths (link ids
// local to the part, 16 bits) into shared memory once, and keeps its
// unfrozen flows as a shared-memory list.  Only link state and the rates are
// touched outside, so a round costs one gather of link state, one of flags
// and two barriers.
constexpr int LDS_FLOWS = 3840;
constexpr int LDS_DEG = 6;
constexpr uint16_t NO_LINK = 0xFFFF;

struct SolveLds {
  int32_t fid[LDS_FLOWS];
  uint16_t link[LDS_FLOWS * LDS_DEG];
  double mf[LDS_FLOWS];
  uint16_t u[2][LDS_FLOWS];
  int cnt;
  uint64_t clk[9];
};

template <class G, class LK>
__device__ __forceinline__ int solve_lds(G& g, const Params& P, LK& lk, ScenCtl* C, const int32_t* list0,
                                         int n0, int64_t& rounds, int64_t& fsw, int64_t& isw, Clock& clk,
                                         SolveLds& S, bool warm) {
  const int T = g.nthr();
  const int tid = g.tid();
  const int nb = g.nblocks();
  const int per = (n0 + nb - 1) / nb;
  const int c0 = min(n0, g.block_id() * per);
  const int nl = min(n0, c0 + per) - c0;
  const bool one = nb == 1;
  const int l0 = C->l0;
  if (!warm) {
    for (int l = C->l0 + tid; l < C->l1; l += T) {
      lk.set(l, P.R0[l], lk.nactv(l));
      lk.clear_flags(l);
    }
  }
  if (tid == 0)
    for (int k = 0; k < 3; ++k) g.store(&C->rem3[k], 0);
  int bad = 0;
  for (int j = threadIdx.x; j < nl; j += blockDim.x) {
    int f = list0[c0 + j];
    if (!in_range(f, C->f0, C->f1 - C->f0)) { bad = 2; f = C->f0; }
    const int e0 = P.poff[f], e1 = P.poff[f + 1];
    S.fid[j] = f;
#pragma unroll
    for (int k = 0; k < LDS_DEG; ++k)
      S.link[j * LDS_DEG + k] = e0 + k < e1 ? (uint16_t)(P.plink[e0 + k] - l0) : NO_LINK;
    S.u[0][j] = (uint16_t)j;
  }
  int nu = nl;
  g.sync();
  clk.lap(2);
  int total = n0;
  int r = 0;
  for (;;) {
    const Flags bl = lk.flags(r);
    const Flags bl_next = lk.flags(r + 1);
    const uint16_t* uin = S.u[r & 1];
    uint16_t* uout = S.u[(r & 1) ^ 1];
    if (threadIdx.x == 0) S.cnt = 0;
    if (tid == 0) g.store(&C->rem3[(r + 1) % 3], 0);
    // phase B: smallest share on each path; block links above it
    for (int x = threadIdx.x; x < nu; x += blockDim.x) {
      const int j = uin[x];
      double sv[LDS_DEG];
      int lv[LDS_DEG];
      double m = INF;
#pragma unroll
      for (int k = 0; k < LDS_DEG; ++k) {
        const uint16_t u = S.link[j * LDS_DEG + k];
        lv[k] = u == NO_LINK ? -1 : l0 + (int)u;
        if (lv[k] >= 0) {
          sv[k] = lk.share(lv[k]);
          m = sv[k] < m ? sv[k] : m;
          isw += 1;
        }
      }
      const double thr = m * THR;
#pragma unroll
      for (int k = 0; k < LDS_DEG; ++k)
        if (lv[k] >= 0 && sv[k] > thr) bl[lv[k]] = 1;
      if (!(m > 0.0) || !(m < INF)) bad = 1;
      S.mf[j] = m;
    }
    clk.lap(3);
    g.sync();
    clk.lap(4);
    // phase C: freeze flows crossing an unblocked link; keep the rest
    for (int base = 0; base < nu; base += blockDim.x) {
      const int x = base + (int)threadIdx.x;
      bool keep = false;
      int j = 0;
      if (x < nu) {
        j = uin[x];
        bool frozen = false;
#pragma unroll
        for (int k = 0; k < LDS_DEG; ++k) {
          const uint16_t u = S.link[j * LDS_DEG + k];
          if (u != NO_LINK) frozen |= (bl[l0 + (int)u] == 0);
        }
        if (frozen) {
          const double m = S.mf[j];
          P.rate[S.fid[j]] = m;
          const int64_t qv = (int64_t)__builtin_rint(m * P.scale);
#pragma unroll
          for (int k = 0; k < LDS_DEG; ++k) {
            const uint16_t u = S.link[j * LDS_DEG + k];
            if (u != NO_LINK) {
              lk.addR(g, l0 + (int)u, -qv);
              lk.addN(g, l0 + (int)u, (int64_t)-1);
            }
          }
        } else {
          keep = true;
        }
      }
      const uint64_t mask = __ballot(keep);
      if (mask) {
        const int lane = lane_id();
        const int leader = __ffsll((unsigned long long)mask) - 1;
        int b = 0;
        if (lane == leader) b = atomicAdd(&S.cnt, (int)__popcll(mask));
        b = __shfl(b, leader, 64);
        if (keep) uout[b + (int)__popcll(mask & ((1ull << lane) - 1ull))] = (uint16_t)j;
      }
    }
    if (!one)
      for (int l = C->l0 + tid; l < C->l1; l += T) bl_next[l] = 0;
    if (bad) g.store(&C->fault_info, bad);
    __syncthreads();
    const int nu_new = S.cnt;
    if (one) {
      // clear exactly what this round may have flagged (every read is done)
      for (int x = threadIdx.x; x < nu; x += blockDim.x) {
        const int j = uin[x];
#pragma unroll
        for (int k = 0; k < LDS_DEG; ++k) {
          const uint16_t u = S.link[j * LDS_DEG + k];
          if (u != NO_LINK) bl[l0 + (int)u] = 0;
        }
      }
    }
    if (threadIdx.x == 0 && nu_new > 0) g.add(&C->rem3[r % 3], (int32_t)nu_new);
    clk.lap(5);
    g.sync();
    clk.lap(6);
    rounds += 1;
    fsw += total;
    if (g.aborted()) return ST_BARRIER;
    if (g.load(&C->fault_info) != 0) return g.load(&C->fault_info) == 2 ? ST_OVERFLOW : ST_BAD_SHARE;
    const int left = g.load(&C->rem3[r % 3]);
    if (left == 0) {
      if (!one)
        for (int l = C->l0 + tid; l < C->l1; l += T) bl[l] = 0;
      return 0;
    }
    if (left >= total) return ST_BAD_SHARE;  // a round must freeze something
    if (++r > P.max_rounds) return ST_ROUNDS;
    total = left;
    nu = nu_new;
  }
}

// Releases flow h whose last predecessor finished at t (called once per h).
template <class G, class LK>
__device__ __forceinline__ void release_one(G& g, const Params& P, LK& lk, ScenCtl* C, int h, double t,
                                            int ob, int ib, int ev, int32_t* actOut,
                                            int32_t* pendOut, int32_t* arrOut, int32_t* cout,
                                            int32_t* coutCnt, int cap, int& err) {
  const double rl = P.start[h] + t;
  if (rl <= t) {
    if (P.nbytes[h] == 0.0) {
      P.finish[h] = rl;
      const int s = g.add(coutCnt, 1);
      if (s < cap) cout[s] = h; else err = 1;
    } else {
      P.rem[h] = P.nbytes[h];
      P.born[h] = ev;
      for (int j = P.poff[h]; j < P.poff[h + 1]; ++j) lk.addNact(g, P.plink[j], 1);
      const int s = g.add(&C->cnt_act[ob], 1);
      if (s < cap) actOut[s] = h; else err = 1;
      const int a = g.add(&C->cnt_arr, 1);
      if (a < cap) arrOut[a] = h; else err = 1;
      g.store(&C->changed[ib], 1);
    }
  } else {
    P.rel[h] = rl;
    const int s = g.add(&C->cnt_pend[ob], 1);
    if (s < cap) pendOut[s] = h; else err = 1;
  }
}

// ------------------------------------------------------------- event loop
// Incremental re-solve.  At the end of every solve all active flows are
// frozen: each link holds R0 minus the fixed-point rates of its active flows
// and an unfrozen count of zero.  When an event finishes flows with rates
// r_c and activates flows g, progressive filling on the new active set agrees
// with the previous one on every bottleneck level below
//   theta = min( min_c r_c, min over links l of every g of c_l / n_l(new) ):
// a finished flow's links were never bottlenecks below its rate, and a link
// of a new flow cannot reach a share below its initial share.  So every flow
// whose rate is below theta keeps it; the others (and the new flows) have
// their contributions taken back and are re-solved from that state.  Rates
// are identical to a full re-solve in exact arithmetic, and kept flows keep
// their bits.  Re-solves that fit in one workgroup's shared memory run on
// workgroup 0 alone, with workgroup barriers.
constexpr double KEEP = 1.0 - 1e-9;  // safety margin below theta

template <class G, class LK>
__device__ __forceinline__ void event_loop(G& g, const Params& P, LK& lk, const int sc, SolveLds& S) {
  ScenCtl* C = &P.ctl[sc];
  const int f0 = C->f0;
  const int cap = C->f1 - C->f0;
  int32_t* act[2] = {P.act0 + f0, P.act1 + f0};
  int32_t* pend[2] = {P.pend0 + f0, P.pend1 + f0};
  int32_t* comp[3] = {P.comp0 + f0, P.comp1 + f0, P.comp2 + f0};
  int32_t* unf_a = P.unf0 + f0;
  int32_t* unf_b = P.unf1 + f0;
  int32_t* arrs = P.arr + f0;
  const int T = g.nthr();
  const int tid = g.tid();
  const int b0 = g.block_base();
  const int w0 = tid - lane_id();
  Clock clk(tid == 0, S.clk);
  // links at rest: nothing active; no component has changed yet
  for (int l = C->l0 + tid; l < C->l1; l += T) lk.reset(l, P.R0[l]);
  const uint64_t INF_BITS = (uint64_t)__double_as_longlong(INF);
  for (int c = C->c0 + tid; c < C->c0 + C->nc; c += T) P.theta[c] = INF_BITS;
  double t = 0.0;
  int64_t events = 0, solves = 0, rounds = 0, fsw = 0, isw = 0, asw = 0, psw = 0;
  int64_t sel = 0, wide = 0;
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
      g.store(&C->succ_flag[ib], 0);
      g.store(&C->cnt_arr, 0);
      g.store(&C->cnt_sel, 0);
    }
    // next event time: earliest completion or release
    double loc = INF;
    for (int i = tid; i < nAct; i += T) {
      const int f = actIn[i];
      if (!in_range(f, f0, cap)) { g.store(&C->fault_info, 2); continue; }
      const double dt = P.rem[f] / P.rate[f];
      const double tau = t + dt;
      loc = tau < loc ? tau : loc;
    }
    for (int i = tid; i < nPend; i += T) {
      const int f = pendIn[i];
      if (!in_range(f, f0, cap)) { g.store(&C->fault_info, 2); continue; }
      const double rl = P.rel[f];
      loc = rl < loc ? rl : loc;
    }
    asw += nAct;
    psw += nPend;
    const double tn = g.min_all(loc);
    clk.lap(0);
    if (g.aborted()) { status = ST_BARRIER; break; }
    if (g.load(&C->fault_info) != 0) { status = ST_OVERFLOW; break; }
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
    for (int base = b0; base < nAct; base += T) {
      const int i = base + (int)threadIdx.x;
      bool done = false, keep = false;
      int f = -1;
      if (i < nAct) f = actIn[i];
      if (i < nAct && !in_range(f, f0, cap)) err = 1;
      if (i < nAct && in_range(f, f0, cap)) {
        const double r = P.rate[f];
        const double dt = P.rem[f] / r;
        const double tau = t + dt;
        if (tau <= thr) {
          done = true;
          P.finish[f] = tn;
          g.amin(&P.theta[P.comp[f]], (uint64_t)__double_as_longlong(r));
          const int64_t qv = (int64_t)__builtin_rint(r * P.scale);
          for (int k = P.poff[f]; k < P.poff[f + 1]; ++k) {
            const int l = P.plink[k];
            lk.addNact(g, l, -1);
            lk.addR(g, l, qv);  // its share returns to the link
          }
          if (P.soff[f + 1] > P.soff[f]) g.store(&C->succ_flag[ib], 1);
        } else {
          keep = true;
          const double moved = r * step;
          P.rem[f] = P.rem[f] - moved;
        }
      }
      int32_t* const cnts[2] = {compCnt, &C->cnt_act[ob]};
      const bool pr[2] = {done, keep};
      int slot[2];
      block_append<2>(g, cnts, pr, slot);
      if (done) { if (slot[0] < cap) compOut[slot[0]] = f; else err = 1; }
      if (keep) { if (slot[1] < cap) actOut[slot[1]] = f; else err = 1; }
      if (done) g.store(&C->changed[ib], 1);
    }
    // releases due now
    for (int base = b0; base < nPend; base += T) {
      const int i = base + (int)threadIdx.x;
      bool zero = false, start = false, keep = false;
      int f = -1;
      if (i < nPend) f = pendIn[i];
      if (i < nPend && !in_range(f, f0, cap)) err = 1;
      if (i < nPend && in_range(f, f0, cap)) {
        const double rl = P.rel[f];
        if (rl <= tn) {
          if (P.nbytes[f] == 0.0) {
            zero = true;
            P.finish[f] = rl;
            if (P.soff[f + 1] > P.soff[f]) g.store(&C->succ_flag[ib], 1);
          } else {
            start = true;
            P.rem[f] = P.nbytes[f];
            P.born[f] = e;
            for (int k = P.poff[f]; k < P.poff[f + 1]; ++k) lk.addNact(g, P.plink[k], 1);
          }
        } else {
          keep = true;
        }
      }
      int32_t* const cnts[4] = {compCnt, &C->cnt_act[ob], &C->cnt_pend[ob], &C->cnt_arr};
      const bool pr[4] = {zero, start, keep, start};
      int slot[4];
      block_append<4>(g, cnts, pr, slot);
      if (zero) { if (slot[0] < cap) compOut[slot[0]] = f; else err = 1; }
      if (start) {
        if (slot[1] < cap) actOut[slot[1]] = f; else err = 1;
        if (slot[3] < cap) arrs[slot[3]] = f; else err = 1;
        g.store(&C->changed[ib], 1);
      }
      if (keep) { if (slot[2] < cap) pendOut[slot[2]] = f; else err = 1; }
    }
    if (err) g.store(&C->fault_info, 2);
    g.sync();
    t = tn;
    q += 1;
    // dependants of finished flows, to a fixpoint through zero-byte flows.
    // A lane releases the successors of its own finished flow when it has a
    // few; long successor lists (a barrier's) are shared by the whole wave.
    int nc = g.load(&C->succ_flag[ib]) ? g.load(&C->cnt_comp[(q - 1) % 3]) : 0;
    while (nc > 0) {
      const int32_t* cin = comp[(q - 1) % 3];
      int32_t* cout = comp[q % 3];
      int32_t* coutCnt = &C->cnt_comp[q % 3];
      if (tid == 0) g.store(&C->cnt_comp[(q + 1) % 3], 0);
      for (int i0 = w0; i0 < nc; i0 += T) {
        const int i = i0 + lane_id();
        int k0 = 0, k1 = 0;
        if (i < nc) {
          const int f = cin[i];
          if (in_range(f, f0, cap)) {
            k0 = P.soff[f];
            k1 = P.soff[f + 1];
          } else {
            err = 1;
          }
        }
        const bool big = k1 - k0 > 8;
        if (!big) {
          for (int k = k0; k < k1; ++k) {
            const int h = P.succ[k];
            if (g.add(&P.cnt[h], -1) == 1)
              release_one(g, P, lk, C, h, t, ob, ib, e, actOut, pendOut, arrs, cout, coutCnt, cap,
                          err);
          }
        }
        uint64_t mask = __ballot(big);
        while (mask) {
          const int j = __ffsll((unsigned long long)mask) - 1;
          mask &= mask - 1;
          const int a = __shfl(k0, j, 64), z = __shfl(k1, j, 64);
          for (int k = a + lane_id(); k < z; k += 64) {
            const int h = P.succ[k];
            if (g.add(&P.cnt[h], -1) == 1)
              release_one(g, P, lk, C, h, t, ob, ib, e, actOut, pendOut, arrs, cout, coutCnt, cap,
                          err);
          }
        }
      }
      if (err) g.store(&C->fault_info, 2);
      g.sync();
      q += 1;
      nc = g.load(&C->cnt_comp[(q - 1) % 3]);
    }
    clk.lap(1);
    if (g.aborted()) { status = ST_BARRIER; break; }
    if (g.load(&C->fault_info) != 0) { status = ST_OVERFLOW; break; }
    const int nNew = g.load(&C->cnt_act[ob]);
    const int pNew = g.load(&C->cnt_pend[ob]);
    if (g.load(&C->changed[ib]) && nNew > 0) {
      // theta of each component: below it every rate stays as it was.
      // Finished flows have fed it their rates; new flows feed the initial
      // share of their links.
      const int nArr = g.load(&C->cnt_arr);
      for (int i = tid; i < nArr; i += T) {
        const int f = arrs[i];
        if (!in_range(f, f0, cap)) continue;
        double lo = INF;
        for (int k = P.poff[f]; k < P.poff[f + 1]; ++k) {
          const int l = P.plink[k];
          const double s0 = ((double)P.R0[l] / (double)lk.nactv(l)) * P.inv_scale;
          lo = s0 < lo ? s0 : lo;
        }
        g.amin(&P.theta[P.comp[f]], (uint64_t)__double_as_longlong(lo));
      }
      // take back the flows at or above their component's theta (and the new
      // ones) for re-solving
      g.sync();
      for (int base = b0; base < nNew; base += T) {
        const int i = base + (int)threadIdx.x;
        bool upper = false;
        int f = -1;
        if (i < nNew) {
          f = actOut[i];
          if (in_range(f, f0, cap)) {
            const bool fresh = P.born[f] == e;
            const double r = P.rate[f];
            const double th = __longlong_as_double((long long)g.load(&P.theta[P.comp[f]]));
            upper = fresh || !(r < th * KEEP);
            if (upper) {
              const int64_t qv = fresh ? 0 : (int64_t)__builtin_rint(r * P.scale);
              for (int k = P.poff[f]; k < P.poff[f + 1]; ++k) {
                const int l = P.plink[k];
                if (!fresh) lk.addR(g, l, qv);
                lk.addN(g, l, (int64_t)1);
              }
            }
          } else {
            err = 1;
          }
        }
        int32_t* const cnts[1] = {&C->cnt_sel};
        const bool pr[1] = {upper};
        int slot[1];
        block_append<1>(g, cnts, pr, slot);
        if (upper) { if (slot[0] < cap) arrs[slot[0]] = f; else err = 1; }
      }
      if (err) g.store(&C->fault_info, 2);
      g.sync();
      clk.lap(7);
      for (int c = C->c0 + tid; c < C->c0 + C->nc; c += T) P.theta[c] = INF_BITS;
      const int nSel = g.load(&C->cnt_sel);
      if (P.debug) {
        // blocked flags must be clean between solves
        for (int l = C->l0 + tid; l < C->l1; l += T)
          if (lk.flags(0)[l] | lk.flags(1)[l]) {
            g.store(&C->dbg[0], (int64_t)(e + 1));
            g.store(&C->dbg[1], (int64_t)l);
          }
        g.sync();
        if (g.load(&C->dbg[0]) != 0 && status == ST_DONE) { status = -8; break; }
      }
      sel += nSel;
      wide += nSel > LDS_FLOWS ? 1 : 0;
      int rc = 0;
      if (nSel > 0) {
        if (P.debug && tid == 0) g.store(&C->dbg[2], (int64_t)(nSel <= LDS_FLOWS ? 1 : nSel <= g.nblocks() * LDS_FLOWS ? 2 : 3));
        if (C->lds_paths && nSel <= LDS_FLOWS) {
          if (g.nblocks() == 1) {
            rc = solve_lds(g, P, lk, C, arrs, nSel, rounds, fsw, isw, clk, S, true);
          } else {
            if (g.block_id() == 0) {
              BlockG b{g.lds, g.ldsi};
              const int r1 = solve_lds(b, P, lk, C, arrs, nSel, rounds, fsw, isw, clk, S, true);
              if (threadIdx.x == 0) g.store(&C->solve_rc, r1);
            }
            g.sync();
            rc = g.load(&C->solve_rc);
          }
        } else if (C->lds_paths && nSel <= g.nblocks() * LDS_FLOWS) {
          rc = solve_lds(g, P, lk, C, arrs, nSel, rounds, fsw, isw, clk, S, true);
        } else {
          rc = solve(g, P, lk, C, arrs, nSel, unf_a, unf_b, cap, rounds, fsw, isw, clk, true);
        }
      }
      solves += 1;  // the active set changed: one rate solve (possibly empty)
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
    C->reselected = sel;
    C->wide_solves = wide;
    C->status = status;
    for (int k = 0; k < 8; ++k) C->ticks[k] = (int64_t)S.clk[k];
  }
}

template <class G>
__device__ __forceinline__ void solve_only(G& g, const Params& P, const int sc, SolveLds& S) {
  LinksGlobal lk{P.lst, P.nact, P.blocked0, P.blocked1, P.inv_scale};
  ScenCtl* C = &P.ctl[sc];
  const int f0 = C->f0;
  int64_t rounds = 0, fsw = 0, isw = 0;
  Clock clk(g.tid() == 0, S.clk);
  int rc = 0;
  if (C->n_solve > 0)
    rc = (C->lds_paths && C->n_solve <= g.nblocks() * LDS_FLOWS)
             ? solve_lds(g, P, lk, C, P.act0 + f0, C->n_solve, rounds, fsw, isw, clk, S, false)
             : solve(g, P, lk, C, P.act0 + f0, C->n_solve, P.unf0 + f0, P.unf1 + f0, C->f1 - f0,
                     rounds, fsw, isw, clk, false);
  g.add(&C->incidences_swept, isw);
  if (g.tid() == 0) {
    C->solves = C->n_solve > 0 ? 1 : 0;
    C->rounds = rounds;
    C->flows_swept = fsw;
    C->status = rc;
    for (int k = 0; k < 8; ++k) C->ticks[k] = (int64_t)S.clk[k];
  }
}

}  // namespace

// One workgroup per part.  A part whose links fit keeps its link state in
// shared memory for the whole run.
__global__ __launch_bounds__(1024) void netsim_block_kernel(Params P) {
  __shared__ double lds[32];
  __shared__ int ldsi[128];
  __shared__ SolveLds S;
  __shared__ LinkLds LL;
  BlockG g{lds, ldsi};
  for (int sc = blockIdx.x; sc < P.num_scen; sc += gridDim.x) {
    const ScenCtl* C = &P.ctl[sc];
    if (P.mode != 0) {
      solve_only(g, P, sc, S);
    } else if (C->l1 - C->l0 <= LDS_LINKS) {
      LinksShared lk{&LL, C->l0, P.inv_scale};
      event_loop(g, P, lk, sc, S);
    } else {
      LinksGlobal lk{P.lst, P.nact, P.blocked0, P.blocked1, P.inv_scale};
      event_loop(g, P, lk, sc, S);
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(1024) void netsim_grid_kernel(Params P) {
  __shared__ double lds[32];
  __shared__ int ldsi[128];
  __shared__ int flag;
  __shared__ SolveLds S;
  GridG g{lds, ldsi, &flag, P.bar, P.slots, 0u, 0u, false, 0u, 0u, 0u};
  g.init();
  LinksGlobal lk{P.lst, P.nact, P.blocked0, P.blocked1, P.inv_scale};
  for (int sc = 0; sc < P.num_scen; ++sc) {
    if (P.mode == 0) event_loop(g, P, lk, sc, S);
    else solve_only(g, P, sc, S);
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
