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
// The same code runs over a "group" of threads: one workgroup per part of a
// scenario (BlockG, workgroup barriers) or the whole grid on one part at a time
// (GridG, an atomic grid barrier with a time-out).  Every loop exit depends
// only on values read after a group barrier, so all waves leave together.
#include "device.h"

#include <math.h>

namespace netsim_dev {

namespace {

constexpr double THR = 1.000000000001;
constexpr double INF = __builtin_huge_val();
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
  Lists* lst;  // list counters: shared memory (block kernel, zeroed when a part
               // starts) or the part's control block (a solve run by one workgroup
               // of the grid)
  __device__ Lists* lists(ScenCtl*) const { return lst; }
  __device__ int tid() const { return threadIdx.x; }
  __device__ int block_base() const { return 0; }
  __device__ int nblocks() const { return 1; }
  __device__ int block_id() const { return 0; }
  __device__ int nthr() const { return blockDim.x; }
  __device__ bool aborted() const { return false; }
  __device__ void sync() { __syncthreads(); }
  __device__ __forceinline__ double min_all(double v) {
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
  __device__ void amax(uint64_t* p, uint64_t v) {
    __hip_atomic_fetch_max(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  }
};

// Barrier words (uint32 indices into Params::bar, 64-byte lines apart):
constexpr int BAR_COUNT = 0, BAR_GEN = 1, BAR_ABORT = 16, BAR_REG = 32, BAR_REG_GEN = 33;
constexpr int BAR_XCD = 64;        // XCD x: arrivals at 64 + 32x, generation at 64 + 32x + 16
constexpr int BAR_XCD_BLOCKS = 640;  // blocks resident on XCD x (of 1024 words)

__device__ __forceinline__ unsigned xcc_id() {
  return __builtin_amdgcn_s_getreg(6164) & 15u;  // hwreg(HW_REG_XCC_ID, 0, 4)
}

struct GridG {
  double* lds;
  int* ldsi;
  __device__ Lists* lists(ScenCtl* C) const { return &C->k; }
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
  __device__ void amax(uint64_t* p, uint64_t v) {
    __hip_atomic_fetch_max(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
};

// Cluster kernel words.  XCD x counts its workgroups in XREG_BASE + 16x; its
// workgroups form up to CL_MAXC clusters (a leader and its helpers), and
// cluster k of XCD x owns CL_STRIDE words from CL_BASE + CL_STRIDE*(x*CL_MAXC + k)
// (offsets below, 64-byte lines apart where several writers meet).
constexpr int BAR_NEXT = 48;  // next part to be claimed by a leader
constexpr int XREG_BASE = 672;
constexpr int CL_MAXC = 4;
constexpr int CL_BASE = 1024, CL_STRIDE = 128;
constexpr int CL_MB = 16;                 // jobs posted so far, or CL_CLOSED
constexpr int CL_SC = 17, CL_N = 18;      // posted job: part, number of flows,
constexpr int CL_AB = 19, CL_SNEW = 20;   //   slot buffer, first slot activated at this event,
constexpr int CL_T = 22;                  //   event time (double)
constexpr int CL_DONE = 32;               // jobs finished, summed over the helpers
constexpr int CL_RC = 33;                 // job status (first helper)
constexpr int CL_ROUNDS = 34, CL_FSW = 36;  // job rounds and flows swept (int64, first helper)
constexpr int CL_ISW = 48;                // incidences swept (int64, summed over the helpers)
constexpr int CL_CLK = 96;                // job phase times of the first helper (int64 [8])
constexpr uint32_t CL_CLOSED = 0xFFFFFFFFu;
// Helper arrival lines: cluster k owns CL_LINES lines of 128 bytes from
// CL_ARRIVE + CL_ARRIVE_STRIDE*k; helper h writes only line h.
constexpr int CL_ARRIVE = 9216, CL_LINES = 32, CL_LINE_WORDS = 32;
constexpr int CL_ARRIVE_STRIDE = CL_LINES * CL_LINE_WORDS;
constexpr int NOT_TAKEN = 2;              // the helpers have left: solve locally
// A helper with no job for this long leaves (its leader then solves alone).
constexpr uint64_t IDLE_TICKS = 6000000000ull;  // 60 s at 100 MHz
// Test hooks (Params::debug): helpers that leave as soon as they have no job
// (their leader then solves alone), and a helper barrier that gives up at
// once (the launch aborts and the part reports a barrier time-out).  Both
// only shorten the kernel's own bounded waits.
constexpr int DEBUG_HELPERS_LEAVE = 4, DEBUG_HELPER_BARRIER_GIVES_UP = 8;
static_assert(XREG_BASE + 16 * 16 <= CL_BASE, "registration words");
static_assert(CL_BASE + 16 * CL_MAXC * CL_STRIDE <= CL_ARRIVE, "cluster words");
static_assert(CL_ARRIVE + 16 * CL_MAXC * CL_ARRIVE_STRIDE <= BAR_WORDS, "arrival lines");

// Waits (one thread) until *p != v, giving up when the abort word is set or
// after `ticks` (then raising it).  Returns false if it gave up.
__device__ __forceinline__ bool wait_ne(uint32_t* bar, uint32_t* p, uint32_t v, uint64_t ticks) {
  const uint64_t t0 = wall_clock64();
  while (__hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == v) {
    __builtin_amdgcn_s_sleep(1);
    if (__hip_atomic_load(&bar[BAR_ABORT], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0) return false;
    if (wall_clock64() - t0 > ticks) {
      __hip_atomic_store(&bar[BAR_ABORT], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      return false;
    }
  }
  return true;
}

// Waits for this wave's outstanding memory operations (stores and atomics
// included), so that a later release by another wave of the workgroup
// covers them.
__device__ __forceinline__ void drain() { __builtin_amdgcn_s_waitcnt(0); }

// The release before a signal to other workgroups of the same XCD: by
// default each wave drains its memory operations (enough there, see
// ClusterG); with options.debug bit 6 an agent-scope release fence, the
// memory model's own form (it also writes the L2 back, for other XCDs).
constexpr int DEBUG_FORMAL_RELEASE = 64;
__device__ __forceinline__ void xcd_release(bool formal) {
  if (formal) __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
  else drain();
}

// The helper workgroups of one XCD (all but its leader), solving one job at a
// time with a barrier of their own.
//
// Everything the helpers and their leader share lives in device memory and
// is exchanged inside one XCD, whose L2 they all use.  So a helper's release
// needs no L2 write-back (what the agent-scope release adds, for other XCDs):
// each wave drains its stores and atomics (they are then in that L2, or
// performed at agent scope) before its workgroup signals.  Within a job the
// helpers update link state only with agent-scope atomics and stamps only
// with plain stores.  An acquire stays agent-scope: it drops this CU's L1 and
// the L2's clean copies (measured: dropping only the L1 reads stale link
// state).  The leader hands link state over with agent-scope stores (or,
// when the state lives in global memory, after a full agent-scope release),
// so the helpers' atomics never follow plain stores to the same words.
//
// Barrier: each helper has an arrival line of its own (no two arrivals touch
// one word, so none waits for another's read-modify-write) and, at its k-th
// barrier, stores (k, payload) into word k mod 2 of it; lane h of the first
// wave of every helper polls helper h's line until all of them show k.  The
// payload (the helper's count of unfrozen flows and a fault bit) reaches
// every helper with the arrival itself, so a round needs no counter in
// memory.  Two words per line: a helper can be at most one barrier ahead of
// the slowest poller (it cannot pass barrier k + 1 before that poller
// arrives there), so word k mod 2 still holds barrier k's payload while
// anybody polls it.  A wait longer than `patience` (BARRIER_TIMEOUT_TICKS)
// raises the launch's abort word.
struct ClusterG {
  double* lds;
  int* ldsi;
  int* flag;      // shared [2]: abort state as seen by this block's first wave, payload sum
  uint32_t* bar;  // launch words (abort flag)
  uint32_t* cw;   // this XCD's cluster words
  uint32_t gen;
  int rank, nh;   // rank among the helpers, number of helpers
  bool ab;
  uint64_t patience;  // barrier time-out (ticks)
  bool formal;        // agent-scope release fences instead of drains (debug)
  uint64_t* lines;    // this cluster's arrival lines (CL_LINE_WORDS / 2 words apart)
  int64_t* dR;        // shared memory: per-link deltas of this helper (residual,
  int32_t* dn;        //   unfrozen count), folded into link state once per phase
  int dcap;           // links the delta arrays hold
  __device__ Lists* lists(ScenCtl* C) const { return &C->k; }
  __device__ int tid() const { return rank * blockDim.x + threadIdx.x; }
  __device__ int block_base() const { return rank * blockDim.x; }
  __device__ int nblocks() const { return nh; }
  __device__ int block_id() const { return rank; }
  __device__ int nthr() const { return nh * blockDim.x; }
  __device__ bool aborted() const { return ab; }
  __device__ __forceinline__ void sync() { (void)sync_sum(0u); }
  // The barrier; returns the sum over the helpers of their payloads (low 31
  // bits) with bit 31 set if any helper's payload had it.
  __device__ __forceinline__ uint32_t sync_sum(uint32_t payload) {
    xcd_release(formal);
    __syncthreads();
    if (threadIdx.x < 64) {
      const int lane = (int)threadIdx.x;
      const uint32_t target = gen + 1;
      const int w = (int)(target & 1u);
      uint32_t a = 0;
      if (lane == 0) {
        // the arrival and a look at the abort word travel together; an abort
        // raised meanwhile is seen at a later barrier or in a wait (the word
        // stays set, so a helper that leaves early cannot strand the others)
        a = __hip_atomic_load(&bar[BAR_ABORT], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(lines + (size_t)rank * (CL_LINE_WORDS / 2) + w,
                           ((uint64_t)target << 32) | payload, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      a = (uint32_t)__shfl((int)a, 0, 64);
      uint64_t* mine = lines + (size_t)(lane < nh ? lane : 0) * (CL_LINE_WORDS / 2) + w;
      uint64_t v = 0;
      if (a == 0) {
        const uint64_t t0 = wall_clock64();
        for (uint32_t i = 1;; ++i) {
          bool here = true;
          if (lane < nh) {
            v = __hip_atomic_load(mine, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            here = (int32_t)((uint32_t)(v >> 32) - target) >= 0;
          }
          if (__all(here)) break;
          __builtin_amdgcn_s_sleep(1);
          if ((i & 15) != 1) continue;
          if (lane == 0) {
            a = __hip_atomic_load(&bar[BAR_ABORT], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (a == 0 && wall_clock64() - t0 > patience) {
              __hip_atomic_store(&bar[BAR_ABORT], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
              a = 1;
            }
          }
          a = (uint32_t)__shfl((int)a, 0, 64);
          if (a != 0) break;
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
      uint32_t sum = lane < nh ? (uint32_t)v & 0x7FFFFFFFu : 0u;
      uint32_t any = lane < nh ? (uint32_t)v & 0x80000000u : 0u;
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) {
        sum += (uint32_t)__shfl_xor((int)sum, o, 64);
        any |= (uint32_t)__shfl_xor((int)any, o, 64);
      }
      if (lane == 0) {
        flag[0] = (int)a;
        flag[1] = (int)(sum | any);
      }
    }
    gen += 1;
    __syncthreads();
    ab = flag[0] != 0;
    return (uint32_t)flag[1];
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

template <class G> struct IsGrid { static constexpr bool value = false; };
template <> struct IsGrid<GridG> { static constexpr bool value = true; };
template <class G> struct IsCluster { static constexpr bool value = false; };
template <> struct IsCluster<ClusterG> { static constexpr bool value = true; };

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

// For every item i < n of the group: x = fetch(i) (loads only), then
// decide(i, x, pred) (pred[k]: the item goes to list k, counted by
// counters[k]), then put(k, slot, x) for every list it goes to.  One
// workgroup fetches four items of a thread at a time (their loads in flight
// together) and appends with one ballot and one shared-memory atomic per
// wave and list, so the sweep needs no workgroup barrier (list order is
// arbitrary; nothing depends on it).  The grid appends chunks of one item per
// thread with block_append.  Every thread of the group must call it.
template <int NL, class G, class Fetch, class Decide, class Put>
__device__ __forceinline__ void sweep_append(G& g, int n, int32_t* const* counters, Fetch fetch,
                                             Decide decide, Put put) {
  const int T = g.nthr();
  if constexpr (!IsGrid<G>::value) {
    using Item = decltype(fetch(0));
    for (int j0 = 0; j0 * T < n; j0 += 4) {
      Item x[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = (int)threadIdx.x + (j0 + u) * T;
        if (i < n) x[u] = fetch(i);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = (int)threadIdx.x + (j0 + u) * T;
        bool pr[NL] = {};
        if (i < n) decide(i, x[u], pr);
#pragma unroll
        for (int k = 0; k < NL; ++k) {
          const int slot = wave_append(g, counters[k], pr[k]);
          if (pr[k]) put(k, slot, x[u]);
        }
      }
    }
    return;
  }
  for (int base = g.block_base(); base < n; base += T) {
    const int i = base + (int)threadIdx.x;
    bool pr[NL] = {};
    decltype(fetch(0)) x{};
    if (i < n) {
      x = fetch(i);
      decide(i, x, pr);
    }
    int slot[NL];
    block_append<NL>(g, counters, pr, slot);
#pragma unroll
    for (int k = 0; k < NL; ++k)
      if (pr[k]) put(k, slot[k], x);
  }
}

// What a sweep loads for one item before deciding about it.
struct FlowVal {
  int f = -1;
  int k = 0;
  double a = 0.0, b = 0.0;
};

// Per-phase wall-clock accounting by the group's first thread, kept in
// shared memory (acc[0..8) and the last reading in acc[8]).
struct Clock {
  bool on;
  uint64_t* acc;
  __device__ __forceinline__ Clock(bool o, uint64_t* a) : on(o), acc(a) {
    if (threadIdx.x == 0)
      for (int k = 0; k < 8; ++k) acc[k] = 0;
    if (on) acc[8] = wall_clock64();
  }
  __device__ __forceinline__ void lap(int k) {
    if (on) {
      const uint64_t now = wall_clock64();
      acc[k] += now - acc[8];
      acc[8] = now;
    }
  }
  // restarts the current lap without counting the time since the last one
  __device__ __forceinline__ void skip() {
    if (on) acc[8] = wall_clock64();
  }
};

// Counters of a part's run, in shared memory, advanced by each workgroup's
// first thread only (they are the same for every thread of the group).
struct Tally {
  uint64_t clk[9];
  int64_t solves, rounds, fsw, asw, psw, sel, wide, asst;
};

// A flow id read from a work list must lie in the scenario's range.
__device__ __forceinline__ bool in_range(int f, int f0, int cap) {
  return (unsigned)(f - f0) < (unsigned)cap;
}

// ------------------------------------------------------------ link state
// Per link: residual capacity R (fixed point), unfrozen flows n, active flows
// nact and a "blocked" stamp: a link is blocked in a freezing round iff its
// stamp equals that round's number, so flags never need clearing (round
// numbers keep growing through a part's solves; see first_round).  Two homes
// for the state, with one interface taking device link ids:
//   LinksGlobal - global memory; any group (the whole grid, or a workgroup
//                 on a part too large for shared memory);
//   LinksShared - the shared memory of the one workgroup running a part
//                 whose links fit there; its atomics stay inside the CU.
struct LinksGlobal {
  static constexpr bool kTable = false;  // shares computed where they are needed
  int64_t* lst;      // [2L] (R, n) pairs: one 16-byte load per link
  int32_t* nact;
  uint32_t* fl;
  double inv;
  __device__ __forceinline__ double share(int l) const {
    const longlong2 v = *reinterpret_cast<const longlong2*>(lst + 2 * l);
    return ((double)v.x / (double)v.y) * inv;
  }
  __device__ __forceinline__ void set(int l, int64_t R, int64_t n) {
    lst[2 * l] = R;
    lst[2 * l + 1] = n;
  }
  __device__ __forceinline__ int64_t nfree(int l) const { return lst[2 * l + 1]; }
  __device__ __forceinline__ int nactv(int l) const { return nact[l]; }
  __device__ __forceinline__ void clear_flag(int l) { fl[l] = 0; }
  // link at rest: full capacity, no flow
  __device__ __forceinline__ void reset(int l, int64_t R) {
    set(l, R, 0);
    nact[l] = 0;
    fl[l] = 0;
  }
  __device__ __forceinline__ void block(int l, uint32_t st) { fl[l] = st; }
  __device__ __forceinline__ bool blocked(int l, uint32_t st) const { return fl[l] == st; }
  template <class G> __device__ __forceinline__ void addR(G& g, int l, int64_t v) { g.add(&lst[2 * l], v); }
  template <class G> __device__ __forceinline__ void addN(G& g, int l, int64_t v) { g.add(&lst[2 * l + 1], v); }
  template <class G> __device__ __forceinline__ void addNact(G& g, int l, int32_t v) { g.add(&nact[l], v); }
};

// Shared-memory pool of the block kernel: a part whose links fit keeps its
// link state there (LINK_LDS_BYTES per link) and uses the rest as a cache of
// path records for the flows of its solves (FLOW_LDS_BYTES per flow).
constexpr int POOL_BYTES = 152 * 1024;
constexpr int LINK_LDS_BYTES = 28;  // R 8, n 4, nact 4, stamp 4, share 8
constexpr int FLOW_LDS_BYTES = 20;  // path record 16, flow id 4

struct LinksShared {
  static constexpr bool kTable = true;  // shares of a round in a table (link pass)
  int64_t* R;
  double* sh;
  int32_t* n;
  int32_t* nact;
  uint32_t* fl;
  int l0;
  double inv;
  // Carves the link arrays for nl links and one sentinel entry (link id
  // first + nl: share +inf, never stamped; what absent path entries point
  // at, so that path gathers need no guard) out of the pool (16-byte aligned).
  __device__ __forceinline__ LinksShared(unsigned char* pool, int first, int nl, double inv_scale)
      : l0(first), inv(inv_scale) {
    const int nl2 = (nl + 2) & ~1;
    R = reinterpret_cast<int64_t*>(pool);
    sh = reinterpret_cast<double*>(pool + 8 * nl2);
    n = reinterpret_cast<int32_t*>(pool + 16 * nl2);
    nact = n + nl2;
    fl = reinterpret_cast<uint32_t*>(nact + nl2);
  }
  __device__ __forceinline__ double share(int l) const {
    const int i = l - l0;
    return ((double)R[i] / (double)n[i]) * inv;
  }
  __device__ __forceinline__ double table(int l) const { return sh[l - l0]; }
  __device__ __forceinline__ uint32_t stamp(int l) const { return fl[l - l0]; }
  // the sentinel after the nl links of the part
  __device__ __forceinline__ void set_sentinel(int nl) {
    R[nl] = 0;
    n[nl] = 0;
    nact[nl] = 0;
    fl[nl] = 0;
    sh[nl] = INF;
  }
  // link pass of a round: the share of every link with an unfrozen flow;
  // returns how many of those this thread saw
  __device__ __forceinline__ int fill_table(int tid, int T, int nl) {
    int c = 0;
    for (int i = tid; i < nl; i += T)
      if (n[i] > 0) {
        sh[i] = ((double)R[i] / (double)n[i]) * inv;
        ++c;
      }
    return c;
  }
  __device__ __forceinline__ void set(int l, int64_t Rv, int64_t nv) {
    R[l - l0] = Rv;
    n[l - l0] = (int32_t)nv;
  }
  __device__ __forceinline__ int64_t nfree(int l) const { return n[l - l0]; }
  __device__ __forceinline__ int nactv(int l) const { return nact[l - l0]; }
  __device__ __forceinline__ void clear_flag(int l) { fl[l - l0] = 0; }
  __device__ __forceinline__ void reset(int l, int64_t Rv) {
    set(l, Rv, 0);
    nact[l - l0] = 0;
    fl[l - l0] = 0;
  }
  __device__ __forceinline__ void block(int l, uint32_t st) { fl[l - l0] = st; }
  __device__ __forceinline__ bool blocked(int l, uint32_t st) const { return fl[l - l0] == st; }
  template <class G> __device__ __forceinline__ void addR(G&, int l, int64_t v) {
    __hip_atomic_fetch_add(&R[l - l0], v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  }
  template <class G> __device__ __forceinline__ void addN(G&, int l, int64_t v) {
    __hip_atomic_fetch_add(&n[l - l0], (int32_t)v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  }
  template <class G> __device__ __forceinline__ void addNact(G&, int l, int32_t v) {
    __hip_atomic_fetch_add(&nact[l - l0], v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  }
};

// Bytes of the pool taken by the link arrays of nl links and the sentinel.
__host__ __device__ constexpr int link_pool_bytes(int nl) { return LINK_LDS_BYTES * ((nl + 2) & ~1); }

// First round number of a solve of part C (read by every thread after a
// group barrier).  Far from wrapping every stamp is cleared and numbering
// restarts, so a stale stamp can never equal a live round number.
template <class G, class LK>
__device__ __forceinline__ uint32_t first_round(G& g, const Params& P, LK& lk, ScenCtl* C) {
  Lists* K = g.lists(C);
  uint32_t base = g.load(&K->stamp);
  if (base > 0x7FFFFFFFu) {
    for (int l = C->l0 + g.tid(); l < C->l1; l += g.nthr()) lk.clear_flag(l);
    g.sync();
    base = 0;
  }
  return base + 1;
}

// Cold start of a solve (no event loop before it): capacities, the active
// counts as unfrozen counts, no stamps.
template <class G, class LK>
__device__ __forceinline__ void cold_links(G& g, const Params& P, LK& lk, ScenCtl* C) {
  for (int l = C->l0 + g.tid(); l < C->l1; l += g.nthr()) {
    lk.set(l, P.R0[l], lk.nactv(l));
    lk.clear_flag(l);
  }
}

// Phase B for one flow: the smallest fair share on its path, and a stamp on
// every link of the path whose share exceeds it by more than the tie band.
// Returns the smallest share (bad = 1 when it is not a positive finite
// number).
template <class LK>
__device__ __forceinline__ double share_of(const LK& lk, int l) {
  if constexpr (LK::kTable) return lk.table(l);
  else return lk.share(l);
}

// Link pass of a round when the link store keeps a share table: every
// link's share, computed once, then read by all flows of the round.
template <class G, class LK>
__device__ __forceinline__ void round_table(G& g, LK& lk, const ScenCtl* C) {
  if constexpr (LK::kTable) {
    int c = lk.fill_table(g.tid(), g.nthr(), C->l1 - C->l0);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o, 64);
    if (lane_id() == 0 && c > 0) g.add(&g.lists(const_cast<ScenCtl*>(C))->lsw, (int64_t)c);
    g.sync();
  }
}

template <class LK>
__device__ __forceinline__ double share_and_block(LK& lk, const int* lv, int deg, uint32_t st,
                                                  int& bad, uint32_t* at_min = nullptr) {
  double sv[6];
  double m = INF;
#pragma unroll
  for (int k = 0; k < 6; ++k)
    if (k < deg) {
      sv[k] = share_of(lk, lv[k]);
      m = sv[k] < m ? sv[k] : m;
    }
  const double thr = m * THR;
  uint32_t cm = 0;  // links of the path within the tie band of its minimum
#pragma unroll
  for (int k = 0; k < 6; ++k)
    if (k < deg) {
      if (sv[k] > thr) lk.block(lv[k], st);
      else cm |= 1u << k;
    }
  if (!(m > 0.0) || !(m < INF)) bad = 1;
  if (at_min) *at_min = cm;
  return m;
}

// Unpacks a 16-byte path record: up to six link ids local to the part (16
// bits each, NO_LINK = unused) into device link ids; returns the degree.
constexpr uint32_t NO_LINK = 0xFFFFu;
__device__ __forceinline__ int unpack_path(const uint4 rec, int l0, int* lv) {
  const uint32_t w[3] = {rec.x, rec.y, rec.z};
  int deg = 0;
#pragma unroll
  for (int k = 0; k < 6; ++k) {
    const uint32_t u = (w[k >> 1] >> (16 * (k & 1))) & 0xFFFFu;
    lv[k] = l0 + (int)u;
    deg += u != NO_LINK;
  }
  return deg;  // links are packed first, so lv[0..deg) are the path
}

// ------------------------------------------------------------- rate solve
// Max-min rates of the n0 flows listed in list0 (all active), with work
// lists in global memory (any group, any path length).  Cold (warm = false):
// link state starts from the capacities and the active counts; warm: from
// the residual state the event loop prepared.  Returns 0 or a negative
// status.
template <class G, class LK>
__device__ __forceinline__ int solve(G& g, const Params& P, LK& lk, ScenCtl* C, const int32_t* list0,
                                     int n0, int32_t* unf_a, int32_t* unf_b, int cap, int64_t& rounds,
                                     int64_t& fsw, int64_t& isw, Clock& clk, bool warm) {
  Lists* K = g.lists(C);
  const int T = g.nthr();
  const int tid = g.tid();
  const int b0 = g.block_base();
  if (!warm) cold_links(g, P, lk, C);
  if (tid == 0) {
    g.store(&K->unf[0], 0);
    g.store(&K->unf[1], 0);
  }
  g.sync();
  const uint32_t st0 = first_round(g, P, lk, C);
  clk.lap(2);
  const int32_t* in = list0;
  int n = n0;
  int r = 0;
  int bad = 0;
  int rc = 0;
  for (;;) {
    const uint32_t st = st0 + (uint32_t)r;
    int32_t* out = (r & 1) ? unf_b : unf_a;
    int32_t* out_cnt = &K->unf[r & 1];
    if (tid == 0 && r > 0) g.store(out_cnt, 0);
    round_table(g, lk, C);
    clk.lap(2);
    // phase B: smallest share on each path; block links above it
    for (int i = tid; i < n; i += T) {
      const int f = in[i];
      if (!in_range(f, C->f0, cap)) { bad = 2; continue; }
      const int e0 = P.poff[f], e1 = P.poff[f + 1];
      const int deg = e1 - e0;
      isw += deg;
      double m;
      if (deg <= 6) {
        int lv[6];
#pragma unroll
        for (int k = 0; k < 6; ++k) lv[k] = k < deg ? P.plink[e0 + k] : 0;
        m = share_and_block(lk, lv, deg, st, bad);
      } else {
        m = INF;
        for (int e = e0; e < e1; ++e) {
          const double sh = share_of(lk, P.plink[e]);
          m = sh < m ? sh : m;
        }
        const double thr = m * THR;
        for (int e = e0; e < e1; ++e)
          if (share_of(lk, P.plink[e]) > thr) lk.block(P.plink[e], st);
        if (!(m > 0.0) || !(m < INF)) bad = 1;
      }
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
        for (int e = e0; e < e1; ++e) frozen |= !lk.blocked(P.plink[e], st);
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
    if (bad) g.store(&K->fault, bad);
    clk.lap(5);
    g.sync();
    clk.lap(6);
    if (threadIdx.x == 0) {
      rounds += 1;
      fsw += n;
    }
    if (g.aborted()) return ST_BARRIER;
    const int nout = g.load(out_cnt);
    if (g.load(&K->fault) != 0) { rc = g.load(&K->fault) == 2 ? ST_OVERFLOW : ST_BAD_SHARE; break; }
    if (nout == 0) break;
    if (nout >= n) { rc = ST_BAD_SHARE; break; }  // a round must freeze something
    if (++r > P.max_rounds) { rc = ST_ROUNDS; break; }
    in = out;
    n = nout;
  }
  if (tid == 0) g.store(&K->stamp, st0 + (uint32_t)r);
  return rc;
}

// ---------------------------------------- one workgroup, unfrozen set as bit masks
// Path records and ids of the first `cap` flows of a solve, in shared memory.
struct FlowCache {
  uint4* path;
  int32_t* fid;
  int cap;
};

// Active flows live in slots: per part, the flow id, predicted completion
// time tau and rate of every active flow (see the event loop).
struct Slots {
  int32_t* id;
  double* tau;
  double* rate;
};

// An incremental re-solve of the flows list[0..n): item i sits in slot at[i];
// slots at or above s_new were activated at this event and hold no rate yet.
// Before solving, each flow's contribution is taken back from its links and
// its remaining bytes are brought up to time t; after solving, its slot gets
// the new rate and predicted completion.
struct Resel {
  Slots sl;
  const int32_t* at;
  int s_new;
  double t;
};

// Remaining bytes at t of a flow that had rem at tref and ran at rate r
// (the same roundings in every solve variant: nothing is contracted).
__device__ __forceinline__ double rem_at(double rem, double r, double t, double tref) {
  const double moved = r * (t - tref);
  return rem - moved;
}

// Bit k set for every item t + k*T < n of this thread (k < 64).
__device__ __forceinline__ uint64_t low_items(int n, int T) {
  const int t = threadIdx.x;
  const int c = n > t ? (n - t - 1) / T + 1 : 0;
  return c >= 64 ? ~0ull : (1ull << c) - 1ull;
}

// Calls body(k, i, cached, rec) for every item k set in `mask` (item
// i = t + k*T) with its path record: from the shared-memory cache for the
// items in cmask, from the item-indexed staging buffer for the others.  The
// records of four items are loaded before the first of them is processed,
// so their latencies overlap.  Two separate loops, so that the two kinds of
// read are never merged into one access through a generic pointer.
template <class Body>
__device__ __forceinline__ void for_items(uint64_t mask, uint64_t cmask, const FlowCache& fc,
                                          const uint4* stg, int T, Body body) {
  for (uint64_t m = mask & cmask; m;) {
    int k[4];
    uint4 r[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      k[u] = m ? __ffsll((unsigned long long)m) - 1 : -1;
      m &= m - 1;
      if (k[u] >= 0) r[u] = fc.path[(int)threadIdx.x + k[u] * T];
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (k[u] >= 0) body(k[u], (int)threadIdx.x + k[u] * T, true, r[u]);
  }
  for (uint64_t m = mask & ~cmask; m;) {
    int k[4];
    uint4 r[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      k[u] = m ? __ffsll((unsigned long long)m) - 1 : -1;
      m &= m - 1;
      if (k[u] >= 0) r[u] = stg[(int)threadIdx.x + k[u] * T];
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (k[u] >= 0) body(k[u], (int)threadIdx.x + k[u] * T, false, r[u]);
  }
}

// Thread t of the workgroup owns the flows list[t + k*T], k < 64, and keeps
// which of them are still unfrozen as a 64-bit mask, so a round needs no list
// compaction: the workgroup barriers, the path reads (one 16-byte record per
// flow: from the shared-memory cache for the first fc.cap items, from the
// staging buffer P.stage, indexed by item, for the rest; both filled once per
// solve), the link-state gathers and the freezing atomics.  With a share
// table the smallest share of a frozen flow is read again from the table in
// phase C (the table does not change within a round).  With rs, the
// re-solve's take-back is done while the records are gathered and the slots
// are written as flows freeze.  Paths must fit the record (<= 6 links,
// part-local ids below 0xFFFF); n <= 64*T.
template <class LK>
__device__ __forceinline__ int solve_mask(BlockG& g, const Params& P, LK& lk, ScenCtl* C,
                                          const int32_t* list, int n, int64_t& rounds, int64_t& fsw,
                                          int64_t& isw, Clock& clk, bool warm, const FlowCache& fc,
                                          const Resel* rs) {
  Lists* K = g.lists(C);
  const int T = blockDim.x;
  const int l0 = C->l0;
  const int f0 = C->f0, cap = C->f1 - C->f0;
  uint4* stg = P.stage + f0;
  double* mfi = P.mf + f0;  // smallest share per item (link state without a table)
  const int lsent = C->l1;  // the sentinel's id (link state with a table)
  int* cntr = g.ldsi + 112;  // three rotating counters of unfrozen flows
  int bad = 0;
  if (!warm) cold_links(g, P, lk, C);
  const uint64_t alive0 = low_items(n, T);
  uint64_t alive = alive0;
  const int nc = min(n, fc.cap);
  const uint64_t cmask = low_items(nc, T);  // items served from the cache
  // gather: ids, path records (and, re-solving, the rates and remaining
  // bytes to take back), four items of a thread in flight at a time
  for (int j0 = 0; j0 * T < n; j0 += 4) {
    int fv[4], sv[4];
    uint4 rv[4];
    double rr[4], tr[4], rm[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = (int)threadIdx.x + (j0 + u) * T;
      fv[u] = i < n ? list[i] : f0;
      sv[u] = (rs && i < n) ? rs->at[i] : 0;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = (int)threadIdx.x + (j0 + u) * T;
      const bool ok = i < n && in_range(fv[u], f0, cap) && (unsigned)sv[u] < (unsigned)cap;
      rv[u] = ok ? P.path16[fv[u]] : make_uint4(~0u, ~0u, ~0u, ~0u);
      if (rs && ok && sv[u] < rs->s_new) {
        rr[u] = rs->sl.rate[sv[u]];
        tr[u] = P.tref[fv[u]];
        rm[u] = P.rem[fv[u]];
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = (int)threadIdx.x + (j0 + u) * T;
      if (i >= n) continue;
      const int f = fv[u];
      if (!in_range(f, f0, cap) || (unsigned)sv[u] >= (unsigned)cap) bad = 2;
      if (i < nc) {
        fc.fid[i] = f;
        fc.path[i] = rv[u];
      } else {
        stg[i] = rv[u];
      }
      if (rs && in_range(f, f0, cap)) {
        const bool fresh = sv[u] >= rs->s_new;
        int lv[6];
        const int deg = unpack_path(rv[u], l0, lv);
        int64_t qv = 0;
        if (!fresh) {
          P.rem[f] = rem_at(rm[u], rr[u], rs->t, tr[u]);
          P.tref[f] = rs->t;
          qv = (int64_t)__builtin_rint(rr[u] * P.scale);
        }
#pragma unroll
        for (int j = 0; j < 6; ++j)
          if (j < deg) {
            if (!fresh) lk.addR(g, lv[j], qv);
            lk.addN(g, lv[j], (int64_t)1);
          }
      }
    }
  }
  if (threadIdx.x < 3) cntr[threadIdx.x] = 0;
  if (bad) g.store(&K->fault, bad);
  __syncthreads();
  const uint32_t st0 = first_round(g, P, lk, C);
  clk.lap(2);
  int total = n;
  int r = 0;
  int rc = 0;
  if (g.load(&K->fault) != 0) rc = ST_OVERFLOW;
  for (; rc == 0;) {
    const uint32_t st = st0 + (uint32_t)r;
    if (threadIdx.x == 0) cntr[(r + 1) % 3] = 0;
    round_table(g, lk, C);
    clk.lap(2);
    // phase B: smallest share on each path; block links above it.  The
    // record's spare word keeps which of the flow's links are at its
    // minimum: the others carry its own stamp, so phase C looks only at those
    for_items(alive, cmask, fc, stg, T, [&](int, int i, bool cached, uint4 rec) {
      int lv[6];
      const int deg = unpack_path(rec, l0, lv);
      isw += deg;
      uint32_t cm = 0;
      if constexpr (LK::kTable) {
        // six unguarded gathers (absent links read the sentinel's +inf),
        // all in flight before the first is used
        double sv[6];
#pragma unroll
        for (int k = 0; k < 6; ++k) {
          lv[k] = min(lv[k], lsent);
          sv[k] = lk.table(lv[k]);
        }
        double m = sv[0];
#pragma unroll
        for (int k = 1; k < 6; ++k) m = sv[k] < m ? sv[k] : m;
        const double thr = m * THR;
#pragma unroll
        for (int k = 0; k < 6; ++k) {
          if (!(sv[k] > thr)) cm |= 1u << k;
          else if (sv[k] < INF) lk.block(lv[k], st);
        }
        if (!(m > 0.0) || !(m < INF)) bad = 1;
      } else {
        mfi[i] = share_and_block(lk, lv, deg, st, bad, &cm);
      }
      if (cached) fc.path[i].w = cm;
      else reinterpret_cast<uint32_t*>(stg + i)[3] = cm;
    });
    clk.lap(3);
    __syncthreads();
    clk.lap(4);
    // phase C: freeze flows crossing an unblocked link
    uint64_t frozen_mask = 0;
    for_items(alive, cmask, fc, stg, T, [&](int k, int i, bool cached, uint4 rec) {
      int lv[6];
      const int deg = unpack_path(rec, l0, lv);
      const uint32_t cm = rec.w;
      bool frozen = false;
      double mv;
      if constexpr (LK::kTable) {
        // only the links at the flow's minimum (usually one): a stamp tells
        // whether it is blocked, the table the share it freezes at
        mv = INF;
        for (uint32_t rest = cm; rest; rest &= rest - 1) {
          const int j = __ffs(rest) - 1;
          const int l = j == 0 ? lv[0] : j == 1 ? lv[1] : j == 2 ? lv[2]
                      : j == 3 ? lv[3] : j == 4 ? lv[4] : lv[5];
          frozen |= lk.stamp(l) != st;
          const double sv = lk.table(l);
          mv = sv < mv ? sv : mv;
        }
        if (!frozen) return;
      } else {
#pragma unroll
        for (int j = 0; j < 6; ++j)
          if (j < deg && ((cm >> j) & 1u)) frozen |= !lk.blocked(lv[j], st);
        if (!frozen) return;
        mv = mfi[i];
      }
      if constexpr (LK::kTable) mfi[i] = mv;  // the rate, by item (written out after the rounds)
      const int64_t qv = (int64_t)__builtin_rint(mv * P.scale);
#pragma unroll
      for (int j = 0; j < 6; ++j)
        if (j < deg) {
          lk.addR(g, lv[j], -qv);
          lk.addN(g, lv[j], (int64_t)-1);
        }
      frozen_mask |= 1ull << k;
    });
    alive &= ~frozen_mask;
    int c = __popcll(alive);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o, 64);
    if (lane_id() == 0 && c > 0) atomicAdd(&cntr[r % 3], c);
    if (bad) g.store(&K->fault, bad);
    clk.lap(5);
    __syncthreads();
    clk.lap(6);
    if (threadIdx.x == 0) {
      rounds += 1;
      fsw += total;
    }
    if (g.load(&K->fault) != 0) { rc = g.load(&K->fault) == 2 ? ST_OVERFLOW : ST_BAD_SHARE; break; }
    const int left = cntr[r % 3];
    if (left == 0) break;
    if (left >= total) { rc = ST_BAD_SHARE; break; }  // a round must freeze something
    if (++r > P.max_rounds) { rc = ST_ROUNDS; break; }
    total = left;
  }
  if (threadIdx.x == 0) g.store(&K->stamp, st0 + (uint32_t)r);
  if (rc == 0) {
    // rates by flow (and, re-solving, the slots' rates and predicted
    // completions), four items of a thread in flight at a time
    for (int j0 = 0; j0 * T < n; j0 += 4) {
      int fv[4], sv[4];
      double mv[4], rm[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = (int)threadIdx.x + (j0 + u) * T;
        if (i < n) {
          fv[u] = i < nc ? fc.fid[i] : list[i];
          mv[u] = mfi[i];
          sv[u] = rs ? rs->at[i] : 0;
        }
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = (int)threadIdx.x + (j0 + u) * T;
        if (i < n && rs) rm[u] = P.rem[fv[u]];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = (int)threadIdx.x + (j0 + u) * T;
        if (i >= n) continue;
        P.rate[fv[u]] = mv[u];
        if (rs) {
          rs->sl.rate[sv[u]] = mv[u];
          rs->sl.tau[sv[u]] = rs->t + rm[u] / mv[u];
        }
      }
    }
  }
  return rc;
}

// The take-back of an incremental re-solve (see Resel) as a pass of its
// own, for the solve variants that do not fuse it: any group, any path.
template <class G, class LK>
__device__ __forceinline__ void take_back(G& g, const Params& P, LK& lk, const int32_t* list, int n,
                                          const Resel& rs, int f0, int cap, int& err) {
  for (int j = g.tid(); j < n; j += g.nthr()) {
    const int f = list[j];
    const int s = rs.at[j];
    if (!in_range(f, f0, cap) || (unsigned)s >= (unsigned)cap) { err = 1; continue; }
    const bool fresh = s >= rs.s_new;
    int64_t qv = 0;
    if (!fresh) {
      const double r = rs.sl.rate[s];
      P.rem[f] = rem_at(P.rem[f], r, rs.t, P.tref[f]);
      P.tref[f] = rs.t;
      qv = (int64_t)__builtin_rint(r * P.scale);
    }
    for (int k = P.poff[f]; k < P.poff[f + 1]; ++k) {
      const int l = P.plink[k];
      if (!fresh) lk.addR(g, l, qv);
      lk.addN(g, l, (int64_t)1);
    }
  }
}

// ---------------------------------------------- shared-memory-resident solve
// Grid layout: each workgroup takes every nb-th flow of the active list (at
// most LDS_FLOWS flows), copies the flow ids and their path records into
// shared memory once, and keeps its unfrozen flows as a shared-memory list.
// Only link state and the rates are touched outside, so a round costs one
// gather of link state, one of stamps and two grid barriers.
constexpr int LDS_FLOWS = 3840;

struct SolveLds {
  int32_t fid[LDS_FLOWS];
  uint4 path[LDS_FLOWS];
  double mf[LDS_FLOWS];
  uint16_t u[2][LDS_FLOWS];
  int cnt;
  int anybad;  // some thread of the workgroup met a fault (cluster helpers)
};

// A helper's update of link l (residual r, unfrozen count c): into its
// shared-memory deltas when it has them (dR non-null, uniform over the
// workgroup), else straight into the link state.
template <class G, class LK>
__device__ __forceinline__ void link_add(G& g, LK& lk, int64_t* dR, int32_t* dn, int l0, int l, int64_t r,
                                         int32_t c, bool with_r) {
  if (dR) {
    if (with_r) __hip_atomic_fetch_add(&dR[l - l0], r, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    __hip_atomic_fetch_add(&dn[l - l0], c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  } else {
    if (with_r) lk.addR(g, l, r);
    lk.addN(g, l, (int64_t)c);
  }
}

// Folds a helper's deltas into the link state (one atomic per link and
// field it changed, instead of one per flow and link) and clears them.
// Integer sums: the link state ends bit-identical to per-flow updates.
// Follows a workgroup barrier after the last delta update.
template <class G, class LK>
__device__ __forceinline__ void fold_deltas(G& g, LK& lk, int64_t* dR, int32_t* dn, int l0, int nl) {
  for (int i = threadIdx.x; i < nl; i += blockDim.x) {
    const int64_t r = dR[i];
    const int32_t c = dn[i];
    if (r != 0) {
      lk.addR(g, l0 + i, r);
      dR[i] = 0;
    }
    if (c != 0) {
      lk.addN(g, l0 + i, (int64_t)c);
      dn[i] = 0;
    }
  }
}

template <class G, class LK>
__device__ __forceinline__ int solve_lds(G& g, const Params& P, LK& lk, ScenCtl* C, const int32_t* list0,
                                         int n0, int64_t& rounds, int64_t& fsw, int64_t& isw, Clock& clk,
                                         SolveLds& S, bool warm, const Resel* rs = nullptr) {
  Lists* K = g.lists(C);
  const int tid = g.tid();
  const int nb = g.nblocks();
  // items b, b + nb, b + 2nb, ... of the list: interleaved, so every
  // workgroup keeps a like share of unfrozen flows through the rounds (the
  // list follows activation order, and contiguous slices freeze unevenly)
  const int b0 = g.block_id();
  const int nl = b0 < n0 ? (n0 - 1 - b0) / nb + 1 : 0;
  const int l0 = C->l0;
  const int cap = C->f1 - C->f0;
  int* bc = g.ldsi + 120;  // counters read by thread 0 after a barrier, for the block
  if (!warm) cold_links(g, P, lk, C);
  if (tid == 0)
    for (int k = 0; k < 3; ++k) g.store(&K->rem3[k], 0);
  // a helper whose part's links fit its delta arrays updates link state
  // through them (folded before each barrier)
  const int nlk = C->l1 - C->l0;
  int64_t* dR = nullptr;
  int32_t* dn = nullptr;
  if constexpr (IsCluster<G>::value) {
    if (threadIdx.x == 0) S.anybad = 0;
    if (nlk <= g.dcap) {
      dR = g.dR;
      dn = g.dn;
      for (int i = threadIdx.x; i < nlk; i += blockDim.x) {
        dR[i] = 0;
        dn[i] = 0;
      }
    }
    __syncthreads();
  }
  int bad = 0;
  // ids and path records into shared memory; re-solving (rs), each flow's
  // take-back too: remaining bytes brought up to rs->t, its rate and one
  // unfrozen flow returned to its links
  for (int j = threadIdx.x; j < nl; j += blockDim.x) {
    int f = list0[b0 + j * nb];
    const bool ok = in_range(f, C->f0, cap);
    if (!ok) { bad = 2; f = C->f0; }
    const uint4 rec = P.path16[f];
    S.fid[j] = f;
    S.path[j] = rec;
    S.u[0][j] = (uint16_t)j;
    if (rs && ok) {
      const int sl = rs->at[b0 + j * nb];
      if ((unsigned)sl >= (unsigned)cap) { bad = 2; continue; }
      const bool fresh = sl >= rs->s_new;
      int64_t qv = 0;
      if (!fresh) {
        const double rt = rs->sl.rate[sl];
        P.rem[f] = rem_at(P.rem[f], rt, rs->t, P.tref[f]);
        P.tref[f] = rs->t;
        qv = (int64_t)__builtin_rint(rt * P.scale);
      }
      int lv[6];
      const int deg = unpack_path(rec, l0, lv);
#pragma unroll
      for (int k = 0; k < 6; ++k)
        if (k < deg) link_add(g, lk, dR, dn, l0, lv[k], qv, 1, !fresh);
    }
  }
  int nu = nl;
  if (bad) g.store(&K->fault, bad);
  if constexpr (IsCluster<G>::value) {
    if (bad) S.anybad = 1;
    if (dR) {
      __syncthreads();
      fold_deltas(g, lk, dR, dn, l0, nlk);
    }
  }
  g.sync();
  const uint32_t st0 = first_round(g, P, lk, C);
  clk.lap(2);
  int total = n0;
  int r = 0;
  int rc = 0;
  for (;;) {
    const uint32_t st = st0 + (uint32_t)r;
    const uint16_t* uin = S.u[r & 1];
    uint16_t* uout = S.u[(r & 1) ^ 1];
    if (threadIdx.x == 0) S.cnt = 0;
    if constexpr (!IsCluster<G>::value)
      if (tid == 0) g.store(&K->rem3[(r + 1) % 3], 0);
    round_table(g, lk, C);
    clk.lap(2);
    // phase B: smallest share on each path; block links above it
    for (int x = threadIdx.x; x < nu; x += blockDim.x) {
      const int j = uin[x];
      int lv[6];
      const int deg = unpack_path(S.path[j], l0, lv);
      isw += deg;
      S.mf[j] = share_and_block(lk, lv, deg, st, bad);
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
        int lv[6];
        const int deg = unpack_path(S.path[j], l0, lv);
        bool frozen = false;
#pragma unroll
        for (int k = 0; k < 6; ++k)
          if (k < deg) frozen |= !lk.blocked(lv[k], st);
        if (frozen) {
          const double m = S.mf[j];
          P.rate[S.fid[j]] = m;
          const int64_t qv = (int64_t)__builtin_rint(m * P.scale);
#pragma unroll
          for (int k = 0; k < 6; ++k)
            if (k < deg) link_add(g, lk, dR, dn, l0, lv[k], -qv, -1, true);
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
    if (bad) g.store(&K->fault, bad);
    int ft, left;
    int nu_new;
    if constexpr (IsCluster<G>::value) {
      // the unfrozen count and a fault bit travel with the barrier's arrival
      if (bad) S.anybad = 1;
      __syncthreads();
      nu_new = S.cnt;
      if (dR) fold_deltas(g, lk, dR, dn, l0, nlk);
      clk.lap(5);
      const uint32_t res = g.sync_sum((uint32_t)nu_new | (S.anybad ? 0x80000000u : 0u));
      clk.lap(6);
      if (threadIdx.x == 0) {
        rounds += 1;
        fsw += total;
      }
      if (g.aborted()) return ST_BARRIER;
      ft = 0;
      if (res & 0x80000000u) {  // some helper met a fault: which one
        if (threadIdx.x == 0) bc[0] = g.load(&K->fault);
        __syncthreads();
        ft = bc[0];
      }
      left = (int)(res & 0x7FFFFFFFu);
    } else {
      __syncthreads();
      nu_new = S.cnt;
      if (threadIdx.x == 0 && nu_new > 0) g.add(&K->rem3[r % 3], (int32_t)nu_new);
      clk.lap(5);
      g.sync();
      clk.lap(6);
      if (threadIdx.x == 0) {
        rounds += 1;
        fsw += total;
      }
      if (g.aborted()) return ST_BARRIER;
      // one read of the two counters per workgroup, shared through shared memory
      if (threadIdx.x == 0) {
        bc[0] = g.load(&K->fault);
        bc[1] = g.load(&K->rem3[r % 3]);
      }
      __syncthreads();
      ft = bc[0];
      left = bc[1];
    }
    if (ft != 0) { rc = ft == 2 ? ST_OVERFLOW : ST_BAD_SHARE; break; }
    if (left == 0) break;
    if (left >= total) { rc = ST_BAD_SHARE; break; }  // a round must freeze something
    if (++r > P.max_rounds) { rc = ST_ROUNDS; break; }
    total = left;
    nu = nu_new;
  }
  if (tid == 0) g.store(&K->stamp, st0 + (uint32_t)r);
  if (rs && rc == 0) {
    // each re-solved flow's slot: its rate (the share it froze at) and
    // predicted completion, by the thread that took it back
    for (int j = threadIdx.x; j < nl; j += blockDim.x) {
      const int f = S.fid[j];
      const int sl = rs->at[b0 + j * nb];
      if ((unsigned)sl >= (unsigned)cap) continue;
      const double m = S.mf[j];
      rs->sl.rate[sl] = m;
      rs->sl.tau[sl] = rs->t + P.rem[f] / m;
    }
  }
  return rc;
}

// ------------------------------------------------- helper workgroups (cluster kernel)
// A leader without helpers.
struct NoAssist {
  static constexpr bool kOn = false;
};

// A leader's side of its XCD's helpers: a large re-solve is posted as a job;
// the helpers take the flows back, run solve_lds over link state in global
// memory and write the rates by flow and the slots (rate, predicted
// completion), as the fused block solve does.  A leader whose link
// state lives in shared memory copies residual capacities and unfrozen
// counts out before and back after (their stamps are a separate sequence
// in global memory: C->k.stamp over Params::fl); one whose state is global
// hands over its stamp counter instead, so both sides number rounds in one
// sequence over the one stamp array.  Only thread 0 touches the mailbox.
struct Assist {
  static constexpr bool kOn = true;
  uint32_t* bar;
  uint32_t* cw;   // this XCD's cluster words
  int nh;         // helper workgroups
  int min_n;      // smallest solve handed over
  uint32_t seq;   // jobs posted so far (every thread keeps the same value)
  int* box;       // shared memory [2]: result broadcast
  __device__ bool takes(int n) const { return nh > 0 && n >= min_n && n <= nh * LDS_FLOWS; }

  // Re-solve of the part's list of n flows (the event loop's re-solve list
  // and the slot of each in slot buffer ab; slots from s_new on were
  // activated at time t): the job's status, or NOT_TAKEN if the helpers
  // have left (nothing changed then).
  template <class LK>
  __device__ __forceinline__ int solve(BlockG& g, const Params& P, LK& lk, ScenCtl* C, int sc, int n,
                                       int ab, int s_new, double t, int64_t& rounds, int64_t& fsw,
                                       int64_t& isw) {
    const int T = blockDim.x;
    const int l0 = C->l0, nl = C->l1 - C->l0;
    if constexpr (LK::kTable) {
      // agent-scope stores, as the helpers' updates of these words are
      for (int i = threadIdx.x; i < nl; i += T) {
        __hip_atomic_store(&P.lst[2 * (l0 + i)], lk.R[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(&P.lst[2 * (l0 + i) + 1], (int64_t)lk.n[i], __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    xcd_release(P.debug & DEBUG_FORMAL_RELEASE);
    __syncthreads();
    if (threadIdx.x == 0) {
      int res = NOT_TAKEN, posted = 0;
      if constexpr (!LK::kTable)
        __hip_atomic_store(&C->k.stamp, g.lst->stamp, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&cw[CL_SC], (uint32_t)sc, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&cw[CL_N], (uint32_t)n, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&cw[CL_AB], (uint32_t)ab, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&cw[CL_SNEW], (uint32_t)s_new, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(reinterpret_cast<uint64_t*>(cw + CL_T), (uint64_t)__double_as_longlong(t),
                         __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      // the job's words must be performed before the post that publishes
      // them (a helper that sees the new count reads them next).  Link state
      // in global memory was last updated by this workgroup's
      // workgroup-scope atomics: a full agent-scope release (an L2
      // write-back) puts it where the helpers' agent-scope atomics act on it
      // and covers the job's words too; a copied-out state was stored at
      // agent scope and is drained already, so the job's words need only
      // their own drain
      if constexpr (!LK::kTable) __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
      else xcd_release(P.debug & DEBUG_FORMAL_RELEASE);
      uint32_t expect = seq;
      if (__hip_atomic_compare_exchange_strong(&cw[CL_MB], &expect, seq + 1, __ATOMIC_RELAXED,
                                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
        posted = 1;
        const uint32_t want = (seq + 1) * (uint32_t)nh;
        const uint64_t t0 = wall_clock64();
        bool ok = true;
        while (__hip_atomic_load(&cw[CL_DONE], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != want) {
          __builtin_amdgcn_s_sleep(2);
          if (__hip_atomic_load(&bar[BAR_ABORT], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0 ||
              wall_clock64() - t0 > IDLE_TICKS) {
            __hip_atomic_store(&bar[BAR_ABORT], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            ok = false;
            break;
          }
        }
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        // a helper that gave up at a barrier raised the abort word before it
        // counted itself done, even if the others finished the job without it
        if (ok && __hip_atomic_load(&bar[BAR_ABORT], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0)
          ok = false;
        if (ok) {
          res = (int)__hip_atomic_load(&cw[CL_RC], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          auto w64 = [&](int k) { return reinterpret_cast<uint64_t*>(cw + k); };
          rounds += (int64_t)__hip_atomic_load(w64(CL_ROUNDS), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          fsw += (int64_t)__hip_atomic_load(w64(CL_FSW), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          isw += (int64_t)__hip_atomic_load(w64(CL_ISW), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          __hip_atomic_store(w64(CL_ISW), (uint64_t)0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          if constexpr (!LK::kTable)
            g.lst->stamp = __hip_atomic_load(&C->k.stamp, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        } else {
          res = ST_BARRIER;
        }
      }
      box[0] = res;
      box[1] = posted;
    }
    __syncthreads();
    const int res = box[0];
    seq += (uint32_t)box[1];
    if constexpr (LK::kTable) {
      if (res != NOT_TAKEN)
        for (int i = threadIdx.x; i < nl; i += T) {
          lk.R[i] = P.lst[2 * (l0 + i)];
          lk.n[i] = (int32_t)P.lst[2 * (l0 + i) + 1];
        }
    }
    __syncthreads();
    return res;
  }
};

// A helper workgroup: waits for its leader's jobs and solves them with the
// XCD's other helpers until the leader closes the mailbox, the launch aborts
// or no job comes for IDLE_TICKS (then it closes the mailbox itself, unless a
// job arrived meanwhile).
__device__ __forceinline__ void helper_loop(const Params& P, ClusterG& cg, SolveLds& S, Tally* tl,
                                            int* box, double* tjob) {
  uint32_t* cw = cg.cw;
  const uint64_t idle = (P.debug & DEBUG_HELPERS_LEAVE) ? 0 : IDLE_TICKS;
  uint32_t seen = 0;
  for (;;) {
    if (threadIdx.x == 0) {
      int leave = 0;
      uint32_t v = seen;
      const uint64_t t0 = wall_clock64();
      for (;;) {
        v = __hip_atomic_load(&cw[CL_MB], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (v != seen) break;
        if (__hip_atomic_load(&P.bar[BAR_ABORT], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0) {
          leave = 1;
          break;
        }
        if (wall_clock64() - t0 > idle) {
          uint32_t e = seen;
          if (__hip_atomic_compare_exchange_strong(&cw[CL_MB], &e, CL_CLOSED, __ATOMIC_RELAXED,
                                                   __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
            v = CL_CLOSED;
            break;
          }
        }
        __builtin_amdgcn_s_sleep(10);  // ~270 ns: 31 pollers stay light on the L2
      }
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
      if (leave)  // later posts must fail rather than wait for helpers that left
        __hip_atomic_exchange(&cw[CL_MB], CL_CLOSED, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (leave || v == CL_CLOSED) {
        box[0] = -1;
      } else {
        box[0] = (int)__hip_atomic_load(&cw[CL_SC], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        box[1] = (int)__hip_atomic_load(&cw[CL_N], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        box[2] = (int)v;
        box[3] = (int)__hip_atomic_load(&cw[CL_AB], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        box[4] = (int)__hip_atomic_load(&cw[CL_SNEW], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        tjob[0] = __longlong_as_double((long long)__hip_atomic_load(
            reinterpret_cast<uint64_t*>(cw + CL_T), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
      }
    }
    __syncthreads();
    const int sc = box[0], n = box[1], ab = box[3], s_new = box[4];
    const double t = tjob[0];
    seen = (uint32_t)box[2];
    __syncthreads();
    if (sc < 0) break;
    int rc = ST_OVERFLOW;
    int64_t rr = 0, ff = 0, is = 0;
    // the same job for every helper: all of them solve it or none does
    if (sc < P.num_scen && n > 0 && n <= cg.nh * LDS_FLOWS && n <= P.ctl[sc].f1 - P.ctl[sc].f0 &&
        P.ctl[sc].lds_paths && (ab == 0 || ab == 1) && s_new >= 0 &&
        s_new <= P.ctl[sc].f1 - P.ctl[sc].f0) {
      ScenCtl* C = &P.ctl[sc];
      const int f0 = C->f0;
      const Slots sl = ab ? Slots{P.act1 + f0, P.tau1 + f0, P.srate1 + f0}
                          : Slots{P.act0 + f0, P.tau0 + f0, P.srate0 + f0};
      const Resel rs{sl, P.arrslot + f0, s_new, t};
      LinksGlobal lk{P.lst, P.nact, P.fl, P.inv_scale};
      // the first helper times the job's phases (debug bit 1) for its leader
      Clock clk((P.debug & 2) && cg.rank == 0 && threadIdx.x == 0, tl->clk);
      rc = solve_lds(cg, P, lk, C, P.arr + f0, n, rr, ff, is, clk, S, true, &rs);
    }
    long w = (long)is;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) w += __shfl_xor(w, o, 64);
    if (lane_id() == 0 && w != 0)
      __hip_atomic_fetch_add(reinterpret_cast<uint64_t*>(cw + CL_ISW), (uint64_t)w, __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
    if (cg.rank == 0 && threadIdx.x == 0) {
      if (P.debug & 2)
        for (int k = 2; k < 7; ++k)
          __hip_atomic_store(reinterpret_cast<uint64_t*>(cw + CL_CLK) + k, tl->clk[k], __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&cw[CL_RC], (uint32_t)rc, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(reinterpret_cast<uint64_t*>(cw + CL_ROUNDS), (uint64_t)rr, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(reinterpret_cast<uint64_t*>(cw + CL_FSW), (uint64_t)ff, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    }
    xcd_release(P.debug & DEBUG_FORMAL_RELEASE);
    __syncthreads();
    if (threadIdx.x == 0)  // drained above: rates and statistics are in the XCD's L2
      __hip_atomic_fetch_add(&cw[CL_DONE], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
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
// their bits.  theta is kept per link component (flows of different
// components share no link).
//
// Active flows live in slots: per part, the flow id, predicted completion
// time tau and rate of every active flow, in two buffers used alternately
// across compactions.  Remaining bytes are kept lazily: rem[f] is the value
// at time tref[f], brought up to date (rem - rate * elapsed) only when the
// flow's rate is re-solved, after which tau = t + rem / rate.  So an event
// reads a kept flow's tau (next-event search) and rate (re-solve selection)
// and writes nothing for it.  A finished flow leaves a hole (id -1, tau
// +inf); when holes are more than an eighth of the slots, the live ones are
// compacted into the other buffer.
constexpr double KEEP = 1.0 - 1e-9;  // safety margin below theta

// Flow f becomes active at time t: remaining bytes, active counts on its
// links, a new slot (tau set after its first solve) and the arrivals list.
template <bool HIST, class G, class LK>
__device__ __forceinline__ void activate(G& g, const Params& P, LK& lk, Lists* K, int f, double t,
                                         const Slots& sl, int32_t* arrOut, int ib, int cap,
                                         int ev, int& err) {
  P.rem[f] = P.nbytes[f];
  P.tref[f] = t;
  if constexpr (HIST) P.eva[f] = ev;
  for (int j = P.poff[f]; j < P.poff[f + 1]; ++j) lk.addNact(g, P.plink[j], 1);
  const int s = g.add(&K->slots, 1);
  if (s < cap) {
    sl.id[s] = f;
    sl.tau[s] = INF;
    sl.rate[s] = 0.0;
  } else {
    err = 1;
  }
  const int a = g.add(&K->arr, 1);
  if (a < cap) arrOut[a] = f; else err = 1;
  g.store(&K->changed[ib], 1);
}

// Releases flow h at event time t, once its predecessors have all finished,
// the latest of them at `base` (>= t) (called once per h).
template <bool HIST, class G, class LK>
__device__ __forceinline__ void release_one(G& g, const Params& P, LK& lk, Lists* K, int h, double t,
                                            double base, int ob, int ib, const Slots& sl,
                                            int32_t* pendOut, int32_t* arrOut, int32_t* cout,
                                            int32_t* coutCnt, int cap, int ev, int& err) {
  const double rl = P.start[h] + base;
  P.base[h] = base;
  P.rel[h] = rl;
  if constexpr (HIST) P.evr[h] = ev;
  if (rl <= t) {
    if (P.nbytes[h] == 0.0) {
      P.finish[h] = rl;
      if constexpr (HIST) {
        P.eva[h] = ev;
        P.evd[h] = ev;
      }
      const int s = g.add(coutCnt, 1);
      if (s < cap) cout[s] = h; else err = 1;
    } else {
      activate<HIST>(g, P, lk, K, h, t, sl, arrOut, ib, cap, ev, err);
    }
  } else {
    const int s = g.add(&K->pend[ob], 1);
    if (s < cap) pendOut[s] = h; else err = 1;
  }
}

// HIST: keep the rollback history (per-flow event indices, undo and event
// records); the cluster kernel is built without it.
template <bool HIST, class G, class LK, class AS = NoAssist>
__device__ __forceinline__ void event_loop(G& g, const Params& P, LK& lk, const int sc, SolveLds* S,
                                           Tally* tl, const FlowCache& fc, AS* as = nullptr) {
  ScenCtl* C = &P.ctl[sc];
  Lists* K = g.lists(C);
  const int f0 = C->f0;
  const int cap = C->f1 - C->f0;
  // alternating arrays, picked with selects (not runtime-indexed arrays,
  // which would hide that they live in global memory)
  auto slots = [&](int b) {
    return b ? Slots{P.act1 + f0, P.tau1 + f0, P.srate1 + f0} : Slots{P.act0 + f0, P.tau0 + f0, P.srate0 + f0};
  };
  auto pend = [&](int k) { return k ? P.pend1 + f0 : P.pend0 + f0; };
  auto comp = [&](int k) { return k == 0 ? P.comp0 + f0 : k == 1 ? P.comp1 + f0 : P.comp2 + f0; };
  int32_t* unf_a = P.unf0 + f0;
  int32_t* unf_b = P.unf1 + f0;
  int32_t* arrs = P.arr + f0;
  int32_t* arrSlot = P.arrslot + f0;
  const int T = g.nthr();
  const int tid = g.tid();
  const int w0 = tid - lane_id();
  Clock clk(tid == 0 && (P.debug & 2), tl->clk);
  const bool resume = P.resume && C->started;
  if (threadIdx.x == 0) {
    // statistics accumulate over the launches that continue a part
    tl->solves = resume ? C->solves : 0;
    tl->rounds = resume ? C->rounds : 0;
    tl->fsw = resume ? C->flows_swept : 0;
    tl->asw = resume ? C->active_swept : 0;
    tl->psw = resume ? C->pending_swept : 0;
    tl->sel = resume ? C->reselected : 0;
    tl->wide = resume ? C->wide_solves : 0;
    tl->asst = resume ? C->assisted : 0;
    g.store(&K->lsw, (int64_t)0);  // this launch's share-table passes
  }
  int64_t& rounds = tl->rounds;
  int64_t& fsw = tl->fsw;
  // links at rest: nothing active; no component has changed yet
  for (int l = C->l0 + tid; l < C->l1; l += T) lk.reset(l, P.R0[l]);
  if constexpr (LK::kTable) {
    if (tid == 0) lk.set_sentinel(C->l1 - C->l0);
  }
  const uint64_t INF_BITS = (uint64_t)__double_as_longlong(INF);
  for (int c = C->c0 + tid; c < C->c0 + C->nc; c += T) P.theta[c] = INF_BITS;
  double t = resume ? C->t : 0.0;
  int64_t events = resume ? C->events : 0, isw = 0;
  const int64_t events0 = events;
  int ab = resume ? C->ab : 0;          // slot buffer in use
  int nSlots = resume ? C->nslots : 0;  // slots in use (flows or holes)
  int nPend = resume ? C->npend : C->n_pend0;
  int e = resume ? C->e : 0;  // event index: pend[e&1] is this event's pending list
  int q = resume ? C->q : 0;  // completion-list phase index (three rotating lists)
  int64_t hp = resume ? C->hpos : 0;  // undo records written (rollback history)
  const bool hist = HIST && P.hist != nullptr && C->hcap > 0;
  int status = ST_DONE;
  if (resume) {
    // link state of the active flows, rebuilt exactly (integer sums): every
    // active flow holds rint(rate * scale) of each of its links; all are frozen
    g.sync();
    const Slots s0 = slots(ab);
    for (int s = tid; s < nSlots; s += T) {
      const int f = s0.id[s];
      if (!in_range(f, f0, cap)) continue;
      const int64_t qv = (int64_t)__builtin_rint(s0.rate[s] * P.scale);
      for (int k = P.poff[f]; k < P.poff[f + 1]; ++k) {
        lk.addNact(g, P.plink[k], 1);
        lk.addR(g, P.plink[k], -qv);
      }
    }
    if (tid == 0) {
      g.store(&K->slots, nSlots);
      g.store(&K->holes, C->holes);
    }
  }
  g.sync();
  for (;;) {
    const int ib = e & 1, ob = ib ^ 1;
    const Slots sl = slots(ab);
    const int32_t* pendIn = pend(ib);
    int32_t* pendOut = pend(ob);
    if (tid == 0) {
      g.store(&K->pend[ob], 0);
      g.store(&K->changed[ib], 0);
      g.store(&K->succ_flag[ib], 0);
      g.store(&K->arr, 0);
      g.store(&K->sel, 0);
      g.store(&K->slots2, 0);
    }
    // next event time: earliest predicted completion or release (four
    // slots of a thread in flight at a time).  Each thread also keeps the
    // slot of its earliest completion and its second earliest time: when
    // only the earliest is due the thread finishes it without looking again.
    double mine = INF, mine2 = INF;
    int smin = 0;
    for (int s0 = tid; s0 < nSlots; s0 += 4 * T) {
      double v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int s = s0 + u * T;
        v[u] = s < nSlots ? sl.tau[s] : INF;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        if (v[u] < mine) {
          mine2 = mine;
          mine = v[u];
          smin = s0 + u * T;
        } else if (v[u] < mine2) {
          mine2 = v[u];
        }
      }
    }
    double loc = mine;
    for (int i = tid; i < nPend; i += T) {
      const int f = pendIn[i];
      if (!in_range(f, f0, cap)) { g.store(&K->fault, 2); continue; }
      const double rl = P.rel[f];
      loc = rl < loc ? rl : loc;
    }
    if (threadIdx.x == 0) {
      tl->asw += nSlots;
      tl->psw += nPend;
    }
    const double tn = g.min_all(loc);
    clk.lap(0);
    if (g.aborted()) { status = ST_BARRIER; break; }
    if (g.load(&K->fault) != 0) { status = ST_OVERFLOW; break; }
    if (!(tn < INF)) break;
    if ((P.max_events > 0 && events - events0 >= P.max_events) || tn > P.until) {
      status = ST_STOPPED;
      break;
    }
    events += 1;
    const double thr = tn * THR;
    const int slots0 = nSlots;  // slots at or above this one are activated in this event
    int32_t* compOut = comp(q % 3);
    int32_t* compCnt = &K->comp[q % 3];
    if (tid == 0) g.store(&K->comp[(q + 1) % 3], 0);
    int err = 0;
    // completions: only threads holding a slot that is due look at it
    auto finish_slot = [&](int s) {
      const int f = sl.id[s];
      if (!in_range(f, f0, cap)) { err = 1; return; }
      const double r = sl.rate[s];
      // the last byte leaves now; it arrives the path latency later
      P.finish[f] = P.lat ? tn + P.lat[f] : tn;
      if constexpr (HIST) P.evd[f] = e;
      g.amin(&P.theta[P.comp[f]], (uint64_t)__double_as_longlong(r));
      const int64_t qv = (int64_t)__builtin_rint(r * P.scale);
      for (int k = P.poff[f]; k < P.poff[f + 1]; ++k) {
        const int l = P.plink[k];
        lk.addNact(g, l, -1);
        lk.addR(g, l, qv);  // its share returns to the link
      }
      if (P.soff[f + 1] > P.soff[f]) g.store(&K->succ_flag[ib], 1);
      g.store(&K->changed[ib], 1);
      sl.id[s] = -1;
      sl.tau[s] = INF;
      g.add(&K->holes, 1);
      const int c = g.add(compCnt, 1);
      if (c < cap) compOut[c] = f; else err = 1;
    };
    if (mine <= thr && !(mine2 <= thr)) {
      finish_slot(smin);  // the thread's only due slot
    } else if (mine <= thr) {
      // several due slots: look at every slot again, four in flight
      for (int s0 = tid; s0 < nSlots; s0 += 4 * T) {
        double v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int s = s0 + u * T;
          v[u] = s < nSlots ? sl.tau[s] : INF;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
          if (v[u] <= thr) finish_slot(s0 + u * T);
      }
    }
    // releases due now
    {
      int32_t* const cnts[2] = {compCnt, &K->pend[ob]};
      sweep_append<2>(
          g, nPend, cnts,
          [&](int i) {
            FlowVal x;
            x.f = pendIn[i];
            if (in_range(x.f, f0, cap)) x.a = P.rel[x.f];
            return x;
          },
          [&](int i, const FlowVal& x, bool* pr) {
            const int f = x.f;
            if (!in_range(f, f0, cap)) { err = 1; return; }
            const double rl = x.a;
            if (rl <= tn) {
              if (P.nbytes[f] == 0.0) {
                pr[0] = true;
                P.finish[f] = rl;
                if constexpr (HIST) {
                  P.eva[f] = e;
                  P.evd[f] = e;
                }
                if (P.soff[f + 1] > P.soff[f]) g.store(&K->succ_flag[ib], 1);
              } else {
                activate<HIST>(g, P, lk, K, f, tn, sl, arrs, ib, cap, e, err);
              }
            } else {
              pr[1] = true;
            }
          },
          [&](int k, int slot, const FlowVal& x) {
            int32_t* out = k == 0 ? compOut : pendOut;
            if (slot < cap) out[slot] = x.f; else err = 1;
          });
    }
    if (err) g.store(&K->fault, 2);
    g.sync();
    t = tn;
    q += 1;
    // dependants of finished flows, to a fixpoint through zero-byte flows.
    // A lane releases the successors of its own finished flow when it has a
    // few; long successor lists (a barrier's) are shared by the whole wave.
    int nc = g.load(&K->succ_flag[ib]) ? g.load(&K->comp[(q - 1) % 3]) : 0;
    while (nc > 0) {
      const int32_t* cin = comp((q - 1) % 3);
      int32_t* cout = comp(q % 3);
      int32_t* coutCnt = &K->comp[q % 3];
      if (tid == 0) g.store(&K->comp[(q + 1) % 3], 0);
      // body(f, h) for every (finished flow, successor) pair, once
      auto for_succ = [&](auto body) {
        for (int i0 = w0; i0 < nc; i0 += T) {
          const int i = i0 + lane_id();
          int f = -1, k0 = 0, k1 = 0;
          if (i < nc) {
            f = cin[i];
            if (in_range(f, f0, cap)) {
              k0 = P.soff[f];
              k1 = P.soff[f + 1];
            } else {
              err = 1;
            }
          }
          const bool big = k1 - k0 > 8;
          if (!big)
            for (int k = k0; k < k1; ++k) body(f, P.succ[k]);
          uint64_t mask = __ballot(big);
          while (mask) {
            const int j = __ffsll((unsigned long long)mask) - 1;
            mask &= mask - 1;
            const int a = __shfl(k0, j, 64), z = __shfl(k1, j, 64), fj = __shfl(f, j, 64);
            for (int k = a + lane_id(); k < z; k += 64) body(fj, P.succ[k]);
          }
        }
      };
      if (P.lat) {
        // with latency, a dependant starts after the latest arrival among its
        // predecessors, which need not be the last one to send its last
        // byte: first every finished flow raises its dependants' base to its
        // finish, then (after a barrier) the counts drop and releases read it
        for_succ([&](int f, int h) {
          g.amax(reinterpret_cast<uint64_t*>(&P.base[h]), (uint64_t)__double_as_longlong(P.finish[f]));
        });
        g.sync();
        for_succ([&](int, int h) {
          if (g.add(&P.cnt[h], -1) == 1) {
            const double b = __longlong_as_double((long long)__hip_atomic_load(
                reinterpret_cast<uint64_t*>(&P.base[h]), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
            release_one<HIST>(g, P, lk, K, h, t, b, ob, ib, sl, pendOut, arrs, cout, coutCnt, cap, e, err);
          }
        });
      } else {
        // arrival = last byte: the last predecessor to finish is the latest
        for_succ([&](int, int h) {
          if (g.add(&P.cnt[h], -1) == 1)
            release_one<HIST>(g, P, lk, K, h, t, t, ob, ib, sl, pendOut, arrs, cout, coutCnt, cap, e, err);
        });
      }
      if (err) g.store(&K->fault, 2);
      g.sync();
      q += 1;
      nc = g.load(&K->comp[(q - 1) % 3]);
    }
    clk.lap(1);
    if (g.aborted()) { status = ST_BARRIER; break; }
    if (g.load(&K->fault) != 0) { status = ST_OVERFLOW; break; }
    nSlots = g.load(&K->slots);
    const int pNew = g.load(&K->pend[ob]);
    const int live = nSlots - g.load(&K->holes);
    if (g.load(&K->changed[ib]) && live > 0) {
      // theta of each component: below it every rate stays as it was.
      // Finished flows have fed it their rates; new flows feed the initial
      // share of their links.
      const int nArr = g.load(&K->arr);
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
      g.sync();
      // take back the flows at or above their component's theta (and the new
      // ones) for re-solving; their remaining bytes are brought up to date.
      // With a single link component theta is one value for the whole part.
      {
        const bool one_comp = C->nc == 1;
        const double theta1 = __longlong_as_double((long long)g.load(&P.theta[C->c0]));
        int32_t* const cnts[1] = {&K->sel};
        sweep_append<1>(
            g, nSlots, cnts,
            [&](int s) {
              FlowVal x;
              x.k = s;
              x.f = sl.id[s];
              x.a = sl.rate[s];
              x.b = theta1;
              if (!one_comp && in_range(x.f, f0, cap))
                x.b = __longlong_as_double((long long)g.load(&P.theta[P.comp[x.f]]));
              return x;
            },
            [&](int s, const FlowVal& x, bool* pr) {
              const int f = x.f;
              if (f < 0) return;  // a hole
              if (!in_range(f, f0, cap)) { err = 1; return; }
              pr[0] = s >= slots0 || !(x.a < x.b * KEEP);
            },
            [&](int, int slot, const FlowVal& x) {
              if (slot < cap) {
                arrs[slot] = x.f;
                arrSlot[slot] = x.k;
                if (HIST && hist) {
                  // undo record: the flow's values before this event re-solves it
                  HistUndo u;
                  u.f = x.f;
                  u.ev = e;
                  u.rem = P.rem[x.f];
                  u.tref = P.tref[x.f];
                  u.rate = x.a;
                  P.hist[C->hbase + (hp + slot) % C->hcap] = u;
                }
              } else {
                err = 1;
              }
            });
      }
      if (err) g.store(&K->fault, 2);
      g.sync();
      clk.lap(7);
      for (int c = C->c0 + tid; c < C->c0 + C->nc; c += T) P.theta[c] = INF_BITS;
      const int nSel = g.load(&K->sel);
      if (threadIdx.x == 0) tl->sel += nSel;
      if constexpr (HIST) hp += nSel;
      int rc = 0;
      if (nSel > 0) {
        const Resel rs{sl, arrSlot, slots0, t};
        bool fused = false;  // take-back and slot writes done inside the solve
        if constexpr (!IsGrid<G>::value) {
          int ar = NOT_TAKEN;
          if constexpr (AS::kOn) {
            // a large re-solve goes to the helper workgroups of the XCD, which
            // also take the flows back and write their slots
            if (C->lds_paths && as->takes(nSel)) {
              ar = as->solve(g, P, lk, C, sc, nSel, ab, slots0, t, rounds, fsw, isw);
              if (ar != NOT_TAKEN) {
                // phase times: the first helper's, in place of the hand-over
                clk.skip();
                if (threadIdx.x == 0) {
                  tl->asst += 1;
                  if (P.debug & 2)
                    for (int k = 2; k < 7; ++k)
                      tl->clk[k] += __hip_atomic_load(reinterpret_cast<uint64_t*>(as->cw + CL_CLK) + k,
                                                      __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                }
              }
            }
          }
          if (ar != NOT_TAKEN) {
            rc = ar;
            fused = true;
          } else if (C->lds_paths && nSel <= 64 * (int)blockDim.x) {
            rc = solve_mask(g, P, lk, C, arrs, nSel, rounds, fsw, isw, clk, true, fc, &rs);
            fused = true;
          } else {
            take_back(g, P, lk, arrs, nSel, rs, f0, cap, err);
            if (err) g.store(&K->fault, 2);
            g.sync();
            if (threadIdx.x == 0) tl->wide += 1;
            rc = g.load(&K->fault) != 0 ? ST_OVERFLOW
                 : solve(g, P, lk, C, arrs, nSel, unf_a, unf_b, cap, rounds, fsw, isw, clk, true);
          }
        } else {
          take_back(g, P, lk, arrs, nSel, rs, f0, cap, err);
          if (err) g.store(&K->fault, 2);
          g.sync();
          if (g.load(&K->fault) != 0) {
            rc = ST_OVERFLOW;
          } else if (C->lds_paths && nSel <= LDS_FLOWS) {
            if (g.block_id() == 0) {
              BlockG b{g.lds, g.ldsi, &C->k};  // the grid's counters, in global memory
              const int r1 = solve_mask(b, P, lk, C, arrs, nSel, rounds, fsw, isw, clk, true, fc,
                                        nullptr);
              if (threadIdx.x == 0) g.store(&K->solve_rc, r1);
            }
            g.sync();
            rc = g.load(&K->solve_rc);
          } else if (C->lds_paths && nSel <= g.nblocks() * LDS_FLOWS) {
            rc = solve_lds(g, P, lk, C, arrs, nSel, rounds, fsw, isw, clk, *S, true);
          } else {
            if (threadIdx.x == 0) tl->wide += 1;
            rc = solve(g, P, lk, C, arrs, nSel, unf_a, unf_b, cap, rounds, fsw, isw, clk, true);
          }
        }
        if (!fused) {
          // the re-solved flows' slots: new rate and predicted completion
          for (int j = tid; j < nSel; j += T) {
            const int f = arrs[j];
            const int s = arrSlot[j];
            if (!in_range(f, f0, cap) || (unsigned)s >= (unsigned)cap) continue;
            const double r = P.rate[f];
            sl.rate[s] = r;
            sl.tau[s] = t + P.rem[f] / r;
          }
        }
        g.sync();
      }
      if ((P.debug & 1) && rc == 0) {
        // after a solve every active flow is frozen: no link has an unfrozen flow
        for (int l = C->l0 + tid; l < C->l1; l += T)
          if (lk.nfree(l) != 0) {
            g.store(&C->dbg[0], (int64_t)(e + 1));
            g.store(&C->dbg[1], (int64_t)l);
          }
        g.sync();
        if (g.load(&C->dbg[0]) != 0) { status = -8; break; }
      }
      if (threadIdx.x == 0) tl->solves += 1;  // the active set changed: one rate solve (possibly empty)
      if (rc != 0) { status = rc; break; }
    }
    // compaction: when holes are more than an eighth of the slots, copy the
    // live ones into the other buffer (every event sweeps all slots, holes
    // included, and a compaction costs about one sweep)
    const int holes = g.load(&K->holes);
    if (8 * holes > nSlots) {
      const Slots nx = slots(ab ^ 1);
      int32_t* const cnts[1] = {&K->slots2};
      sweep_append<1>(
          g, nSlots, cnts,
          [&](int s) {
            FlowVal x;
            x.f = sl.id[s];
            x.a = sl.tau[s];
            x.b = sl.rate[s];
            return x;
          },
          [&](int, const FlowVal& x, bool* pr) { pr[0] = x.f >= 0; },
          [&](int, int slot, const FlowVal& x) {
            if (slot < cap) {
              nx.id[slot] = x.f;
              nx.tau[slot] = x.a;
              nx.rate[slot] = x.b;
            } else {
              err = 1;
            }
          });
      if (err) g.store(&K->fault, 2);
      g.sync();
      nSlots = g.load(&K->slots2);
      ab ^= 1;
      g.sync();  // every thread has read the counters before they are reset
      if (tid == 0) {
        g.store(&K->slots, nSlots);
        g.store(&K->holes, 0);
      }
    }
    nPend = pNew;
    if (HIST && hist && tid == 0) {
      HistEv r;
      r.t = t;
      r.hpos = hp;
      r.solves = tl->solves;
      r.rounds = tl->rounds;
      r.flows_swept = tl->fsw;
      r.active_swept = tl->asw;
      r.pending_swept = tl->psw;
      r.reselected = tl->sel;
      r.wide_solves = tl->wide;
      r.assisted = tl->asst;
      P.hev[C->ebase + (int64_t)e % C->ecap] = r;
    }
    e += 1;
  }
  if (tid == 0 && !resume) C->incidences_swept = 0;
  g.sync();
  g.add(&C->incidences_swept, isw);
  if (tid == 0) {
    // position for a later launch that continues the part
    C->started = 1;
    C->e = e;
    C->q = q;
    C->ab = ab;
    C->nslots = nSlots;
    C->holes = g.load(&K->holes);
    C->npend = nPend;
    C->t = t;
    C->events = events;
    C->solves = tl->solves;
    C->rounds = tl->rounds;
    C->flows_swept = tl->fsw;
    C->active_swept = tl->asw;
    C->pending_swept = tl->psw;
    C->reselected = tl->sel;
    C->wide_solves = tl->wide;
    C->assisted = tl->asst;
    C->links_swept = (resume ? C->links_swept : 0) + g.load(&K->lsw);
    if constexpr (HIST) C->hpos = hp;
    C->launch_events = events - events0;
    C->status = status;
    for (int k = 0; k < 8; ++k) C->ticks[k] = (int64_t)tl->clk[k];
  }
}

template <class G>
__device__ __forceinline__ void solve_only(G& g, const Params& P, const int sc, SolveLds* S,
                                           Tally* tl, const FlowCache& fc) {
  LinksGlobal lk{P.lst, P.nact, P.fl, P.inv_scale};
  ScenCtl* C = &P.ctl[sc];
  const int f0 = C->f0;
  if (threadIdx.x == 0) tl->rounds = tl->fsw = 0;
  int64_t& rounds = tl->rounds;
  int64_t& fsw = tl->fsw;
  int64_t isw = 0;
  Clock clk(g.tid() == 0 && (P.debug & 2), tl->clk);
  int rc = 0;
  if (C->n_solve > 0) {
    if constexpr (IsGrid<G>::value) {
      if (C->lds_paths && C->n_solve <= g.nblocks() * LDS_FLOWS)
        rc = solve_lds(g, P, lk, C, P.act0 + f0, C->n_solve, rounds, fsw, isw, clk, *S, false);
      else
        rc = solve(g, P, lk, C, P.act0 + f0, C->n_solve, P.unf0 + f0, P.unf1 + f0, C->f1 - f0,
                   rounds, fsw, isw, clk, false);
    } else {
      if (C->lds_paths && C->n_solve <= 64 * (int)blockDim.x)
        rc = solve_mask(g, P, lk, C, P.act0 + f0, C->n_solve, rounds, fsw, isw, clk, false, fc,
                        nullptr);
      else
        rc = solve(g, P, lk, C, P.act0 + f0, C->n_solve, P.unf0 + f0, P.unf1 + f0, C->f1 - f0,
                   rounds, fsw, isw, clk, false);
    }
  }
  g.add(&C->incidences_swept, isw);
  if (g.tid() == 0) {
    C->solves = C->n_solve > 0 ? 1 : 0;
    C->rounds = tl->rounds;
    C->flows_swept = tl->fsw;
    C->status = rc;
    for (int k = 0; k < 8; ++k) C->ticks[k] = (int64_t)tl->clk[k];
  }
}

}  // namespace

// One workgroup per part.  A part whose links fit keeps its link state in
// shared memory for the whole run; the rest of the pool caches the path
// records of the flows being solved.  Built for workgroups of up to 512
// threads (256 registers per lane) and of up to 1024 (128 per lane).
template <int NT>
__global__ __launch_bounds__(NT) void netsim_block_kernel(Params P) {
  __shared__ double lds[32];
  __shared__ int ldsi[128];
  __shared__ Tally tally;
  __shared__ Lists lists;
  __shared__ __align__(16) unsigned char pool[POOL_BYTES];
  BlockG g{lds, ldsi, &lists};
  for (int sc = blockIdx.x; sc < P.num_scen; sc += gridDim.x) {
    const ScenCtl* C = &P.ctl[sc];
    if (threadIdx.x == 0) lists = Lists{};
    __syncthreads();
    const int nl = C->l1 - C->l0;
    const bool in_lds = P.mode == 0 && link_pool_bytes(nl) <= POOL_BYTES;
    const int used = in_lds ? (link_pool_bytes(nl) + 15) & ~15 : 0;
    const int ncache = (POOL_BYTES - used) / FLOW_LDS_BYTES;
    const FlowCache fc{reinterpret_cast<uint4*>(pool + used),
                       reinterpret_cast<int32_t*>(pool + used + 16 * ncache), ncache};
    if (P.mode != 0) {
      solve_only(g, P, sc, nullptr, &tally, fc);
    } else if (in_lds) {
      LinksShared lk(pool, C->l0, nl, P.inv_scale);
      event_loop<true>(g, P, lk, sc, nullptr, &tally, fc);
    } else {
      LinksGlobal lk{P.lst, P.nact, P.fl, P.inv_scale};
      event_loop<true>(g, P, lk, sc, nullptr, &tally, fc);
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(1024) void netsim_grid_kernel(Params P) {
  __shared__ double lds[32];
  __shared__ int ldsi[128];
  __shared__ int flag;
  __shared__ SolveLds S;
  __shared__ Tally tally;
  GridG g{lds, ldsi, &flag, P.bar, P.slots, 0u, 0u, false, 0u, 0u, 0u};
  g.init();
  LinksGlobal lk{P.lst, P.nact, P.fl, P.inv_scale};
  const FlowCache none{nullptr, nullptr, 0};
  for (int sc = 0; sc < P.num_scen; ++sc) {
    if (P.mode == 0) event_loop<true>(g, P, lk, sc, &S, &tally, none);
    else solve_only(g, P, sc, &S, &tally, none);
    g.sync();
  }
}

// One workgroup per CU, 1024 threads.  Every workgroup registers on its XCD,
// whose workgroups form P.clusters_per_xcd clusters of consecutive ranks (the
// last takes the remainder).  The first workgroup of a cluster leads: it
// claims parts one at a time and runs their event loops as the block kernel
// does, handing re-solves of at least P.assist_min flows to up to
// P.assist_helpers other workgroups of its cluster (its helpers; the
// cluster's remaining workgroups return at once).  With no helpers (a lone
// workgroup, or registration timed out) a leader solves everything itself.
// Every part is claimed by exactly one leader, whatever the number of
// leaders.
__global__ __launch_bounds__(1024) void netsim_cluster_kernel(Params P) {
  __shared__ double lds[32];
  __shared__ int ldsi[128];
  __shared__ Tally tally;
  __shared__ Lists lists;
  __shared__ int flag[2];
  __shared__ int box[8];
  __shared__ double tjob[1];
  __shared__ int claim;
  __shared__ __align__(16) unsigned char pool[POOL_BYTES];
  static_assert(sizeof(SolveLds) <= POOL_BYTES, "helper pool");
  if (threadIdx.x == 0) {
    const uint32_t x = xcc_id();
    uint32_t* xreg = P.bar + XREG_BASE + 16 * x;
    const uint32_t rank = __hip_atomic_fetch_add(xreg, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const uint32_t prev =
        __hip_atomic_fetch_add(&P.bar[BAR_REG], 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    bool ok = true;
    if (prev == gridDim.x - 1)
      __hip_atomic_store(&P.bar[BAR_REG_GEN], 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    else
      ok = wait_ne(P.bar, &P.bar[BAR_REG_GEN], 0u, BARRIER_TIMEOUT_TICKS);
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    const int on_xcd = (int)__hip_atomic_load(xreg, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    // clusters of consecutive ranks; without a complete registration every
    // workgroup is its own leader's only member (no helpers)
    const int nc = ok ? max(1, min(min(P.clusters_per_xcd, CL_MAXC), on_xcd)) : 1;
    const int size = max(on_xcd / nc, 1);
    const int cid = min((int)rank / size, nc - 1);
    const int members = cid == nc - 1 ? on_xcd - cid * size : size;
    box[0] = (int)x * CL_MAXC + cid;
    box[1] = (int)rank - cid * size;  // rank in the cluster
    // helpers: the cluster's other workgroups, at most P.assist_helpers of
    // them and one per arrival line
    box[2] = ok ? min(min(members - 1, max(P.assist_helpers, 0)), CL_LINES) : 0;
  }
  __syncthreads();
  const int cl = box[0], rank = box[1], nh = box[2];
  uint32_t* cw = P.bar + CL_BASE + CL_STRIDE * cl;
  __syncthreads();
  if (rank != 0) {  // workgroups beyond the helpers have nothing to do
    if (nh > 0 && rank <= nh) {
      const uint64_t patience = (P.debug & DEBUG_HELPER_BARRIER_GIVES_UP) ? 0 : BARRIER_TIMEOUT_TICKS;
      // per-link deltas in the pool after the solve's own arrays
      constexpr int off = (int)((sizeof(SolveLds) + 15) & ~size_t(15));
      constexpr int dcap = (POOL_BYTES - off) / 12;
      ClusterG cg{lds, ldsi, flag, P.bar, cw, 0u, rank - 1, nh, false, patience,
                  (P.debug & DEBUG_FORMAL_RELEASE) != 0,
                  reinterpret_cast<uint64_t*>(P.bar + CL_ARRIVE + CL_ARRIVE_STRIDE * cl),
                  reinterpret_cast<int64_t*>(pool + off), reinterpret_cast<int32_t*>(pool + off + 8 * dcap),
                  dcap};
      helper_loop(P, cg, *reinterpret_cast<SolveLds*>(pool), &tally, box, tjob);
    }
    return;
  }
  BlockG g{lds, ldsi, &lists};
  Assist as{P.bar, cw, nh, P.assist_min > 0 ? P.assist_min : 1, 0u, box};
  for (;;) {
    if (threadIdx.x == 0)
      claim = (int)__hip_atomic_fetch_add(&P.bar[BAR_NEXT], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    const int sc = claim;
    __syncthreads();
    if (sc >= P.num_scen) break;
    ScenCtl* C = &P.ctl[sc];
    if (threadIdx.x == 0) {
      lists = Lists{};
      C->k = Lists{};  // counters of the helpers' solves
    }
    const int nl = C->l1 - C->l0;
    const bool in_lds = link_pool_bytes(nl) <= POOL_BYTES;
    if (in_lds)  // the helpers' stamps start from zero with their counter
      for (int l = C->l0 + (int)threadIdx.x; l < C->l1; l += blockDim.x) P.fl[l] = 0;
    __syncthreads();
    const int used = in_lds ? (link_pool_bytes(nl) + 15) & ~15 : 0;
    const int ncache = (POOL_BYTES - used) / FLOW_LDS_BYTES;
    const FlowCache fc{reinterpret_cast<uint4*>(pool + used),
                       reinterpret_cast<int32_t*>(pool + used + 16 * ncache), ncache};
    if (in_lds) {
      LinksShared lk(pool, C->l0, nl, P.inv_scale);
      event_loop<false>(g, P, lk, sc, nullptr, &tally, fc, &as);
    } else {
      LinksGlobal lk{P.lst, P.nact, P.fl, P.inv_scale};
      event_loop<false>(g, P, lk, sc, nullptr, &tally, fc, &as);
    }
    __syncthreads();
  }
  // no more jobs: the helpers leave
  if (threadIdx.x == 0)
    __hip_atomic_exchange(&cw[CL_MB], CL_CLOSED, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}

hipError_t launch_block(const Params& p, int blocks, int threads, hipStream_t s) {
  if (threads <= 512)
    hipLaunchKernelGGL(netsim_block_kernel<512>, dim3(blocks), dim3(threads), 0, s, p);
  else
    hipLaunchKernelGGL(netsim_block_kernel<1024>, dim3(blocks), dim3(threads), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_grid(const Params& p, int blocks, int threads, hipStream_t s) {
  Params copy = p;
  void* args[] = {&copy};
  return hipLaunchCooperativeKernel((const void*)netsim_grid_kernel, dim3(blocks), dim3(threads),
                                    args, 0, s);
}

hipError_t launch_cluster(const Params& p, int blocks, hipStream_t s) {
  Params copy = p;
  void* args[] = {&copy};
  return hipLaunchCooperativeKernel((const void*)netsim_cluster_kernel, dim3(blocks), dim3(1024), args, 0,
                                    s);
}

hipError_t cluster_capacity(int device, int* blocks) {
  int per_cu = 0;
  hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, netsim_cluster_kernel, 1024, 0);
  if (e != hipSuccess) return e;
  hipDeviceProp_t prop;
  e = hipGetDeviceProperties(&prop, device);
  if (e != hipSuccess) return e;
  *blocks = per_cu * prop.multiProcessorCount;
  return hipSuccess;
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
