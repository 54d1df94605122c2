// Exact progressive filling over the whole GPU: one wide rate solve (a
// single part whose active set is too large for one workgroup to sweep
// quickly), with the arithmetic of exact.hip, as a sequence of kernels on
// one stream.  Section 4.2's water-filling, one bottleneck level per
// iteration:
//   count  (solve start) -- per-link unfrozen counts n_l by wave-shuffle
//          segmented reductions over the link-major incidence (each lane one
//          incidence, consecutive lanes consecutive incidences of a link;
//          one atomic per segment piece);
//   links  (per level)   -- apply the last level's freezes
//          (R_l -= k_l*s*, n_l -= k_l), share s_l = R_l/n_l, compact the
//          links that still carry unfrozen flows, and the level minimum s*
//          (wave shuffles, then one value per wave in shared memory, then one
//          atomic minimum on the bit pattern per workgroup: positive doubles
//          order like their bit patterns);
//   freeze (per level)   -- coalesced sweep of the unfrozen flows' path
//          records: a flow crossing a link with s_l <= s* * THR gets rate s*
//          and adds 1 to k_l of each of its links; the others are appended to
//          the next unfrozen list.
// Level j's kernels read and write buffers by the parity of j; each kernel
// resets the counters the kernel after the next one appends to, so no
// host work happens between levels.  The first level that starts with no
// unfrozen flow raises a done flag, after which every kernel returns at once
// (the other parity's counters are stale by then), which lets the host
// enqueue levels in batches.
#include "device.h"

#include <math.h>

#include <algorithm>

#pragma clang fp contract(off)

namespace netsim_dev {

namespace {

constexpr double GTHR = 1.000000000001;
constexpr double GINF = __builtin_huge_val();
constexpr unsigned long long GINF_BITS = 0x7FF0000000000000ull;

__device__ __forceinline__ double gwave_min(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const double w = __shfl_xor(v, o, 64);
    v = w < v ? w : v;
  }
  return v;
}

template <class T>
__device__ __forceinline__ T gwave_sum(T v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Appends the lanes with pred to a global list: one device atomic per wave.
__device__ __forceinline__ int gappend(int32_t* counter, bool pred) {
  const uint64_t mask = __ballot(pred);
  if (mask == 0) return -1;
  const int lane = threadIdx.x & 63;
  const int leader = __ffsll((unsigned long long)mask) - 1;
  int base = 0;
  if (lane == leader) base = atomicAdd(counter, (int)__popcll(mask));
  base = __shfl(base, leader, 64);
  return pred ? base + (int)__popcll(mask & ((1ull << lane) - 1ull)) : -1;
}

__device__ __forceinline__ bool first_thread() { return blockIdx.x == 0 && threadIdx.x == 0; }

}  // namespace

// Solve start: link state cleared on the part's links, the active list
// copied to the first unfrozen list and flagged, counters reset.
__global__ __launch_bounds__(256) void exact_init_kernel(Params P, int l0, int l1, int f0, int n,
                                                         XGrid* g) {
  const int stride = gridDim.x * blockDim.x;
  const int i0 = blockIdx.x * blockDim.x + threadIdx.x;
  for (int l = l0 + i0; l < l1; l += stride) {
    P.xn[l] = 0;
    P.xk[l] = 0;
  }
  for (int i = i0; i < n; i += stride) {
    const int f = P.act0[f0 + i];
    P.unf0[f0 + i] = f;
    P.xact[f] = 1;
  }
  if (first_thread()) {
    g->gmin[0] = GINF_BITS;
    g->gmin[1] = GINF_BITS;
    g->cu[0] = n;
    g->cu[1] = 0;
    g->cl[0] = 0;
    g->cl[1] = 0;
    g->fault = 0;
    g->done = 0;
    g->levels = 0;
    g->fsw = 0;
    g->isw = 0;
    g->lsw = 0;
  }
}

// Per-link unfrozen counts: n_l = number of active flows among the flows of
// link l, for the part's incidences [e0, e1) in link-major order (lfid: flow,
// lflink: its link).  Every wave takes 256 consecutive incidences as four
// rounds of 64 (loads of all four in flight), a segmented inclusive scan by
// link over the lanes of each round, and the last lane of each segment piece
// adds the piece's sum.
__global__ __launch_bounds__(256) void exact_count_kernel(Params P, int e0, int e1) {
  const int lane = threadIdx.x & 63;
  const int wave = (blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int waves = (gridDim.x * blockDim.x) >> 6;
  for (int base = e0 + wave * 256; base < e1; base += waves * 256) {
    int fl[4], lk[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int e = base + r * 64 + lane;
      fl[r] = e < e1 ? P.lfid[e] : -1;
      lk[r] = e < e1 ? P.lflink[e] : -1;
    }
    int v[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) v[r] = fl[r] >= 0 ? (int)P.xact[fl[r]] : 0;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      int x = v[r];
      const int l = lk[r];
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x, o, 64);
        const int m = __shfl_up(l, o, 64);
        if (lane >= o && m == l) x += y;
      }
      const int next = __shfl_down(l, 1, 64);
      const bool tail = lane == 63 || next != l;
      if (tail && l >= 0 && x > 0) atomicAdd(&P.xn[l], x);
    }
  }
}

// Level j, links: over the live links (level 0: every link of the part)
// apply the last level's freezes, compute shares, keep the links with
// unfrozen flows for level j + 1 and take the level minimum.
__global__ __launch_bounds__(256) void exact_links_kernel(Params P, int l0, int l1, int j, XGrid* g) {
  __shared__ double wmin[4];
  if (g->done || g->fault) return;  // the solve is over
  if (g->cu[j & 1] == 0) {
    // the last level froze every flow: later levels (and this level's
    // freezing sweep) return at once, whatever the other parity's counters
    // still hold
    if (first_thread()) g->done = 1;
    return;
  }
  const bool first = j == 0;
  const int n_in = first ? l1 - l0 : g->cl[j & 1];
  const int32_t* lin = (j & 1) ? P.xlive1 + l0 : P.xlive0 + l0;
  int32_t* lout = (j & 1) ? P.xlive0 + l0 : P.xlive1 + l0;
  int32_t* cout = &g->cl[(j + 1) & 1];
  const double sprev = first ? 0.0 : __longlong_as_double((long long)g->gmin[(j - 1) & 1]);
  if (first_thread()) g->cu[(j + 1) & 1] = 0;  // this level's freezing sweep appends there
  double loc = GINF;
  const int stride = gridDim.x * blockDim.x;
  for (int b = blockIdx.x * blockDim.x; b < n_in; b += stride) {
    const int i = b + threadIdx.x;
    bool keep = false;
    int l = 0;
    if (i < n_in) {
      l = first ? l0 + i : lin[i];
      int n = P.xn[l];
      double R;
      if (first) {
        R = P.capf[l];
        P.xR[l] = R;
      } else {
        R = P.xR[l];
        const int k = P.xk[l];
        if (k != 0) {
          const double dec = (double)k * sprev;
          R = R - dec;
          n -= k;
          P.xR[l] = R;
          P.xn[l] = n;
          P.xk[l] = 0;
        }
      }
      keep = n > 0;
      if (keep) {
        const double s = R / (double)n;
        P.xs[l] = s;
        loc = s < loc ? s : loc;
      }
    }
    const int slot = gappend(cout, keep);
    if (keep) lout[slot] = l;
  }
  loc = gwave_min(loc);
  if ((threadIdx.x & 63) == 0) wmin[threadIdx.x >> 6] = loc;
  __syncthreads();
  if (threadIdx.x == 0) {
    double m = GINF;
    for (int w = 0; w < (int)(blockDim.x >> 6); ++w) m = wmin[w] < m ? wmin[w] : m;
    if (m < GINF) atomicMin(&g->gmin[j & 1], (unsigned long long)__double_as_longlong(m));
  }
}

// Level j, freezing sweep over the unfrozen flows (path records: six
// part-local 16-bit link ids, 0xFFFF = none).
template <bool REC>
__global__ __launch_bounds__(256) void exact_freeze_kernel(Params P, int l0, int f0, int j, XGrid* g) {
  __shared__ unsigned long long part[2];
  if (g->done || g->fault) return;
  const int nu = g->cu[j & 1];
  if (nu == 0) return;
  const double s = __longlong_as_double((long long)g->gmin[j & 1]);
  if (!(s > 0.0) || !(s < GINF)) {
    if (first_thread()) g->fault = 1;
    return;
  }
  if (threadIdx.x == 0) {
    part[0] = 0;
    part[1] = 0;
  }
  if (first_thread()) {
    g->gmin[(j + 1) & 1] = GINF_BITS;  // the next level's minimum
    g->cl[j & 1] = 0;                  // the next level's link pass appends there
    g->levels += 1;
    g->fsw += (unsigned long long)nu;
    g->lsw += (unsigned long long)g->cl[(j + 1) & 1];  // links whose share this level computed
  }
  __syncthreads();
  const double thr = s * GTHR;
  const int32_t* uin = (j & 1) ? P.unf1 + f0 : P.unf0 + f0;
  int32_t* uout = (j & 1) ? P.unf0 + f0 : P.unf1 + f0;
  int32_t* cout = &g->cu[(j + 1) & 1];
  unsigned long long inc = 0;
  const int stride = gridDim.x * blockDim.x;
  for (int b = blockIdx.x * blockDim.x; b < nu; b += stride) {
    const int i = b + threadIdx.x;
    bool keep = false;
    int f = -1;
    if (i < nu) {
      f = uin[i];
      bool fz = false;
      if constexpr (REC) {
        const uint4 r = P.path16[f];
        const uint32_t w[3] = {r.x, r.y, r.z};
        int lv[6];
        int deg = 0;
#pragma unroll
        for (int q = 0; q < 6; ++q) {
          const uint32_t id = (w[q >> 1] >> (16 * (q & 1))) & 0xFFFFu;
          if (id != 0xFFFFu) lv[deg++] = l0 + (int)id;
        }
        for (int q = 0; q < deg; ++q) fz |= P.xs[lv[q]] <= thr;
        inc += (unsigned long long)deg;
        if (fz)
          for (int q = 0; q < deg; ++q) atomicAdd(&P.xk[lv[q]], 1);
      } else {
        const int e0 = P.poff[f], e1 = P.poff[f + 1];
        for (int e = e0; e < e1; ++e) fz |= P.xs[P.plink[e]] <= thr;
        inc += (unsigned long long)(e1 - e0);
        if (fz)
          for (int e = e0; e < e1; ++e) atomicAdd(&P.xk[P.plink[e]], 1);
      }
      if (fz) {
        P.rate[f] = s;
        P.xact[f] = 0;
      } else {
        keep = true;
      }
    }
    const int slot = gappend(cout, keep);
    if (keep) uout[slot] = f;
  }
  inc = gwave_sum(inc);
  if ((threadIdx.x & 63) == 0) atomicAdd(&part[0], inc);
  __syncthreads();
  if (threadIdx.x == 0) atomicAdd(&g->isw, part[0]);
}

// A streaming write over a buffer of `words` 16-byte words: evicts the L2
// and the Infinity Cache before a cold-cache measurement.
__global__ __launch_bounds__(256) void flush_kernel(uint4* buf, size_t words, uint32_t tag) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < words; i += stride)
    buf[i] = make_uint4(tag, (uint32_t)i, tag ^ (uint32_t)i, 0u);
}

namespace {

int blocks_for(int64_t items, int per_thread, int cap) {
  const int64_t b = (items + 256LL * per_thread - 1) / (256LL * per_thread);
  return (int)std::max<int64_t>(1, std::min<int64_t>(b, cap));
}

}  // namespace

hipError_t grid_solve_begin(const Params& P, const ScenCtl& C, int n, hipStream_t s) {
  hipLaunchKernelGGL(exact_init_kernel, dim3(blocks_for(std::max(n, C.l1 - C.l0), 1, 4096)), dim3(256), 0,
                     s, P, C.l0, C.l1, C.f0, n, P.xgrid);
  return hipGetLastError();
}

hipError_t grid_solve_count(const Params& P, int e0, int e1, hipStream_t s) {
  if (e1 <= e0) return hipSuccess;
  hipLaunchKernelGGL(exact_count_kernel, dim3(blocks_for(e1 - e0, 4, 8192)), dim3(256), 0, s, P, e0, e1);
  return hipGetLastError();
}

hipError_t grid_solve_links(const Params& P, const ScenCtl& C, int j, hipStream_t s) {
  hipLaunchKernelGGL(exact_links_kernel, dim3(blocks_for(C.l1 - C.l0, 1, 4096)), dim3(256), 0, s, P, C.l0,
                     C.l1, j, P.xgrid);
  return hipGetLastError();
}

hipError_t grid_solve_freeze(const Params& P, const ScenCtl& C, int n, int j, hipStream_t s) {
  const dim3 grid(blocks_for(n, 1, 8192));
  if (C.lds_paths)
    hipLaunchKernelGGL(exact_freeze_kernel<true>, grid, dim3(256), 0, s, P, C.l0, C.f0, j, P.xgrid);
  else
    hipLaunchKernelGGL(exact_freeze_kernel<false>, grid, dim3(256), 0, s, P, C.l0, C.f0, j, P.xgrid);
  return hipGetLastError();
}

hipError_t launch_flush(void* buf, size_t bytes, uint32_t tag, hipStream_t s) {
  hipLaunchKernelGGL(flush_kernel, dim3(4096), dim3(256), 0, s, static_cast<uint4*>(buf), bytes / 16, tag);
  return hipGetLastError();
}

}  // namespace netsim_dev
