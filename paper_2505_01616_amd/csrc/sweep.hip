// Exact progressive filling over the whole GPU: one wide rate solve (a
// single part whose active set is too large for one workgroup to sweep
// quickly), with the arithmetic of exact.hip, as a sequence of kernels on
// one stream.  Section 4.2's water-filling, one bottleneck level per
// iteration:
//   count  (solve start) -- per-link unfrozen counts n_l by wave-level
//          segmented reductions over the link-major incidence (each lane one
//          incidence, consecutive lanes consecutive incidences of a link;
//          segment starts and sums from wave ballots; one atomic per
//          segment piece);
//   links  (per level)   -- apply the last level's freezes
//          (R_l -= k_l*s*, n_l -= k_l), share s_l = R_l/n_l, keep the links
//          that still carry unfrozen flows, and the level minimum s*
//          (wave shuffles, then one value per wave in shared memory, then one
//          value per workgroup, which the freezing sweep's workgroups reduce);
//   bottlenecks (per level) -- the level minimum s* and one byte per live
//          link: s_l <= s* * THR (THR = 1 + 1e-12), the freeze mask;
//   freeze (per level)   -- coalesced sweep of the unfrozen flows' path
//          records: a flow crossing a bottleneck link gets rate s* and adds 1
//          to k_l of each of its links; the others are kept for the next
//          level.
// Both lists are kept in per-workgroup segments (workgroup b of a sweep owns
// its slice of the list and a count), so compaction uses shared-memory
// counters only: no workgroup waits on an atomic in global memory.
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

__device__ __forceinline__ bool first_thread() { return blockIdx.x == 0 && threadIdx.x == 0; }

}  // namespace

// Workgroups and segment size of a sweep over n entries.
__host__ __device__ inline void segments(int n, int* blocks, int* seg) {
  const int b = (n + 255) / 256;
  *blocks = b < 1 ? 1 : (b > XG_MAX_BLOCKS ? XG_MAX_BLOCKS : b);
  *seg = (n + *blocks - 1) / *blocks;
  if (*seg < 1) *seg = 1;
}

// Solve start, first kernel: link state cleared on the part's links, the
// active-flow mask cleared on the part's flows (whole words: a word shared
// with a neighbouring part only holds bits nobody reads during this solve).
__global__ __launch_bounds__(256) void exact_init_kernel(Params P, int l0, int l1, int f0, int f1) {
  const int stride = gridDim.x * blockDim.x;
  const int i0 = blockIdx.x * blockDim.x + threadIdx.x;
  for (int l = l0 + i0; l < l1; l += stride) {
    P.xn[l] = 0;
    P.xk[l] = 0;
  }
  if (f1 > f0)
    for (int w = (f0 >> 5) + i0; w <= ((f1 - 1) >> 5); w += stride) P.xmask[w] = 0u;
}

// Solve start, second kernel: the active list copied to the first unfrozen
// list (entry i in segment i / useg), its flows set in the mask, counters
// reset.
__global__ __launch_bounds__(256) void exact_mark_kernel(Params P, int l0, int l1, int f0, int n,
                                                         XGrid* g) {
  int ub, us;
  segments(n, &ub, &us);
  const int stride = gridDim.x * blockDim.x;
  const int i0 = blockIdx.x * blockDim.x + threadIdx.x;
  for (int i = i0; i < n; i += stride) {
    const int f = P.act0[f0 + i];
    P.unf0[f0 + i] = f;
    atomicOr(&P.xmask[f >> 5], 1u << (f & 31));
  }
  int lb, ls;
  segments(l1 - l0, &lb, &ls);
  for (int b = i0; b < ub; b += stride) {
    const int c = n - b * us;
    g->ucnt[0][b] = c < 0 ? 0 : (c > us ? us : c);
    g->ucnt[1][b] = 0;
    g->isw[b] = 0;
  }
  for (int b = i0; b < lb; b += stride) g->lsw[b] = 0;
  if (first_thread()) {
    g->fault = 0;
    g->done = 0;
    g->ublocks = ub;
    g->useg = us;
    g->lblocks = lb;
    g->lseg = ls;
    g->levels = 0;
    g->fsw = 0;
  }
}

// Appends the lanes with pred to a workgroup's segment: one shared-memory
// atomic per wave.
__device__ __forceinline__ int sappend(int* counter, bool pred) {
  const uint64_t mask = __ballot(pred);
  if (mask == 0) return -1;
  const int lane = threadIdx.x & 63;
  const int leader = __ffsll((unsigned long long)mask) - 1;
  int base = 0;
  if (lane == leader) base = atomicAdd(counter, (int)__popcll(mask));
  base = __shfl(base, leader, 64);
  return pred ? base + (int)__popcll(mask & ((1ull << lane) - 1ull)) : -1;
}

// Per-link unfrozen counts: n_l = number of active flows among the flows of
// link l, over the part's incidences [e0, e1) in link-major order (lfid: the
// flows of link l are lfid[lfoff[l] .. lfoff[l+1]-1]; every link has at
// least one).  A flow's flag is one bit of the active-flow mask.  The
// incidences are taken in chunks of 256, one chunk per wave at a time as four
// rounds of 64 consecutive incidences (the loads of four chunks in flight
// together).  lfchunk[c] is the link of the chunk's first incidence and
// lfhead holds one bit per incidence, set where a link starts, so within a
// round an incidence's link is lfchunk[c] plus the link starts after the
// chunk's first incidence up to it, and the segmented sum of the 0/1 flags
// is a population count of the wave's ballot between the segment start and
// the lane: no shuffles for the scan.  The last lane of each segment piece
// adds the piece's count.  (Staging the mask in shared memory was measured:
// copying it into every compute unit cost as much as the gathers it saves.)
__global__ __launch_bounds__(256) void exact_count_kernel(Params P, int e0, int e1,
                                                          unsigned long long* stamps) {
  if (stamps && threadIdx.x == 0) stamps[2 * blockIdx.x] = wall_clock64();
  const int lane = threadIdx.x & 63;
  const uint64_t below = lane == 63 ? ~0ull : (2ull << lane) - 1ull;  // lanes 0..lane
  const int wave = (blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int waves = (gridDim.x * blockDim.x) >> 6;
  // a wave takes chunks c, c + waves, c + 2 waves, c + 3 waves at a time:
  // sixteen rounds of loads in flight
  constexpr int NC = 4;
  for (int c0 = e0 / 256 + wave; c0 * 256 < e1; c0 += NC * waves) {
    int fl[NC][4];
    uint64_t hm[NC][4];
    int lc[NC];
    // the chunks' link-start words and first links: lane q < 16 loads word
    // q & 3 of chunk q >> 2, lane q < NC the first link of chunk q (vector
    // loads, then broadcast by shuffles: uniform loads with this little
    // locality are slow through the scalar cache)
    const int hk = (lane >> 2) & (NC - 1), hr = lane & 3;
    const int hc = c0 + hk * waves;
    const uint64_t hv = hc * 256 < e1 ? P.lfhead[hc * 4 + hr] : ~0ull;
    const int cc = c0 + (lane & (NC - 1)) * waves;
    const int cv = cc * 256 < e1 ? P.lfchunk[cc] : 0;
#pragma unroll
    for (int k = 0; k < NC; ++k) {
      const int base = (c0 + k * waves) * 256;
      const bool live = base < e1;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int e = base + r * 64 + lane;
        fl[k][r] = live && e >= e0 && e < e1 ? P.lfid[e] : -1;
      }
    }
#pragma unroll
    for (int k = 0; k < NC; ++k) {
#pragma unroll
      for (int r = 0; r < 4; ++r) hm[k][r] = __shfl(hv, k * 4 + r, 64);
      lc[k] = __shfl(cv, k, 64);
    }
#pragma unroll
    for (int k = 0; k < NC; ++k) {
      bool v[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int f = fl[k][r];
        const uint32_t w = f >= 0 ? P.xmask[f >> 5] : 0u;
        v[r] = (w >> (f & 31)) & 1u;
      }
      int carry = 0;  // links started after the chunk's first incidence, in earlier rounds
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        // the chunk's first incidence starts (or continues) link lc itself
        const uint64_t h = r == 0 ? hm[k][r] & ~1ull : hm[k][r];
        const int l = lc[k] + carry + (int)__popcll(h & below);
        const uint64_t vm = __ballot(v[r]);
        // start of this lane's segment piece: the last link start at or
        // before it in the round, else the round's first lane
        const uint64_t starts = (h | 1ull) & below;
        const int sl = 63 - __clzll(starts);
        const int x = (int)__popcll(vm & below & ~((1ull << sl) - 1ull));
        const bool tail = lane == 63 || ((h >> (lane + 1)) & 1ull);
        if (fl[k][r] >= 0 && tail && x > 0) atomicAdd(&P.xn[l], x);
        carry += (int)__popcll(h);
      }
    }
  }
  if (stamps) {
    __syncthreads();
    if (threadIdx.x == 0) stamps[2 * blockIdx.x + 1] = wall_clock64();
  }
}

// Level j, links: workgroup b takes its segment of the live links (level 0:
// links l0 + [b * seg, (b + 1) * seg) of the part), applies the last level's
// freezes, computes shares, keeps the links with unfrozen flows in its
// segment of the other list and takes the level minimum.
__global__ __launch_bounds__(256) void exact_links_kernel(Params P, int l0, int l1, int j, XGrid* g) {
  __shared__ double wmin[4], pmin[4];
  __shared__ int kept, total[4];
  if (g->done || g->fault) return;  // the solve is over
  const bool first = j == 0;
  const int b = blockIdx.x, seg = g->lseg, nl = l1 - l0, tid = threadIdx.x;
  const int n_in = first ? max(0, min(seg, nl - b * seg)) : g->lcnt[j & 1][b];
  const int32_t* lin = ((j & 1) ? P.xlive1 : P.xlive0) + l0 + b * seg;
  int32_t* lout = ((j & 1) ? P.xlive0 : P.xlive1) + l0 + b * seg;
  // this thread's first link and its state, loaded before the reductions
  // below so that their latencies overlap
  int l = -1, n = 0, k = 0;
  double R = 0.0;
  if (tid < n_in) {
    l = first ? l0 + b * seg + tid : lin[tid];
    n = P.xn[l];
    R = first ? P.capf[l] : P.xR[l];
    k = first ? 0 : P.xk[l];
  }
  // unfrozen flows entering this level (the freezing sweep's segment counts;
  // level 0: the whole list) and the last level's minimum (over its link
  // pass's workgroups), one value per thread, then per wave, then per block
  int nu = 0;
  for (int q = tid; q < g->ublocks; q += blockDim.x) nu += g->ucnt[j & 1][q];
  double pm = GINF;
  if (!first)
    for (int q = tid; q < (int)gridDim.x; q += blockDim.x) {
      const double v = g->bmin[(j - 1) & 1][q];
      pm = v < pm ? v : pm;
    }
  nu = gwave_sum(nu);
  pm = gwave_min(pm);
  if ((tid & 63) == 0) {
    total[tid >> 6] = nu;
    pmin[tid >> 6] = pm;
  }
  if (tid == 0) kept = 0;
  __syncthreads();
  nu = total[0] + total[1] + total[2] + total[3];
  double sprev = pmin[0];
  for (int w = 1; w < 4; ++w) sprev = pmin[w] < sprev ? pmin[w] : sprev;
  if (nu == 0) {
    // the last level froze every flow: this level's freezing sweep and every
    // later kernel return at once
    if (first_thread()) g->done = 1;
    return;
  }
  if (first_thread()) g->fsw += (unsigned long long)nu;
  double loc = GINF;
  for (int i0 = 0; i0 < n_in; i0 += blockDim.x) {
    const int i = i0 + tid;
    bool keep = false;
    if (i < n_in) {
      if (i0 > 0) {
        l = first ? l0 + b * seg + i : lin[i];
        n = P.xn[l];
        R = first ? P.capf[l] : P.xR[l];
        k = first ? 0 : P.xk[l];
      }
      if (first) {
        P.xR[l] = R;
      } else if (k != 0) {
        const double dec = (double)k * sprev;
        R = R - dec;
        n -= k;
        P.xR[l] = R;
        P.xn[l] = n;
        P.xk[l] = 0;
      }
      keep = n > 0;
      if (keep) {
        const double s = R / (double)n;
        P.xs[l] = s;
        loc = s < loc ? s : loc;
      }
    }
    const int slot = sappend(&kept, keep);
    if (keep) lout[slot] = l;
  }
  loc = gwave_min(loc);
  if ((tid & 63) == 0) wmin[tid >> 6] = loc;
  __syncthreads();
  if (tid == 0) {
    double m = GINF;
    for (int w = 0; w < (int)(blockDim.x >> 6); ++w) m = wmin[w] < m ? wmin[w] : m;
    g->bmin[j & 1][b] = m;
    g->lcnt[(j + 1) & 1][b] = kept;
    g->lsw[b] += (unsigned long long)kept;
  }
}

// Level j, bottlenecks: the level minimum s* (over the link pass's
// per-workgroup minima; workgroup 0 records it for the freezing sweep) and,
// for each live link of the workgroup's segment, one byte: s_l <= s* * THR.
// The freezing sweep reads these bytes (a table small enough to stay in each
// compute unit's L1) instead of gathering 8-byte shares.
__global__ __launch_bounds__(256) void exact_bottleneck_kernel(Params P, int l0, int j, XGrid* g) {
  __shared__ double smin[4];
  if (g->done || g->fault) return;
  const int b = blockIdx.x, seg = g->lseg, tid = threadIdx.x;
  const int n_in = g->lcnt[(j + 1) & 1][b];  // the live links the link pass kept
  const int32_t* lv = ((j & 1) ? P.xlive0 : P.xlive1) + l0 + b * seg;
  int l = -1;
  double sv = 0.0;
  if (tid < n_in) {
    l = lv[tid];
    sv = P.xs[l];
  }
  double m = GINF;
  for (int q = tid; q < (int)gridDim.x; q += blockDim.x) {
    const double v = g->bmin[j & 1][q];
    m = v < m ? v : m;
  }
  m = gwave_min(m);
  if ((tid & 63) == 0) smin[tid >> 6] = m;
  __syncthreads();
  double s = smin[0];
  for (int w = 1; w < 4; ++w) s = smin[w] < s ? smin[w] : s;
  if (!(s > 0.0) || !(s < GINF)) {
    if (first_thread()) g->fault = 1;
    return;
  }
  if (first_thread()) g->sstar[j & 1] = s;
  const double thr = s * GTHR;
  for (int i0 = 0; i0 < n_in; i0 += blockDim.x) {
    const int i = i0 + tid;
    if (i < n_in) {
      if (i0 > 0) {
        l = lv[i];
        sv = P.xs[l];
      }
      P.xfz[l] = sv <= thr ? 1 : 0;
    }
  }
}

// Level j, freezing sweep: workgroup b takes its segment of the unfrozen
// flows (path records: six part-local 16-bit link ids, 0xFFFF = none; or
// the path CSR), freezes every flow crossing a bottleneck link (its byte from
// the bottleneck pass) at rate s* and keeps the others in its segment of the
// other list.
template <bool REC>
__global__ __launch_bounds__(256) void exact_freeze_kernel(Params P, int l0, int f0, int n0, int j,
                                                           XGrid* g, unsigned long long* stamps) {
  if (stamps && threadIdx.x == 0) stamps[2 * blockIdx.x] = wall_clock64();
  __shared__ unsigned long long inc_sum;
  __shared__ int kept;
  if (g->done || g->fault) return;
  const int b = blockIdx.x;
  int seg, n_in;
  if (j == 0) {
    // the first level's segments follow from the list's length
    int blocks;
    segments(n0, &blocks, &seg);
    n_in = max(0, min(seg, n0 - b * seg));
  } else {
    seg = g->useg;
    n_in = g->ucnt[j & 1][b];
  }
  const int32_t* uin = ((j & 1) ? P.unf1 : P.unf0) + f0 + b * seg;
  int32_t* uout = ((j & 1) ? P.unf0 : P.unf1) + f0 + b * seg;
  // this thread's first flow and its path record, loaded before the
  // reduction below so that their latencies overlap
  int f = -1;
  uint4 rec = make_uint4(0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu, 0u);
  if ((int)threadIdx.x < n_in) {
    f = uin[threadIdx.x];
    if constexpr (REC) rec = P.path16[f];
  }
  // the level minimum the bottleneck pass recorded
  const double s = g->sstar[j & 1];
  if (threadIdx.x == 0) {
    inc_sum = 0;
    kept = 0;
  }
  __syncthreads();
  if (first_thread()) g->levels += 1;
  unsigned long long inc = 0;
  for (int i0 = 0; i0 < n_in; i0 += blockDim.x) {
    const int i = i0 + threadIdx.x;
    bool keep = false;
    if (i0 > 0) f = -1;
    if (i < n_in) {
      if (i0 > 0) f = uin[i];
      bool fz = false;
      if constexpr (REC) {
        const uint4 r = i0 > 0 ? P.path16[f] : rec;
        const uint32_t w[3] = {r.x, r.y, r.z};
        int lv[6];
        int deg = 0;
#pragma unroll
        for (int q = 0; q < 6; ++q) {
          const uint32_t id = (w[q >> 1] >> (16 * (q & 1))) & 0xFFFFu;
          if (id != 0xFFFFu) lv[deg++] = l0 + (int)id;
        }
        for (int q = 0; q < deg; ++q) fz |= P.xfz[lv[q]] != 0;
        inc += (unsigned long long)deg;
        if (fz)
          for (int q = 0; q < deg; ++q) atomicAdd(&P.xk[lv[q]], 1);
      } else {
        const int e0 = P.poff[f], e1 = P.poff[f + 1];
        for (int e = e0; e < e1; ++e) fz |= P.xfz[P.plink[e]] != 0;
        inc += (unsigned long long)(e1 - e0);
        if (fz)
          for (int e = e0; e < e1; ++e) atomicAdd(&P.xk[P.plink[e]], 1);
      }
      if (fz) {
        P.rate[f] = s;
      } else {
        keep = true;
      }
    }
    const int slot = sappend(&kept, keep);
    if (keep) uout[slot] = f;
  }
  inc = gwave_sum(inc);
  if ((threadIdx.x & 63) == 0 && inc) atomicAdd(&inc_sum, inc);
  __syncthreads();
  if (threadIdx.x == 0) {
    g->ucnt[(j + 1) & 1][b] = kept;
    g->isw[b] += inc_sum;
    if (stamps) stamps[2 * b + 1] = wall_clock64();
  }
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
  const int words = C.f1 > C.f0 ? ((C.f1 - 1) >> 5) - (C.f0 >> 5) + 1 : 0;
  hipLaunchKernelGGL(exact_init_kernel, dim3(blocks_for(std::max(words, C.l1 - C.l0), 1, 4096)), dim3(256), 0,
                     s, P, C.l0, C.l1, C.f0, C.f1);
  hipLaunchKernelGGL(exact_mark_kernel, dim3(blocks_for(n, 1, 4096)), dim3(256), 0, s, P, C.l0, C.l1, C.f0, n,
                     P.xgrid);
  return hipGetLastError();
}

int count_blocks(int e0, int e1) {
  const int chunks = (e1 - e0 + 255) / 256 + 1;
  return std::max(1, std::min(XG_MAX_BLOCKS, (chunks + 15) / 16));  // four waves, four chunks each
}

hipError_t grid_solve_count(const Params& P, const ScenCtl& C, int e0, int e1, hipStream_t s,
                            unsigned long long* stamps) {
  (void)C;
  if (e1 <= e0) return hipSuccess;
  hipLaunchKernelGGL(exact_count_kernel, dim3(count_blocks(e0, e1)), dim3(256), 0, s, P, e0, e1, stamps);
  return hipGetLastError();
}

hipError_t grid_solve_links(const Params& P, const ScenCtl& C, int j, hipStream_t s) {
  int blocks, seg;
  segments(C.l1 - C.l0, &blocks, &seg);
  hipLaunchKernelGGL(exact_links_kernel, dim3(blocks), dim3(256), 0, s, P, C.l0, C.l1, j, P.xgrid);
  hipLaunchKernelGGL(exact_bottleneck_kernel, dim3(blocks), dim3(256), 0, s, P, C.l0, j, P.xgrid);
  return hipGetLastError();
}

int freeze_blocks(int n) {
  int blocks, seg;
  segments(n, &blocks, &seg);
  return blocks;
}

hipError_t grid_solve_freeze(const Params& P, const ScenCtl& C, int n, int j, hipStream_t s,
                             unsigned long long* stamps) {
  const dim3 grid(freeze_blocks(n));
  if (C.lds_paths)
    hipLaunchKernelGGL(exact_freeze_kernel<true>, grid, dim3(256), 0, s, P, C.l0, C.f0, n, j, P.xgrid, stamps);
  else
    hipLaunchKernelGGL(exact_freeze_kernel<false>, grid, dim3(256), 0, s, P, C.l0, C.f0, n, j, P.xgrid, stamps);
  return hipGetLastError();
}

hipError_t launch_flush(void* buf, size_t bytes, uint32_t tag, hipStream_t s) {
  hipLaunchKernelGGL(flush_kernel, dim3(4096), dim3(256), 0, s, static_cast<uint4*>(buf), bytes / 16, tag);
  return hipGetLastError();
}

}  // namespace netsim_dev
