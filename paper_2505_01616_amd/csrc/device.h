// Internal interface between the host side of libnetsim and its HIP kernels.
// Not part of the public C ABI (include/netsim.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace netsim_dev {

// Counters of the event loop's work lists and flags of the current event.
// Kernel scratch, zero when a part starts: in global memory (the part's
// control block) when the whole grid runs the part, in shared memory when
// one workgroup does.
struct Lists {
  int32_t slots;           // slots in use in the current slot buffer
  int32_t holes;           // slots of finished flows among them
  int32_t slots2;          // slots filled by a compaction
  int32_t pend[2];         // flows waiting for their release time
  int32_t comp[3];         // flows finished in the current wave of releases
  int32_t unf[2];          // unfrozen flows of a solve with global lists
  int32_t changed[2];      // the active set changed in this event
  int32_t rem3[3];         // shared-memory solve: unfrozen flows left, rotating
  int32_t arr;             // flows activated in the current event
  int32_t sel;             // flows taken back for re-solving in the current event
  int32_t succ_flag[2];    // a flow finished in this event has dependants
  int32_t solve_rc;        // status of a solve run by one workgroup
  int32_t fault;           // 1: bad fair share, 2: a work list overflowed or held a bad id
  uint32_t stamp;          // last freezing-round number used by the part's solves
  int32_t pad;
  int64_t lsw;             // links with unfrozen flows summed over the share-table passes
};

// Rollback history (paper Section 4.2: the simulator keeps every flow's
// throughput history so that it can return to the state at any earlier
// event).  Per part two rings in device memory: an undo record for every
// flow taken back for a re-solve, holding its remaining bytes, their time
// and its rate from before that event changed them, and a record of every
// event.  Going back to event e takes the state after the last event,
// applies each flow's first undo record written after e, and rebuilds
// which flows were waiting, pending, active or finished from the events at
// which each flow reached those states.
struct HistUndo {
  int32_t f, ev;           // device flow id; event (index in its part) that re-solved it
  double rem, tref, rate;  // the flow's values before that event
};
struct HistEv {
  double t;                // event time
  int64_t hpos;            // undo records written up to the end of this event
  int64_t solves, rounds, flows_swept, active_swept;  // statistics at its end
  int64_t pending_swept, reselected, wide_solves, assisted;
};
// "Not yet" in the per-flow event indices (Params::evr, eva, evd).
constexpr int32_t EV_NEVER = 0x7F7F7F7F;

// Control block of one part in device memory.  A part is a set of flows of
// one scenario that shares no link and no dependency with the rest of the
// scenario, simulated with its own clock.  The host fills the ranges and the
// initial counters; the kernels keep their list counters here and write the
// results back at the end of the run.
struct ScenCtl {
  int32_t f0, f1;          // device flow range [f0, f1)
  int32_t l0, l1;          // device link range [l0, l1)
  int32_t n_pend0;         // flows initially pending (listed in pend0 + f0)
  int32_t c0, nc;          // this part's link components [c0, c0 + nc)
  int32_t n_solve;         // solve-once: active flows listed in act0 + f0
  int32_t scen;            // the scenario the part belongs to
  int32_t lds_paths;       // every path has <= 6 links and the part < 65535 links
  // event-loop position, saved when a launch stops and read when the next
  // one continues (Params::resume)
  int32_t started;         // 1 once a launch has run the part
  int32_t e, q, ab;        // event index, completion-list phase, slot buffer
  int32_t nslots, holes, npend;  // slots in use, holes among them, pending flows
  // results
  double t;                // simulated time reached
  int64_t events, solves, rounds, flows_swept, incidences_swept;
  int64_t active_swept, pending_swept;
  int64_t reselected, wide_solves;
  int64_t assisted;        // re-solves run by helper workgroups (cluster kernel)
  int64_t links_swept;     // links with unfrozen flows summed over link passes
  // rollback history of the part (hcap = 0: none): undo records
  // hist[hbase + (i mod hcap)] for i < hpos, event records hev[ebase + (e mod ecap)]
  int64_t hpos, hbase, hcap, ebase, ecap;
  int64_t launch_events;   // events processed by the last launch
  int32_t status;          // 0 ran to the end, 1 stopped at a limit, < 0 fault
  int32_t reserved;
  int64_t ticks[8];        // wall-clock ticks per phase (first thread of the group)
  int64_t dbg[4];          // debug checks (options.debug)
  Lists k;                 // list counters in global memory (grid layout)
};

enum : int32_t {
  ST_DONE = 0,
  ST_STOPPED = 1,
  ST_BAD_SHARE = -3,       // non-positive or non-finite fair share
  ST_ROUNDS = -5,          // round watchdog
  ST_BARRIER = -6,         // grid barrier timed out
  ST_OVERFLOW = -7         // a work list exceeded its capacity
};

// Counters of a wide exact solve run by the sweep kernels (sweep.hip), in
// device memory.  The unfrozen-flow and live-link lists are kept in
// per-workgroup segments: workgroup b of a sweep owns entries
// [b * seg, (b + 1) * seg) of its list and its count, so a sweep compacts
// with shared-memory counters only.  Per-workgroup results (minima, counts,
// statistics) go to arrays that the next kernel (or the host) reduces: no
// two workgroups update one word, since atomics on one address serialise in
// the L2.  Header first (the host reads it).
constexpr int XG_MAX_BLOCKS = 8192;
struct XGridHead {
  int32_t fault;           // 1: a non-positive or infinite level minimum
  int32_t done;            // 1 once a level started with no unfrozen flow
  int32_t ublocks, useg;   // freezing sweep: workgroups, entries per segment
  int32_t lblocks, lseg;   // link pass: workgroups, entries per segment
  unsigned long long levels, fsw;  // iterations; flows swept
  double sstar[2];         // level minimum, by parity (bottleneck pass -> freezing sweep)
};
struct XGrid : XGridHead {
  int32_t ucnt[2][XG_MAX_BLOCKS];  // unfrozen flows per segment, by level parity
  int32_t lcnt[2][XG_MAX_BLOCKS];  // live links per segment, by level parity
  double bmin[2][XG_MAX_BLOCKS];   // per-workgroup minimum share of the link pass, by parity
  unsigned long long isw[XG_MAX_BLOCKS];  // incidences swept, per freezing-sweep workgroup
  unsigned long long lsw[XG_MAX_BLOCKS];  // links whose share was computed, per link-pass workgroup
};

struct Params {
  int32_t num_scen;
  int32_t mode;            // 0 event loop, 1 one rate solve per scenario
  int32_t resume;          // 1: continue every started part from its saved position
  int64_t max_events;      // 0 = no limit
  double until;
  int32_t max_rounds;
  int32_t debug;           // run internal consistency checks
  int32_t assist_min;      // cluster kernel: smallest re-solve handed to helper workgroups
  int32_t assist_helpers;  // cluster kernel: helper workgroups per leader (at most)
  int32_t clusters_per_xcd;  // cluster kernel: leaders (with their helpers) per XCD
  double scale;            // fixed-point units per B/s (a power of two)
  double inv_scale;
  // static flow / link data (device order)
  const int32_t* poff;     // [F+1] path offsets
  const int32_t* plink;    // [nnz] device link ids
  const double* nbytes;    // [F]
  const double* start;     // [F]
  const int32_t* soff;     // [F+1] successor offsets
  const int32_t* succ;     // [nsucc]
  const int64_t* R0;       // [L] capacity in fixed point
  const double* lat;       // [F] path latency (the sum over its links), or NULL: none
  const uint4* path16;     // [F] path as six 16-bit part-local link ids (0xFFFF =
                           //     none; valid in parts with lds_paths)
  // dynamic flow state
  double* rem;             // [F] bytes left at time tref (active flows)
  double* tref;            // [F] time at which rem was last brought up to date
  double* rate;            // [F] current rate
  double* finish;          // [F] completion time (NaN until finished)
  double* mf;              // [F] smallest fair share on the path (current round)
  uint4* stage;            // [F] path records of a solve's items, by item (per part on [f0, f1))
  double* rel;             // [F] release time (set when a flow is released or pending)
  double* base;            // [F] release base: finish time of the last predecessor
  int32_t* cnt;            // [F] predecessors not yet finished
  int32_t* evr;            // [F] event (index in the part) at which the flow's last
                           //     predecessor finished (EV_NEVER: not yet or none)
  int32_t* eva;            // [F] event at which it became active (or, zero bytes, finished)
  int32_t* evd;            // [F] event at which it finished
  HistUndo* hist;          // rollback history (NULL: none), ring per part
  HistEv* hev;
  const int32_t* comp;     // [F] component of the flow (flows of different
                           //     components share no link)
  uint64_t* theta;         // [C] per component: lowest level that may change
                           //     in this event (bit pattern of a double)
  // dynamic link state
  int64_t* lst;            // [2L] per link: residual capacity (fixed point), unfrozen flows
  int32_t* nact;           // [L] active flows
  uint32_t* fl;            // [L] number of the freezing round that blocked the link
  // slots of the active flows (two buffers) and work lists, each [F], used per
  // part on [f0, f1)
  int32_t* act0; int32_t* act1;  // slot: flow id, -1 for a hole
  double* tau0; double* tau1;    // slot: predicted completion time
  double* srate0; double* srate1;  // slot: rate
  int32_t* arrslot;        // slot of each entry of the re-solve list
  int32_t* pend0; int32_t* pend1;
  int32_t* comp0; int32_t* comp1; int32_t* comp2;
  int32_t* unf0; int32_t* unf1;
  int32_t* arr;            // flows activated in the current event
  // exact mode (the oracle's arithmetic; exact.hip), per device link
  const double* capf;      // [L] capacity in B/s
  double* xR;              // [L] residual capacity (fp64)
  double* xs;              // [L] fair share of the current level
  int32_t* xn;             // [L] unfrozen flows
  int32_t* xk;             // [L] flows frozen at the current level
  int32_t* xlive0; int32_t* xlive1;  // [L] links with unfrozen flows (per part on [l0, l1))
  // link-major incidence (exact mode): the flows of device link l are
  // lfid[lfoff[l] .. lfoff[l+1]-1] (ascending); lfchunk[c] is the link of
  // entry 256 c (the last link with lfoff[l] <= 256 c)
  const int32_t* lfoff;    // [L+1]
  const int32_t* lfid;     // [nnz]
  const int32_t* lfchunk;  // [nnz/256 + 1]
  const uint64_t* lfhead;  // [(nnz + 256)/64 + 1] bit e: entry e starts a link (or e >= nnz)
  uint32_t* xmask;         // [F/32 + 1] bit f: flow f is active in the wide exact solve
  uint8_t* xfz;            // [L] 1: the link is a bottleneck of the current level
  XGrid* xgrid;            // counters of a wide exact solve
  int32_t exact_lds_bytes; // dynamic shared memory of the exact kernel (link state
                           // of a part with at most exact_lds_bytes / 24 links)
  ScenCtl* ctl;            // [num_scen]
  uint32_t* bar;           // synchronisation words [BAR_WORDS] (layout in kernels.hip)
  uint64_t* slots;         // grid min-reduction slots [4]
};

// Words of Params::bar, cleared before every launch: 9,216 words of
// barrier, registration and cluster words, then the cluster helpers'
// arrival lines (64 clusters x 32 lines of 32 words).
constexpr int BAR_WORDS = 9216 + 64 * 32 * 32;

hipError_t launch_block(const Params& p, int blocks, int threads, hipStream_t s);
hipError_t launch_grid(const Params& p, int blocks, int threads, hipStream_t s);
// Largest co-resident grid for launch_grid at `threads` per block.
hipError_t grid_capacity(int device, int threads, int* blocks);
// One leader workgroup per XCD running the event loops of the parts, the
// other workgroups of its XCD solving its large re-solves (cooperative
// launch, 1024 threads per workgroup; blocks from cluster_capacity).
hipError_t launch_cluster(const Params& p, int blocks, hipStream_t s);
hipError_t cluster_capacity(int device, int* blocks);
// Exact mode: one workgroup per part (one part per scenario), the oracle's
// arithmetic (exact.hip); p.exact_lds_bytes of dynamic shared memory.
hipError_t launch_exact(const Params& p, int blocks, int threads, hipStream_t s);
// Part p (flows [f0, f1)) back to the end of its event es from the rollback
// history (history.hip): rec is the record of event es, hpos_now the undo
// records written so far; cnt0 and rel0 (device, [f1 - f0]) the part's
// initial predecessor counts and release times; first ([f1 - f0]) and
// counters ([2]) device scratch.  Asynchronous on st.
hipError_t history_restore(const Params& P, int p, int f0, int f1, int64_t hbase, int64_t hcap, int32_t es,
                           const HistEv& rec, int64_t hpos_now, const int32_t* cnt0, const double* rel0,
                           int32_t* first, uint32_t* counters, hipStream_t st);
// Bytes of exact-mode link state per link.
int exact_link_bytes();
// A wide exact solve of part C's n flows listed in act0 + C.f0, on the whole
// GPU (sweep.hip): begin (clear link state, mark the flows), count (per-link
// unfrozen counts over the part's link-major incidences [e0, e1)), then per
// level j = 0, 1, ... links and freeze, until xgrid->done or
// xgrid->cu[j & 1] is 0.
hipError_t grid_solve_begin(const Params& P, const ScenCtl& C, int n, hipStream_t s);
hipError_t grid_solve_count(const Params& P, const ScenCtl& C, int e0, int e1, hipStream_t s,
                            unsigned long long* stamps = nullptr);
hipError_t grid_solve_links(const Params& P, const ScenCtl& C, int j, hipStream_t s);
hipError_t grid_solve_freeze(const Params& P, const ScenCtl& C, int n, int j, hipStream_t s,
                             unsigned long long* stamps = nullptr);
// Workgroups of the count and freezing sweeps.  With `stamps` (device,
// 2 x workgroups words) each workgroup's first thread writes the wall clock
// (100 MHz) at its start and end: the sweep's duration inside the kernel.
int count_blocks(int e0, int e1);
int freeze_blocks(int n);
// Streaming write of `bytes` (a multiple of 16) over buf.
hipError_t launch_flush(void* buf, size_t bytes, uint32_t tag, hipStream_t s);

}  // namespace netsim_dev

namespace netsim_host {
// Message returned by netsim_last_error(NULL) on the calling thread.
void set_thread_error(const char* msg);
}  // namespace netsim_host
