/*
 * netsim -- flow-level network simulator with max-min fair bandwidth
 * sharing, solved on an AMD Instinct MI355X (gfx950).
 *
 * What is computed (the communication-time model of the paper's simulator:
 * Section 4.1, the description of netsim, and Section 4.2, the paragraph on
 * the network simulator with time rollback):
 *   - collectives are decomposed into point-to-point flows over a cluster
 *     topology (ring all-reduce / reduce-scatter / all-gather as NCCL's ring
 *     would run them, all-to-all, pipeline send/recv);
 *   - each flow follows one route chosen by the topology's multipath
 *     (ECMP) rule;
 *   - at every instant the rates of the active flows are their max-min fair
 *     (per-flow fair) allocation over the link capacities, and stay constant
 *     between consecutive events;
 *   - an event loop advances simulated time to the next flow arrival or
 *     completion and re-solves the rates; the output is every flow's
 *     completion time.
 *
 * Conventions for every entry point:
 *   - Units: bytes, seconds, bytes per second.
 *   - Pointers are host pointers unless the name says "device".  The caller
 *     owns every array it passes; the library copies what it keeps before
 *     the call returns.  Outputs go to caller-provided buffers.
 *   - Every call returns a netsim_status and never aborts.  On failure the
 *     handle is unchanged and netsim_last_error() describes the problem.
 *   - A handle is not thread-safe; distinct handles may be used from
 *     distinct threads.
 *   - Flow ids are assigned consecutively from 0 in the order flows are
 *     added (across all scenarios of the handle).
 *   - Link ids passed in or out are local to their scenario: 0 .. L_s-1.
 */
#ifndef NETSIM_H
#define NETSIM_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct netsim netsim_t;
typedef int32_t netsim_status;

enum {
  NETSIM_OK = 0,
  NETSIM_E_INVALID = -1, /* bad argument (NULL, out of range, non-finite, ...) */
  NETSIM_E_NOMEM = -2,   /* host or device allocation failed                  */
  NETSIM_E_DEVICE = -3,  /* HIP error, or the device solver reported a fault  */
  NETSIM_E_STATE = -4,   /* call not allowed in the handle's current state    */
  NETSIM_E_LIMIT = -5    /* a size limit or the per-solve round watchdog      */
};

/* Built-in fabrics (netsim_topology.kind). */
enum { NETSIM_TOPO_LEAF_SPINE = 1, NETSIM_TOPO_RAIL = 2, NETSIM_TOPO_FAT_TREE = 3 };
/* Ring collectives (netsim_add_ring kind). */
enum { NETSIM_RING_ALLREDUCE = 0, NETSIM_RING_REDUCE_SCATTER = 1, NETSIM_RING_ALL_GATHER = 2 };
/* Ring decomposition (netsim_add_ring mode). */
enum { NETSIM_MODE_CHAINED = 0, NETSIM_MODE_FLAT = 1, NETSIM_MODE_AGGREGATED = 2 };
/* Execution layout (netsim_options.exec). */
enum {
  NETSIM_EXEC_AUTO = 0,  /* grid for a single part with > 65536 flows without
                            predecessors; cluster with at most 4 parts per XCD
                            and a part with > 16384 of them; else block        */
  NETSIM_EXEC_GRID = 1,  /* whole GPU on one part at a time (grid barriers)      */
  NETSIM_EXEC_BLOCK = 2,  /* one workgroup per part (workgroup barriers)         */
  NETSIM_EXEC_CLUSTER = 3, /* leader workgroups (one per XCD, or up to 4 per XCD
                             when there are more parts than XCDs) run parts as
                             in block mode and hand re-solves of at least
                             assist_min_flows flows to assist_helpers other
                             workgroups of their XCD (one workgroup per CU,
                             cooperative launch); results equal block mode's
                             bit for bit.  Rate solves without an
                             event loop (netsim_solve_once) run as in block mode */
  NETSIM_EXEC_EXACT = 4   /* reported in netsim_stats.layout when
                             netsim_options.exact is set (one workgroup per
                             scenario, the exact-arithmetic kernel)            */
};

/*
 * Parts.  The flows of a scenario fall into groups connected through shared
 * links or dependencies; flows of different groups never influence each
 * other in the fluid model.  By default each group is simulated as its own
 * "part" with its own clock (several parts run concurrently on the GPU), and
 * the finish times are those of one clock per scenario up to rounding.
 * Events are counted per part: an instant at which two parts both have an
 * event counts twice.  single_clock = 1 keeps every scenario one part (one
 * clock), which counts events exactly as one event loop over the scenario.
 */
typedef struct {
  int32_t device;            /* HIP device ordinal                               */
  int32_t exec;              /* NETSIM_EXEC_*                                    */
  int64_t max_events;        /* stop each part after this many events; 0 = no limit */
  double until;              /* do not process events later than this time (s); +inf = none */
  int32_t max_rounds;        /* per-solve round watchdog; 0 = number of flows + 1 */
  int32_t block_threads;     /* threads per workgroup in block mode; 0 = 1024 if
                                a part has > 16384 flows without predecessors,
                                else 512                                        */
  int32_t debug;             /* bit 0: consistency checks on the device; bit 1:
                                phase timers (netsim_stats.phase_seconds); test
                                hooks of NETSIM_EXEC_CLUSTER: bit 2 makes helper
                                workgroups leave as soon as they have no job (the
                                leaders then solve alone), bit 3 makes their
                                barrier give up at once (the run then fails with
                                NETSIM_E_DEVICE, "grid barrier timed out"); bit
                                4 keeps exact-mode link state in global memory
                                even where it fits shared memory; bit 5 runs
                                every exact-mode solve_once on the whole GPU;
                                bit 6 makes every release of NETSIM_EXEC_CLUSTER
                                an agent-scope release fence (slower; results
                                are the same bit for bit)                       */
  int32_t single_clock;      /* 1: one part (one clock) per scenario             */
  int32_t assist_min_flows;  /* NETSIM_EXEC_CLUSTER: smallest re-solve handed to the
                                helper workgroups; 0 = 4096                      */
  int32_t assist_helpers;    /* NETSIM_EXEC_CLUSTER: helper workgroups per leader,
                                at most the other workgroups of its cluster (an
                                XCD's workgroups shared among its leaders); 0 = 15 */
  int32_t exact;             /* 1: the arithmetic of a sequential fp64 program
                                (Section 4.2's water-filling taken literally):
                                one clock per scenario (single_clock implied);
                                each rate solve freezes one bottleneck level per
                                iteration -- s_l = R_l/n_l, s* = min_l s_l, every
                                link with s_l <= s*(1 + 1e-12) is a bottleneck
                                and its unfrozen flows get rate s*, then
                                R_l -= k_l*s* (product rounded, then the
                                difference), n_l -= k_l; every active flow's
                                remaining bytes drop by rate*(t_next - t) at
                                every event; a flow finishes when
                                t + rem/rate <= t_next(1 + 1e-12).  One workgroup
                                per scenario (exec, assist_* ignored; stats.layout
                                = NETSIM_EXEC_EXACT).  Finish times are the same
                                bit for bit for any workgroup size.  0: the
                                default solver (local-minimum rounds, int64
                                residuals, remaining bytes updated when a rate
                                changes, independent parts on their own clocks):
                                the same allocation in exact arithmetic, with
                                different rounding                              */
  int32_t history_mb;        /* MiB of device memory for the rollback history
                                (Section 4.2: the throughput history of every
                                flow): per part a ring of undo records (32 bytes
                                per flow re-solved in an event) and of event
                                records (80 bytes each), shared among the parts
                                in proportion to their flows.  With it,
                                netsim_update_start returns a part to the end of
                                its last event before the changed release, as
                                long as the ring still holds every record since
                                and every launch since t = 0 kept it; otherwise
                                (and with 0, the default) to the latest
                                checkpoint before it.  The cluster layout and
                                exact mode keep no history; with history_mb > 0
                                NETSIM_EXEC_AUTO uses the block layout where it
                                would pick the cluster one                      */
} netsim_options;

/*
 * Built-in fabric.  Directed links; a cable is two links at full rate.
 * Inside a server every ordered GPU pair has its own link (nvlink_Bps).
 *   LEAF_SPINE: servers_per_leaf servers per leaf; every GPU has a NIC to its
 *               leaf; every leaf has one cable to each of `spines` spines.
 *   RAIL:       rail-optimised: local GPU g of the servers_per_leaf servers
 *               of a group attaches to leaf (g, group); leaves as above.
 *   FAT_TREE:   pods x (edges_per_pod edge + aggs_per_pod aggregation
 *               switches); servers_per_leaf servers per edge switch
 *               (servers = pods*edges_per_pod*servers_per_leaf); each edge has
 *               one cable to every aggregation switch of its pod; aggregation
 *               switch a has agg_uplinks cables to cores a*agg_uplinks + u.
 * Link numbering: intra-server links first (server s, pair i->j:
 *   s*G*(G-1) + i*(G-1) + (j<i ? j : j-1)), then cable c gives links
 *   NV+2c (upwards) and NV+2c+1 (downwards).  Cables: the NIC of GPU h is
 *   cable h; LEAF_SPINE/RAIL leaf-spine cables N + leaf*spines + spine
 *   (RAIL leaf = g*groups + group); FAT_TREE edge-agg cables
 *   N + (pod*E + e)*A + a, then agg-core cables N + P*E*A + (pod*A + a)*U + u.
 * Routes: same server -> its one link; same leaf/edge -> NIC up, NIC down;
 *   otherwise up through the tiers and down again, picking the spine (or
 *   aggregation switch a = h mod A and core uplink u = (h / A) mod U) from
 *   h = mix(mix(ecmp_seed) ^ (src << 32 | dst)), mix = SplitMix64's output
 *   function.
 * degraded_cables (num_degraded entries, may be NULL when 0): cable ids whose
 * two links run at degraded_Bps.  Copied by netsim_create_topology.
 * Latency (the flow model's bandwidth sharing is instantaneous; this adds
 * propagation): every intra-server link takes nvlink_latency_s seconds, every
 * cable direction fabric_latency_s (finite, >= 0; 0 = none).  A flow arrives
 * the sum of its path's latencies after its last byte leaves; see
 * netsim_set_link_latency.
 */
typedef struct {
  int32_t kind;
  int32_t servers;
  int32_t gpus_per_server;
  int32_t servers_per_leaf;
  int32_t spines;
  int32_t pods;
  int32_t edges_per_pod;
  int32_t aggs_per_pod;
  int32_t agg_uplinks;
  int32_t reserved;
  double nvlink_Bps;
  double nic_Bps;
  double fabric_Bps;
  uint64_t ecmp_seed;
  int64_t num_degraded;
  const int64_t* degraded_cables;
  double degraded_Bps;
  double fabric_latency_s;
  double nvlink_latency_s;
} netsim_topology;

typedef struct {
  int64_t events;            /* event-loop iterations (arrivals/completions)    */
  int64_t solves;            /* max-min rate solves                              */
  int64_t rounds;            /* freezing rounds over all solves                  */
  int64_t flows_swept;       /* sum over rounds of unfrozen flows visited        */
  int64_t incidences_swept;  /* sum over rounds of their flow-link incidences    */
  int64_t active_swept;      /* sum over events of active flows visited          */
  int64_t pending_swept;     /* sum over events of pending flows visited         */
  int64_t completed_flows;   /* flows with a finish time                         */
  int64_t reselected;        /* sum over solves of flows whose rate was re-solved */
  int64_t wide_solves;       /* solves that needed work lists in global memory     */
  int32_t complete;          /* 1 if every scenario ran to its end               */
  int32_t parts;             /* independent parts simulated (see netsim_options) */
  double sim_time;           /* largest simulated time reached over scenarios    */
  double device_seconds;     /* device time of the last netsim_run (HIP events)  */
  double upload_seconds;     /* host->device preparation of the last run          */
  /* Device time by phase, summed over parts, as seen by the first thread of
   * the group running each part (only with debug bit 1; zero otherwise):
   * [0] next-event search, [1] settling completions and releases, [2] solve
   * set-up and the share table of every round, [3] share/blocking sweep, [4]
   * wait after it, [5] freezing sweep, [6] wait after it, [7] choosing the
   * flows to re-solve.  In the cluster layout a re-solve run by helper
   * workgroups counts with the first helper's times in [2]-[6]; the hand-over
   * itself (copying link state, waking the helpers) is not counted. */
  double phase_seconds[8];
  int64_t assisted_solves;   /* NETSIM_EXEC_CLUSTER: re-solves run by the helper
                                workgroups (counted in solves and rounds too)    */
  int32_t layout;            /* execution layout of the last launch (NETSIM_EXEC_GRID,
                                _BLOCK, _CLUSTER or _EXACT; AUTO resolved)        */
  int32_t reserved;
  int64_t links_swept;       /* sum over rounds of the links whose share the round
                                computed (links with unfrozen flows): every level
                                of exact mode; the share-table passes of the
                                default solver (rounds run by helper workgroups,
                                which have no such pass, add nothing)            */
  int64_t launch_events;     /* events processed by the last launch, summed over
                                parts (a continuation after a rollback re-simulates
                                only from where the part went back to)           */
} netsim_stats;

/* Fills *opt with the defaults (device 0, auto layout, no limits, default solver). */
void netsim_default_options(netsim_options* opt);

/*
 * Explicit topology (Section 4.1: netsim is configured with the cluster
 * topology -- its links and their bandwidths; here directed links with their
 * capacities in bytes per second).  Several independent scenarios per handle
 * are the batched what-if mode: num_scenarios independent scenarios; scenario s owns
 * links link_off[s] .. link_off[s+1]-1 of capacity_Bps (link_off has S+1
 * entries, link_off[0] = 0, non-decreasing).  Capacities must be finite and
 * > 0.  opt may be NULL (defaults).  Flows must then carry explicit paths.
 * No device work happens until netsim_run.
 */
netsim_status netsim_create(netsim_t** out, int32_t num_scenarios, const int64_t* link_off,
                            const double* capacity_Bps, const netsim_options* opt);

/* Built-in fabrics, one per scenario (topos[num_scenarios]): the topology
 * configuration of Section 4.1, with its multipath routing (ECMP) rule. */
netsim_status netsim_create_topology(netsim_t** out, int32_t num_scenarios,
                                     const netsim_topology* topos, const netsim_options* opt);

/* Number of links of scenario scen, and their capacities (cap_out[L_s], may be
 * NULL): the links a built-in fabric created (Section 4.1 topology). */
netsim_status netsim_get_links(const netsim_t* h, int32_t scen, int64_t* num_links,
                               double* cap_out);

/*
 * Appends n flows to scenario scen (Section 4.1: the communication the
 * simulator intercepts becomes flows between GPUs over the topology;
 * Section 4.1's event queue releases an operation only after the ones it
 * depends on, here dependencies between flows).  Flow i: endpoints src[i] -> dst[i]
 * (GPU ranks; may be NULL when paths are given), nbytes[i] >= 0, start[i] >= 0.
 * Path: if path_off is NULL the built-in router chooses it from (src, dst);
 * otherwise flow i crosses links path_link[path_off[i] .. path_off[i+1]-1]
 * (path_off[0] = 0, n+1 entries, local link ids, no link twice).
 * Dependencies (dep_off may be NULL = none): flow i waits for the flows
 * dep_ids[dep_off[i] .. dep_off[i+1]-1], ids of earlier flows of the same
 * scenario (which keeps the graph acyclic).  A flow with no dependencies
 * is released at start[i]; one with dependencies at start[i] + the latest
 * finish time among them.  A zero-byte flow takes no route and finishes at
 * its release time (a barrier).  bytes > 0 with src == dst or with an
 * empty path is invalid.  *first_id (may be NULL) receives the first id.
 */
netsim_status netsim_add_flows(netsim_t* h, int32_t scen, int64_t n, const int32_t* src,
                               const int32_t* dst, const double* nbytes, const double* start,
                               const int64_t* path_off, const int32_t* path_link,
                               const int64_t* dep_off, const int64_t* dep_ids,
                               int64_t* first_id);

/*
 * Ring collective over ranks[0..p) (distinct, p >= 2) of `nbytes` in total
 * on a built-in fabric (Section 4.1: all-reduce as NCCL's ring).  Steps:
 * 2(p-1) for all-reduce, p-1 for reduce-scatter / all-gather; in every step
 * position i sends nbytes/p (fp64 division) from ranks[i] to ranks[(i+1)%p].
 * CHAINED: step k out of position i waits for step k-1 into position i;
 * FLAT: all steps released together; AGGREGATED: one flow per ring edge of
 * steps*(nbytes/p).  Flows are numbered step-major (first + k*p + i).  The
 * first step (every flow, when not chained) waits for the n_after flows in
 * after[] and then `lag` seconds.  *first_id and *count may be NULL.
 */
netsim_status netsim_add_ring(netsim_t* h, int32_t scen, int32_t kind, int32_t mode, int32_t p,
                              const int32_t* ranks, double nbytes, double lag, int64_t n_after,
                              const int64_t* after, int64_t* first_id, int64_t* count);

/*
 * All-to-all among ranks[0..p) (distinct): flow (i, j), j != i, carries
 * nbytes[i*p + j] (row-major p x p; the diagonal is ignored), numbered
 * row-major skipping the diagonal.  Every flow waits for after[] then lag.
 */
netsim_status netsim_add_all_to_all(netsim_t* h, int32_t scen, int32_t p, const int32_t* ranks,
                                    const double* nbytes, double lag, int64_t n_after,
                                    const int64_t* after, int64_t* first_id, int64_t* count);

/*
 * Richer collectives (Section 6 names replacing the plain ring algorithm by
 * NCCL-like ones as a route to accuracy).  Same conventions as
 * netsim_add_ring (ranks distinct endpoints of the scenario's built-in
 * fabric, bytes and lag finite >= 0, `after` flows of the same scenario;
 * *first_id / *count may be NULL; NETSIM_E_STATE after the first run).
 *
 * netsim_add_tree_allreduce: double binary tree over ranks[0..p) (p >= 2).
 * Node numbers u = 1..p; node u of level l = (trailing zero bits of u) >= 1
 * has children u - 2^(l-1) and u + 2^j for the largest j < l with
 * u + 2^j <= p (if any); the root is the largest power of two <= p.  Tree A
 * puts ranks[u-1] at node u, tree B (the mirror) ranks[p-u].  Per tree and
 * edge (child c, parent q): a reduce flow c -> q of nbytes/2 after the reduce
 * flows into c (leaves: after `after`, released `lag` later), and a
 * broadcast flow q -> c after the broadcast flow into q (q the root: after
 * every reduce flow into the root).  Layout: tree A reduce (children by
 * level, lowest first, then node), tree A broadcast (by level, highest
 * first, then node), tree B reduce, tree B broadcast: 4(p-1) flows.
 *
 * netsim_add_hier_allreduce: ranks is an m x g array, row-major (row s: the
 * g ranks of server s), m*g >= 2.  Phase 1 (g > 1): per server, a chained
 * ring reduce-scatter over its row, chunks nbytes/g, step-major per server;
 * phase 2 (m > 1): per column j, a chained ring all-reduce over the m rows,
 * chunks nbytes/(g*m), 2(m-1) steps, step-major per column; phase 3 (g > 1):
 * per server a chained ring all-gather like phase 1.  A rank's first step of
 * a phase waits for its previous phase's last-step flows out of and into
 * it (the first phase: for `after`, released `lag` later).
 */
netsim_status netsim_add_tree_allreduce(netsim_t* h, int32_t scen, int32_t p, const int32_t* ranks,
                                        double nbytes, double lag, int64_t n_after,
                                        const int64_t* after, int64_t* first_id, int64_t* count);
netsim_status netsim_add_hier_allreduce(netsim_t* h, int32_t scen, int32_t m, int32_t g,
                                        const int32_t* ranks, double nbytes, double lag,
                                        int64_t n_after, const int64_t* after, int64_t* first_id,
                                        int64_t* count);

/*
 * The exit flows of the operation appended by the last successful call of
 * netsim_add_ring, netsim_add_all_to_all, netsim_add_tree_allreduce,
 * netsim_add_hier_allreduce or netsim_add_flows on h: the flows a later
 * operation that depends on it waits for (Section 4.1: a collective is
 * complete on a rank when its pattern's last transfers are; taken as a
 * chained ring's last step, every flow of a flat or aggregated ring, of an
 * all-to-all and of a batch of flows, a double binary tree's broadcast
 * flows, a hierarchical all-reduce's last phase's last step), ascending.
 * *n receives their number; ids (may be NULL) receives the *n ids.
 * NETSIM_E_STATE before any such call.
 */
netsim_status netsim_last_exits(const netsim_t* h, int64_t* n, int64_t* ids);

/*
 * Per-link latency of scenario `scen` (num_links = its link count, values
 * finite >= 0, copied), replacing what its built-in fabric set.  A flow
 * sends at its max-min rate as before and frees its links when its last byte
 * leaves; it finishes (its finish time, and the release base of its
 * dependants) the sum of its path's latencies later, summed in path order.
 * NETSIM_E_STATE after the first run.
 */
netsim_status netsim_set_link_latency(netsim_t* h, int32_t scen, int64_t num_links,
                                      const double* latency_s);

/*
 * Event-queue front end (Section 4.1: the simulator's event queue emulates
 * CUDA streams and events -- operations on one stream run in order,
 * operations on different streams are independent unless linked by an
 * event; an NCCL collective starts its flows only once every rank of the
 * communicator has reached it; a stream synchronisation returns the
 * completion time of the stream's last operation).
 *
 * Streams are the caller's int64 ids within a scenario (a stream belongs to
 * one rank; ids need not be dense).  Every call appends flows and returns
 * the id of the zero-byte flow that marks the operation's completion on
 * each participating stream (it becomes that stream's tail).  After a run,
 * the finish time of a stream's tail is what a synchronisation on the
 * stream returns; a tail recorded at some point serves as a CUDA event.
 * A computation of d seconds is a zero-byte flow released d after the
 * stream's tail and the flows it waits for.  A collective or send first
 * appends a rendezvous (zero-byte flow after the tails of every
 * participating stream), then its flows after it (as netsim_add_ring /
 * netsim_add_all_to_all / one routed flow), then per rank a completion flow
 * after the flows out of and into that rank that finish last (chained ring:
 * the last step's; flat ring and all-to-all: all of them; aggregated ring:
 * its two edges).  Built-in fabrics only for communication.  NETSIM_E_STATE
 * after the first run; on error nothing is appended.
 */
netsim_status netsim_stream_compute(netsim_t* h, int32_t scen, int64_t stream, double duration,
                                    int64_t n_wait, const int64_t* wait, int64_t* done);
/* cudaStreamWaitEvent: the stream's next operation also waits for wait[]. */
netsim_status netsim_stream_wait(netsim_t* h, int32_t scen, int64_t stream, int64_t n_wait,
                                 const int64_t* wait);
/* The stream's current tail (-1 for a stream without operations). */
netsim_status netsim_stream_tail(const netsim_t* h, int32_t scen, int64_t stream, int64_t* flow);
/* Ring collective of ranks[i] issued on streams[i] (distinct); done[p]. */
netsim_status netsim_stream_ring(netsim_t* h, int32_t scen, int32_t kind, int32_t mode, int32_t p,
                                 const int32_t* ranks, const int64_t* streams, double nbytes,
                                 int64_t* done);
/* All-to-all of ranks[i] issued on streams[i]; nbytes as netsim_add_all_to_all; done[p]. */
netsim_status netsim_stream_all_to_all(netsim_t* h, int32_t scen, int32_t p, const int32_t* ranks,
                                       const int64_t* streams, const double* nbytes, int64_t* done);
/* Tree / hierarchical all-reduce of ranks[i] issued on streams[i] (p = m*g
 * for the latter, row-major); a rank's completion follows its broadcasts in
 * and out (tree) or its last phase's last-step flows in and out
 * (hierarchical); done[p]. */
netsim_status netsim_stream_tree_allreduce(netsim_t* h, int32_t scen, int32_t p,
                                           const int32_t* ranks, const int64_t* streams,
                                           double nbytes, int64_t* done);
netsim_status netsim_stream_hier_allreduce(netsim_t* h, int32_t scen, int32_t m, int32_t g,
                                           const int32_t* ranks, const int64_t* streams,
                                           double nbytes, int64_t* done);
/* Point-to-point send/recv: src on src_stream, dst on dst_stream (distinct);
 * *done (may be NULL) receives the completion on src_stream (the same flow
 * as dst_stream's new tail). */
netsim_status netsim_stream_send(netsim_t* h, int32_t scen, int32_t src, int64_t src_stream,
                                 int32_t dst, int64_t dst_stream, double nbytes, int64_t* done);

/* Totals over all scenarios: flows, path incidences (flow-link pairs of the
 * Section 4.2 rate solve), dependency entries. */
netsim_status netsim_counts(const netsim_t* h, int64_t* num_flows, int64_t* num_incidences,
                            int64_t* num_deps);

/*
 * Copies the flows as stored (id order; the flows of Section 4.1 with the
 * routes the fabric chose): scenario, endpoints, bytes, start,
 * path CSR (local link ids) and dependency CSR.  Any pointer may be NULL.
 * Sizes: num_flows (+1 for the offsets), num_incidences, num_deps.
 */
netsim_status netsim_export_flows(const netsim_t* h, int32_t* scen, int32_t* src, int32_t* dst,
                                  double* nbytes, double* start, int64_t* path_off,
                                  int32_t* path_link, int64_t* dep_off, int64_t* dep_ids);

/* Replaces the stopping points of later runs (see netsim_options): Section
 * 4.2's advance by a number of steps or up to a time. */
netsim_status netsim_set_limits(netsim_t* h, int64_t max_events, double until);

/*
 * The simulation (Section 4.2, the network simulator with time rollback:
 * between neighbouring events flows keep stable throughputs, the max-min
 * fair allocation found by water-filling; events are processed in time
 * order, completions releasing what depends on them).
 * Simulates every scenario from t = 0 on the device, in one kernel launch
 * (the event loop and the rate solves stay on the GPU), up to the limits of
 * netsim_options / netsim_set_limits.  hip_stream may be NULL (the default
 * stream) or a hipStream_t, e.g. torch.cuda's current stream.  Blocks until
 * the run is done.  May be called again: every call starts over from t = 0
 * with the same flows and drops the checkpoints of netsim_advance.  No flows
 * can be added after the first run (NETSIM_E_STATE).
 */
netsim_status netsim_run(netsim_t* h, void* hip_stream);

/*
 * Time rollback (Section 4.2, the network simulator with time rollback: an
 * API that updates an existing flow's start time, an API that advances the
 * simulation by steps or up to a given time, and garbage collection of the
 * history that no later update can reach).
 *
 * netsim_advance continues every part from where the last netsim_run or
 * netsim_advance stopped (from t = 0 if the handle has not run, or after
 * netsim_run was called), processing events with time <= until and at most
 * max_events more events per part (0 = no limit; a part stops before the
 * event that would exceed either limit).  Afterwards netsim_get_finish /
 * netsim_get_stats describe the position reached (statistics accumulate
 * from t = 0) and the state is kept as a checkpoint in device memory
 * (best effort: without memory for it, rollbacks go further back).
 * Advancing in several calls gives bit for bit the finish times of one
 * call with the same final limit.  Blocks until done; NETSIM_E_INVALID for a
 * NaN limit or max_events < 0.
 */
netsim_status netsim_advance(netsim_t* h, double until, int64_t max_events, void* hip_stream);

/*
 * Sets flow id's start (its absolute start when it has no dependencies, else
 * its lag after the last of them) to `start` (finite, >= 0).  If the
 * simulation of the flow's part has already processed its old or its new
 * release time, the part is rolled back (Section 4.2, time rollback): with
 * the rollback history (options.history_mb) to the end of its last event
 * before the earlier of the two releases, else to the latest checkpoint in
 * which the flow was not yet released and whose last event precedes the new
 * release (t = 0 if there is none); checkpoints after that point no longer
 * apply to the part; other parts keep their position.  The next
 * netsim_advance (or netsim_run, from t = 0) re-simulates with the new
 * start, so completion times that depended on the flow change accordingly
 * (through the dependency graph).  Valid before the first run as well.
 */
netsim_status netsim_update_start(netsim_t* h, int64_t id, double start);

/*
 * Garbage collection: the caller promises that no later netsim_update_start
 * moves a release before t_min.  Checkpoints that no rollback to t_min or
 * later can need are freed (results are unaffected: a rollback never needs
 * more than the latest checkpoint before its target).
 */
netsim_status netsim_gc(netsim_t* h, double t_min);

/* Number of checkpoints held in device memory. */
netsim_status netsim_num_checkpoints(const netsim_t* h, int64_t* n);

/*
 * The output of Section 4.1's netsim: the completion time of every flow.
 * finish[num_flows] (host) receives each flow's completion time (NaN for a
 * flow not finished when the run stopped early); makespan[num_scenarios]
 * (may be NULL) each scenario's largest finish time.  Needs a prior run.
 */
netsim_status netsim_get_finish(const netsim_t* h, double* finish, double* makespan);

/* Same as netsim_get_finish (Section 4.1's completion times), into device
 * memory d_finish[num_flows]. */
netsim_status netsim_get_finish_device(const netsim_t* h, double* d_finish);

/* Counts and times of the last run (netsim_stats above): the events of the
 * Section 4.2 event loop, its max-min rate solves and their rounds, the work
 * swept, device and upload time. */
netsim_status netsim_get_stats(const netsim_t* h, netsim_stats* stats);

/*
 * One rate solve (Section 4.2: the max-min allocation of the flows active
 * at one instant) of the flows active_ids[0..n_active) of scenario scen,
 * ignoring their start times and dependencies.  rates_out[n_active] (host)
 * receives their rates.  Ids must be distinct flows of that scenario with
 * a non-empty path.
 */
netsim_status netsim_solve_once(netsim_t* h, int32_t scen, int64_t n_active,
                                const int64_t* active_ids, double* rates_out);

/*
 * Measurement of the two sweeps of a wide exact rate solve (the link-major
 * per-link unfrozen count that starts the solve, and the first level's
 * freezing sweep over the unfrozen flows' path records), as the whole-GPU
 * solve of netsim_solve_once runs them for active_ids[0..n_active) of
 * scenario scen (handle in exact mode; every id a distinct flow of the
 * scenario with a path).  Each of `reps` repetitions first writes
 * flush_bytes (0: none) of a scratch buffer to evict the caches, then times
 * the count kernel into count_ms[r], writes the buffer again, runs the
 * level's link pass and times the freezing sweep into freeze_ms[r] (HIP
 * events on hip_stream, so dispatch is included).  count_kernel_ms and
 * freeze_kernel_ms (may be NULL) receive the same sweeps timed inside the
 * kernels: from the first workgroup's start to the last one's end on the
 * device's constant wall clock.  Allocates the scratch buffers for the call.
 * Leaves no simulation position: the next netsim_advance starts from t = 0.
 */
netsim_status netsim_bench_sweeps(netsim_t* h, int32_t scen, int64_t n_active,
                                  const int64_t* active_ids, int32_t reps, int64_t flush_bytes,
                                  void* hip_stream, double* count_ms, double* freeze_ms,
                                  double* count_kernel_ms, double* freeze_kernel_ms);

/*
 * Allocation-free rate solve, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc).  The same solve as netsim_solve_once with
 * netsim_options.exact = 1 -- every flow active, one progressive-filling
 * level per iteration in fp64 -- on arrays the caller already holds in
 * device memory, with no handle:
 *   d_capacity_Bps[num_links]      link capacities (finite, > 0);
 *   d_path_off[num_flows + 1]      int32 path offsets (d_path_off[0] = 0);
 *   d_path_link[d_path_off[num_flows]]  int32 link ids (0 .. num_links-1,
 *                                  distinct within a path, every path
 *                                  non-empty);
 *   d_rates[num_flows]             output: the max-min rate of every flow;
 *   d_status[2]                    output (int64): [0] a netsim_status
 *                                  (NETSIM_OK, NETSIM_E_INVALID for a bad
 *                                  path or capacity -- [1] then holds the
 *                                  offending flow index, or num_flows + the
 *                                  link index --, NETSIM_E_LIMIT for the
 *                                  round watchdog), [1] on success the
 *                                  number of progressive-filling iterations.
 * The call only checks its scalar arguments and enqueues one kernel on
 * hip_stream (NULL: the default stream); it never synchronises, so the
 * caller reads d_status and d_rates after the stream has reached that
 * point.  Limits: num_links <= 65536, num_flows <= 262144 (NETSIM_E_LIMIT
 * beyond).  Working memory is one static device array of about 5 MB per
 * device, held until the process ends and found once per device; nothing
 * is allocated or freed by the call.  Calls that overlap on one device
 * (different host threads, or different streams of one device) share that
 * array and race: serialise them.  The caller owns every array; none is
 * retained after the kernel ends.
 */
netsim_status netsim_solve_rates_noalloc(int32_t device, int32_t num_links,
                                         const double* d_capacity_Bps, int32_t num_flows,
                                         const int32_t* d_path_off, const int32_t* d_path_link,
                                         double* d_rates, int64_t* d_status, void* hip_stream);

/* Message of the last failure on h (or of the calling thread when h is NULL). */
const char* netsim_last_error(const netsim_t* h);

/* Frees the handle, its device memory and its rollback checkpoints (Section
 * 4.2's history); NULL is ignored. */
void netsim_destroy(netsim_t* h);

#ifdef __cplusplus
}
#endif

#endif /* NETSIM_H */
