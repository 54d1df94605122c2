// libnetsim: the C ABI of include/netsim.h (host side).
//
// Host work: argument validation, built-in fabrics and ECMP routes,
// decomposition of ring and all-to-all collectives into flows (Section 4.1:
// collectives as communication patterns, all-reduce as NCCL's ring), the
// device layout (flows grouped by scenario, links compacted to the used
// ones, successor lists, fixed-point capacities), upload, one kernel launch
// per run, and results.  Every step of the simulation itself runs in the
// HIP kernels (kernels.hip).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstring>
#include <limits>
#include <string>
#include <unordered_map>
#include <vector>

#include "device.h"
#include "fabric.h"
#include "netsim.h"

using netsim_dev::Params;
using netsim_dev::ScenCtl;

namespace {

thread_local std::string g_thread_err;

struct Scen {
  std::vector<double> cap;
  std::vector<double> lat;     // per link latency in seconds (empty: none)
  bool has_fabric = false;
  netsim_host::Fabric fab;
  std::vector<int64_t> flows;  // ids of this scenario's flows, ascending
  std::unordered_map<int64_t, int64_t> tails;  // stream -> completion flow of its last operation
};

}  // namespace

namespace netsim_host {
void set_thread_error(const char* msg) { g_thread_err = msg; }
}  // namespace netsim_host

struct netsim {
  netsim_options opt{};
  std::vector<Scen> scen;
  // flows in id order
  std::vector<int32_t> f_scen, f_src, f_dst;
  std::vector<double> f_bytes, f_start;
  std::vector<int64_t> p_off{0};
  std::vector<int32_t> p_link;
  std::vector<int64_t> d_off{0};
  std::vector<int64_t> d_ids;
  std::vector<int64_t> last_exits;    // exit flows of the last operation appended
  bool has_exits = false;
  std::string err;
  // device layout (built at the first run)
  bool prepared = false;
  bool has_result = false;
  int64_t F = 0, L = 0, nnz = 0, nsucc = 0;
  int32_t num_parts = 0;              // independent parts (each with its own clock)
  int32_t layout = 0;                 // execution layout of the last launch (NETSIM_EXEC_*)
  std::vector<int32_t> dev_of_flow;   // id -> device flow index
  std::vector<std::vector<int32_t>> dev_link;  // scenario, local link -> device link (-1 unused)
  std::vector<int32_t> h_cnt0;
  std::vector<double> h_rel0;
  std::vector<int32_t> h_pend0;
  std::vector<ScenCtl> h_ctl0;
  std::vector<int32_t> h_lfoff;       // exact mode: link-major incidence offsets
  double scale = 1.0;
  void* d_block = nullptr;            // one allocation holding every device array
  void* d_hist = nullptr;             // rollback history (options.history_mb; exact mode: none)
  bool hist_ok = false;               // every launch since t = 0 kept the history
  char* persist = nullptr;            // the persistent dynamic state inside it
  size_t persist_bytes = 0;
  bool has_state = false;             // the device holds a simulation position
  struct Checkpoint {
    void* dev = nullptr;              // copy of the persistent state
    std::vector<double> t;            // per part: time of its last processed event
    std::vector<char> valid;          // per part: still on the current history
  };
  std::vector<Checkpoint> checkpoints;
  std::vector<double> part_t;         // per part: time of its last processed event (-inf: none)
  Params prm{};
  // results
  std::vector<double> finish;         // id order
  std::vector<double> makespan;
  netsim_stats stats{};
};

namespace {

netsim_status fail(const netsim_t* h, netsim_status code, const std::string& msg) {
  if (h) const_cast<netsim_t*>(h)->err = msg;
  else g_thread_err = msg;
  return code;
}

bool finite_nonneg(double x) { return std::isfinite(x) && x >= 0.0; }

netsim_status hip_fail(const netsim_t* h, hipError_t e, const char* what) {
  return fail(h, NETSIM_E_DEVICE, std::string(what) + ": " + hipGetErrorString(e));
}

// The exit flows of the operation just appended (see netsim_last_exits).
void set_exits(netsim_t* h, int64_t f0, int64_t f1) {
  h->last_exits.resize((size_t)(f1 - f0));
  for (int64_t f = f0; f < f1; ++f) h->last_exits[(size_t)(f - f0)] = f;
  h->has_exits = true;
}
void set_exits(netsim_t* h, const std::vector<std::vector<int64_t>>& per_rank) {
  std::vector<int64_t> all;
  for (const auto& v : per_rank) all.insert(all.end(), v.begin(), v.end());
  std::sort(all.begin(), all.end());
  all.erase(std::unique(all.begin(), all.end()), all.end());
  h->last_exits = all;
  h->has_exits = true;
}

// Validates and appends n flows (all or nothing).  paths: explicit CSR or
// NULL (route with the scenario's fabric).  deps: CSR of earlier ids or NULL.
netsim_status add_flows_impl(netsim_t* h, int32_t s, int64_t n, const int32_t* src,
                             const int32_t* dst, const double* nbytes, const double* start,
                             const int64_t* path_off, const int32_t* path_link,
                             const int64_t* dep_off, const int64_t* dep_ids, int64_t* first_id) {
  if (h->prepared) return fail(h, NETSIM_E_STATE, "add_flows: flows cannot be added after a run");
  if (s < 0 || s >= (int32_t)h->scen.size()) return fail(h, NETSIM_E_INVALID, "add_flows: bad scenario");
  if (n < 0) return fail(h, NETSIM_E_INVALID, "add_flows: n < 0");
  if (n > 0 && (!nbytes || !start)) return fail(h, NETSIM_E_INVALID, "add_flows: nbytes and start are required");
  Scen& sc = h->scen[s];
  const int64_t first = (int64_t)h->f_bytes.size();
  if (first + n > std::numeric_limits<int32_t>::max())
    return fail(h, NETSIM_E_LIMIT, "add_flows: more than 2^31-1 flows");
  const bool routed = path_off == nullptr;
  if (routed) {
    if (!sc.has_fabric) return fail(h, NETSIM_E_INVALID, "add_flows: no paths given and the scenario has no built-in fabric");
    if (n > 0 && (!src || !dst)) return fail(h, NETSIM_E_INVALID, "add_flows: src and dst are required for routing");
  } else {
    if (!path_link && n > 0 && path_off[n] > 0) return fail(h, NETSIM_E_INVALID, "add_flows: path_link is NULL");
    if (n > 0 && path_off[0] != 0) return fail(h, NETSIM_E_INVALID, "add_flows: path_off[0] must be 0");
  }
  if (dep_off && n > 0 && dep_off[0] != 0) return fail(h, NETSIM_E_INVALID, "add_flows: dep_off[0] must be 0");
  if (dep_off && n > 0 && dep_off[n] > 0 && !dep_ids) return fail(h, NETSIM_E_INVALID, "add_flows: dep_ids is NULL");
  const int64_t L = (int64_t)sc.cap.size();
  const int64_t N = sc.has_fabric ? sc.fab.endpoints() : 0;
  std::vector<int32_t> links;
  std::vector<int64_t> lens((size_t)n, 0);
  int32_t hop[netsim_host::Fabric::kMaxHops];
  for (int64_t i = 0; i < n; ++i) {
    const double b = nbytes[i];
    if (!finite_nonneg(b)) return fail(h, NETSIM_E_INVALID, "add_flows: bytes must be finite and >= 0 (flow " + std::to_string(i) + ")");
    if (!finite_nonneg(start[i])) return fail(h, NETSIM_E_INVALID, "add_flows: start must be finite and >= 0 (flow " + std::to_string(i) + ")");
    if (dep_off) {
      if (dep_off[i + 1] < dep_off[i]) return fail(h, NETSIM_E_INVALID, "add_flows: dep_off must not decrease");
      for (int64_t k = dep_off[i]; k < dep_off[i + 1]; ++k) {
        const int64_t d = dep_ids[k];
        if (d < 0 || d >= first + i) return fail(h, NETSIM_E_INVALID, "add_flows: a dependency must name an earlier flow (flow " + std::to_string(i) + ")");
        if (d >= first) {
          // same batch: same scenario by construction
        } else if (h->f_scen[(size_t)d] != s) {
          return fail(h, NETSIM_E_INVALID, "add_flows: a dependency must be in the same scenario");
        }
      }
    }
    if (routed) {
      if (b == 0.0) continue;  // zero-byte flows take no route
      const int64_t a = src[i], c = dst[i];
      if (a < 0 || a >= N || c < 0 || c >= N) return fail(h, NETSIM_E_INVALID, "add_flows: endpoint out of range (flow " + std::to_string(i) + ")");
      if (a == c) return fail(h, NETSIM_E_INVALID, "add_flows: src == dst with bytes > 0 (flow " + std::to_string(i) + ")");
      const int k = sc.fab.route(a, c, hop);
      lens[(size_t)i] = k;
      links.insert(links.end(), hop, hop + k);
    } else {
      if (path_off[i + 1] < path_off[i]) return fail(h, NETSIM_E_INVALID, "add_flows: path_off must not decrease");
      const int64_t e0 = path_off[i], e1 = path_off[i + 1];
      if (b == 0.0) continue;
      if (e1 == e0) return fail(h, NETSIM_E_INVALID, "add_flows: empty path with bytes > 0 (flow " + std::to_string(i) + ")");
      if (src && dst && src[i] >= 0 && src[i] == dst[i]) return fail(h, NETSIM_E_INVALID, "add_flows: src == dst with bytes > 0");
      for (int64_t e = e0; e < e1; ++e) {
        const int32_t l = path_link[e];
        if (l < 0 || l >= L) return fail(h, NETSIM_E_INVALID, "add_flows: link id out of range (flow " + std::to_string(i) + ")");
        for (int64_t e2 = e0; e2 < e; ++e2)
          if (path_link[e2] == l) return fail(h, NETSIM_E_INVALID, "add_flows: link repeated in a path (flow " + std::to_string(i) + ")");
      }
      lens[(size_t)i] = e1 - e0;
      links.insert(links.end(), path_link + e0, path_link + e1);
    }
  }
  if ((int64_t)h->p_link.size() + (int64_t)links.size() > std::numeric_limits<int32_t>::max())
    return fail(h, NETSIM_E_LIMIT, "add_flows: more than 2^31-1 path incidences");
  // commit
  for (int64_t i = 0; i < n; ++i) {
    h->f_scen.push_back(s);
    h->f_src.push_back(src ? src[i] : -1);
    h->f_dst.push_back(dst ? dst[i] : -1);
    h->f_bytes.push_back(nbytes[i]);
    h->f_start.push_back(start[i]);
    h->p_off.push_back(h->p_off.back() + lens[(size_t)i]);
    if (dep_off) {
      for (int64_t k = dep_off[i]; k < dep_off[i + 1]; ++k) h->d_ids.push_back(dep_ids[k]);
      h->d_off.push_back(h->d_off.back() + (dep_off[i + 1] - dep_off[i]));
    } else {
      h->d_off.push_back(h->d_off.back());
    }
    sc.flows.push_back(first + i);
  }
  h->p_link.insert(h->p_link.end(), links.begin(), links.end());
  if (first_id) *first_id = first;
  return NETSIM_OK;
}

netsim_status check_after(netsim_t* h, int32_t s, int64_t n_after, const int64_t* after) {
  if (n_after < 0 || (n_after > 0 && !after)) return fail(h, NETSIM_E_INVALID, "collective: bad 'after' list");
  const int64_t F = (int64_t)h->f_bytes.size();
  for (int64_t k = 0; k < n_after; ++k)
    if (after[k] < 0 || after[k] >= F || h->f_scen[(size_t)after[k]] != s)
      return fail(h, NETSIM_E_INVALID, "collective: 'after' must name existing flows of the same scenario");
  return NETSIM_OK;
}

netsim_status check_ranks(netsim_t* h, int32_t s, int32_t p, const int32_t* ranks) {
  if (s < 0 || s >= (int32_t)h->scen.size()) return fail(h, NETSIM_E_INVALID, "collective: bad scenario");
  if (!h->scen[s].has_fabric) return fail(h, NETSIM_E_INVALID, "collective: the scenario has no built-in fabric");
  if (p > 0 && !ranks) return fail(h, NETSIM_E_INVALID, "collective: ranks is NULL");
  const int64_t N = h->scen[s].fab.endpoints();
  std::vector<int32_t> r(ranks, ranks + p);
  for (int32_t x : r)
    if (x < 0 || x >= N) return fail(h, NETSIM_E_INVALID, "collective: rank out of range");
  std::sort(r.begin(), r.end());
  if (std::adjacent_find(r.begin(), r.end()) != r.end()) return fail(h, NETSIM_E_INVALID, "collective: ranks must be distinct");
  return NETSIM_OK;
}

// ---------------------------------------------------------- device layout
struct UnionFind {
  std::vector<int32_t> p;
  explicit UnionFind(size_t n) : p(n) {
    for (size_t i = 0; i < n; ++i) p[i] = (int32_t)i;
  }
  int32_t find(int32_t x) {
    while (p[(size_t)x] != x) {
      p[(size_t)x] = p[(size_t)p[(size_t)x]];
      x = p[(size_t)x];
    }
    return x;
  }
  void unite(int32_t a, int32_t b) {
    a = find(a);
    b = find(b);
    if (a != b) p[(size_t)std::max(a, b)] = std::min(a, b);
  }
};

// Largest number of parts a scenario is split into; beyond it consecutive
// groups share a part (and its clock), which is always allowed.
constexpr int32_t kMaxPartsPerScen = 1024;
// Link components per part for the incremental re-solve; more are merged
// into the last one (a coarser partition is still safe).
constexpr int32_t kMaxComp = 4096;
// Cluster layout: smallest re-solve the helper workgroups take by default;
// compute units per XCD on gfx950 (the number of leaders is CUs / this).
constexpr int32_t kAssistMinFlows = 4096;
// helper workgroups per leader by default (measured on the 4096-GPU
// all-to-all: 7 -> 10.7 s, 11-17 -> 9.7-10.1 s, 23 -> 10.0 s, 31 -> 10.9 s)
constexpr int32_t kAssistHelpers = 15;
// leaders per XCD at most (the cluster kernel's word layout has room for 4)
constexpr int kMaxClustersPerXcd = 4;
constexpr int kCusPerXcd = 32;
// Exact mode: dynamic shared memory for link state (24 bytes per link: up
// to 6,485 links per part) and threads per workgroup.
constexpr int64_t kExactLdsBytes = 152 * 1024;
constexpr int kExactThreads = 512;
// Exact mode: a rate solve without an event loop of at least this many flows
// runs on the whole GPU (sweep.hip) instead of one workgroup; levels are
// enqueued this many at a time between looks at the unfrozen count.
constexpr int32_t kExactGridMin = 16384;
constexpr int kGridLevelBatch = 64;
constexpr int DEBUG_EXACT_GRID = 32;  // options.debug bit 5: every such solve on the whole GPU

netsim_status prepare(netsim_t* h) {
  const int32_t S = (int32_t)h->scen.size();
  const int64_t F = (int64_t)h->f_bytes.size();
  h->F = F;
  // Parts: the flows of a scenario that are connected through shared links or
  // dependencies (union-find over the scenario's flows and links).  Flows of
  // different parts never interact in the fluid model, so every part runs
  // with its own clock; the finish times are those of one clock per scenario
  // up to rounding.  options.single_clock keeps each scenario whole.
  std::vector<int32_t> part_of_id((size_t)F, 0);
  std::vector<int32_t> part_scen;
  std::vector<int32_t> loc((size_t)F, 0);  // id -> index inside its scenario
  for (int32_t s = 0; s < S; ++s) {
    const std::vector<int64_t>& fl = h->scen[s].flows;
    for (size_t i = 0; i < fl.size(); ++i) loc[(size_t)fl[i]] = (int32_t)i;
  }
  for (int32_t s = 0; s < S; ++s) {
    const Scen& sc = h->scen[s];
    const int64_t nf = (int64_t)sc.flows.size();
    if (nf == 0) continue;
    const int32_t P0 = (int32_t)part_scen.size();
    if (h->opt.single_clock || h->opt.exact) {
      for (int64_t id : sc.flows) part_of_id[(size_t)id] = P0;
      part_scen.push_back(s);
      continue;
    }
    const int64_t nl = (int64_t)sc.cap.size();
    UnionFind uf((size_t)(nf + nl));
    for (int64_t i = 0; i < nf; ++i) {
      const int64_t id = sc.flows[(size_t)i];
      for (int64_t e = h->p_off[(size_t)id]; e < h->p_off[(size_t)id + 1]; ++e)
        uf.unite((int32_t)i, (int32_t)(nf + h->p_link[(size_t)e]));
      for (int64_t k = h->d_off[(size_t)id]; k < h->d_off[(size_t)id + 1]; ++k)
        uf.unite((int32_t)i, loc[(size_t)h->d_ids[(size_t)k]]);
    }
    std::vector<int32_t> label((size_t)(nf + nl), -1), grp((size_t)nf);
    int32_t T = 0;
    for (int64_t i = 0; i < nf; ++i) {
      const int32_t r = uf.find((int32_t)i);
      if (label[(size_t)r] < 0) label[(size_t)r] = T++;
      grp[(size_t)i] = label[(size_t)r];
    }
    const int32_t np = std::min(T, kMaxPartsPerScen);
    for (int64_t i = 0; i < nf; ++i)
      part_of_id[(size_t)sc.flows[(size_t)i]] =
          P0 + (int32_t)((int64_t)grp[(size_t)i] * np / T);
    for (int32_t k = 0; k < np; ++k) part_scen.push_back(s);
  }
  const int32_t NP = (int32_t)part_scen.size();
  h->num_parts = NP;
  // device flow order: grouped by part, id order inside
  std::vector<ScenCtl> ctl((size_t)NP);
  std::vector<int64_t> pf((size_t)NP + 1, 0);
  for (int64_t id = 0; id < F; ++id) pf[(size_t)part_of_id[(size_t)id] + 1] += 1;
  for (int32_t k = 0; k < NP; ++k) pf[(size_t)k + 1] += pf[(size_t)k];
  h->dev_of_flow.assign((size_t)F, -1);
  std::vector<int32_t> flow_of_dev((size_t)F);
  {
    std::vector<int64_t> fill(pf.begin(), pf.end() - 1);
    for (int64_t id = 0; id < F; ++id) {
      const int64_t d = fill[(size_t)part_of_id[(size_t)id]]++;
      h->dev_of_flow[(size_t)id] = (int32_t)d;
      flow_of_dev[(size_t)d] = (int32_t)id;
    }
  }
  for (int32_t k = 0; k < NP; ++k) {
    ScenCtl c{};
    c.f0 = (int32_t)pf[(size_t)k];
    c.f1 = (int32_t)pf[(size_t)k + 1];
    c.scen = part_scen[(size_t)k];
    ctl[(size_t)k] = c;
  }
  // used links, compacted and grouped by part (a link belongs to the part of
  // every flow that crosses it), scenario-local id order inside a part
  h->dev_link.assign((size_t)S, {});
  std::vector<int64_t> pl((size_t)NP + 1, 0);
  std::vector<std::vector<int32_t>> part_of_link((size_t)S);
  for (int32_t s = 0; s < S; ++s) {
    const Scen& sc = h->scen[s];
    std::vector<int32_t>& m = part_of_link[(size_t)s];
    m.assign(sc.cap.size(), -1);
    for (int64_t id : sc.flows)
      for (int64_t e = h->p_off[(size_t)id]; e < h->p_off[(size_t)id + 1]; ++e)
        m[(size_t)h->p_link[(size_t)e]] = part_of_id[(size_t)id];
    for (int32_t k : m)
      if (k >= 0) pl[(size_t)k + 1] += 1;
  }
  for (int32_t k = 0; k < NP; ++k) pl[(size_t)k + 1] += pl[(size_t)k];
  const int64_t ld = pl[(size_t)NP];
  if (ld > std::numeric_limits<int32_t>::max()) return fail(h, NETSIM_E_LIMIT, "run: more than 2^31-1 used links");
  double maxcap = 0.0;
  {
    std::vector<int64_t> fill(pl.begin(), pl.end() - 1);
    for (int32_t s = 0; s < S; ++s) {
      const Scen& sc = h->scen[s];
      std::vector<int32_t>& m = h->dev_link[(size_t)s];
      m.assign(sc.cap.size(), -1);
      const std::vector<int32_t>& pk = part_of_link[(size_t)s];
      for (size_t l = 0; l < m.size(); ++l)
        if (pk[l] >= 0) {
          m[l] = (int32_t)fill[(size_t)pk[l]]++;
          maxcap = std::max(maxcap, sc.cap[l]);
        }
    }
  }
  for (int32_t k = 0; k < NP; ++k) {
    ctl[(size_t)k].l0 = (int32_t)pl[(size_t)k];
    ctl[(size_t)k].l1 = (int32_t)pl[(size_t)k + 1];
  }
  h->L = ld;
  h->nnz = (int64_t)h->p_link.size();
  // fixed-point scale: largest capacity below 2^61 units
  int ex = 0;
  if (maxcap > 0.0) std::frexp(maxcap, &ex);
  h->scale = std::ldexp(1.0, 61 - ex);
  std::vector<int64_t> R0((size_t)std::max<int64_t>(ld, 1));
  std::vector<double> capf((size_t)std::max<int64_t>(ld, 1), 0.0);
  for (int32_t s = 0; s < S; ++s) {
    const Scen& sc = h->scen[s];
    for (size_t l = 0; l < sc.cap.size(); ++l) {
      const int32_t d = h->dev_link[(size_t)s][l];
      if (d >= 0) {
        R0[(size_t)d] = (int64_t)std::llrint(sc.cap[l] * h->scale);
        capf[(size_t)d] = sc.cap[l];
      }
    }
  }
  // paths, bytes, start in device order
  std::vector<int32_t> poff((size_t)F + 1);
  std::vector<int32_t> plink((size_t)std::max<int64_t>(h->nnz, 1));
  std::vector<double> nbytes((size_t)std::max<int64_t>(F, 1)), start((size_t)std::max<int64_t>(F, 1));
  std::vector<int32_t> ndeps((size_t)std::max<int64_t>(F, 1), 0);
  // path latency per flow: the sum of its links' latencies in path order
  std::vector<double> lat((size_t)std::max<int64_t>(F, 1), 0.0);
  bool any_lat = false;
  int64_t e = 0;
  for (int64_t d = 0; d < F; ++d) {
    const int64_t id = flow_of_dev[(size_t)d];
    const int32_t s = h->f_scen[(size_t)id];
    const std::vector<double>& llat = h->scen[(size_t)s].lat;
    poff[(size_t)d] = (int32_t)e;
    double acc = 0.0;
    for (int64_t k = h->p_off[(size_t)id]; k < h->p_off[(size_t)id + 1]; ++k) {
      const int32_t l = h->p_link[(size_t)k];
      plink[(size_t)e++] = h->dev_link[(size_t)s][(size_t)l];
      if (!llat.empty()) acc = acc + llat[(size_t)l];
    }
    lat[(size_t)d] = acc;
    any_lat = any_lat || acc != 0.0;
    nbytes[(size_t)d] = h->f_bytes[(size_t)id];
    start[(size_t)d] = h->f_start[(size_t)id];
    ndeps[(size_t)d] = (int32_t)(h->d_off[(size_t)id + 1] - h->d_off[(size_t)id]);
  }
  poff[(size_t)F] = (int32_t)e;
  // 16-byte path records (six 16-bit part-local link ids, 0xFFFF = none) for
  // parts whose paths have at most 6 links and whose link ids fit 16 bits
  std::vector<uint16_t> path16((size_t)std::max<int64_t>(F, 1) * 8, 0xFFFF);
  for (int32_t k = 0; k < NP; ++k) {
    ScenCtl& c = ctl[(size_t)k];
    int32_t deg = 0;
    for (int32_t d = c.f0; d < c.f1; ++d) deg = std::max(deg, poff[(size_t)d + 1] - poff[(size_t)d]);
    c.lds_paths = (deg <= 6 && c.l1 - c.l0 < 0xFFFF) ? 1 : 0;
    if (!c.lds_paths) continue;
    for (int32_t d = c.f0; d < c.f1; ++d)
      for (int32_t j = poff[(size_t)d]; j < poff[(size_t)d + 1]; ++j)
        path16[(size_t)d * 8 + (size_t)(j - poff[(size_t)d])] = (uint16_t)(plink[(size_t)j] - c.l0);
  }
  // link components per part (union-find over links only): flows of
  // different components never share a link, so a change in one cannot move
  // a rate in another
  std::vector<int32_t> comp_of_dev((size_t)std::max<int64_t>(F, 1), 0);
  int32_t ncomp_total = 0;
  {
    UnionFind uf((size_t)std::max<int64_t>(ld, 1));
    for (int64_t d = 0; d < F; ++d)
      for (int32_t k = poff[(size_t)d] + 1; k < poff[(size_t)d + 1]; ++k)
        uf.unite(plink[(size_t)poff[(size_t)d]], plink[(size_t)k]);
    std::vector<int32_t> label((size_t)std::max<int64_t>(ld, 1), -1);
    for (int32_t p = 0; p < NP; ++p) {
      ScenCtl& cs = ctl[(size_t)p];
      int32_t n = 0;
      for (int32_t d = cs.f0; d < cs.f1; ++d) {
        int32_t k = 0;
        if (poff[(size_t)d + 1] > poff[(size_t)d]) {
          const int32_t r = uf.find(plink[(size_t)poff[(size_t)d]]);
          if (label[(size_t)r] < 0) label[(size_t)r] = n < kMaxComp ? n++ : kMaxComp - 1;
          k = label[(size_t)r];
        }
        comp_of_dev[(size_t)d] = ncomp_total + k;
      }
      cs.c0 = ncomp_total;
      cs.nc = std::max<int32_t>(n, 1);
      ncomp_total += cs.nc;
    }
  }
  // successor lists (device ids)
  std::vector<int32_t> soff((size_t)F + 1, 0);
  for (int64_t id = 0; id < F; ++id)
    for (int64_t k = h->d_off[(size_t)id]; k < h->d_off[(size_t)id + 1]; ++k)
      soff[(size_t)h->dev_of_flow[(size_t)h->d_ids[(size_t)k]] + 1] += 1;
  for (int64_t d = 0; d < F; ++d) soff[(size_t)d + 1] += soff[(size_t)d];
  h->nsucc = soff[(size_t)F];
  std::vector<int32_t> succ((size_t)std::max<int64_t>(h->nsucc, 1));
  {
    std::vector<int32_t> fill(soff.begin(), soff.end() - 1);
    for (int64_t id = 0; id < F; ++id)
      for (int64_t k = h->d_off[(size_t)id]; k < h->d_off[(size_t)id + 1]; ++k) {
        const int32_t pred = h->dev_of_flow[(size_t)h->d_ids[(size_t)k]];
        succ[(size_t)fill[(size_t)pred]++] = h->dev_of_flow[(size_t)id];
      }
  }
  // link-major incidence (exact mode's wide solves): flows of each device
  // link in ascending device order, and each entry's link
  const bool exact = h->opt.exact != 0;
  std::vector<int32_t> lfoff, lfid, lfchunk;
  std::vector<uint64_t> lfhead;
  if (exact) {
    lfoff.assign((size_t)ld + 1, 0);
    for (int64_t k = 0; k < h->nnz; ++k) lfoff[(size_t)plink[(size_t)k] + 1] += 1;
    for (int64_t l = 0; l < ld; ++l) lfoff[(size_t)l + 1] += lfoff[(size_t)l];
    lfid.assign((size_t)std::max<int64_t>(h->nnz, 1), 0);
    std::vector<int32_t> fill(lfoff.begin(), lfoff.end() - 1);
    for (int64_t d = 0; d < F; ++d)
      for (int32_t k = poff[(size_t)d]; k < poff[(size_t)d + 1]; ++k) {
        const int32_t l = plink[(size_t)k];
        lfid[(size_t)fill[(size_t)l]++] = (int32_t)d;
      }
    // the link of every 256th entry: the last link whose entries start at or
    // before it (links without entries skipped)
    lfchunk.assign((size_t)(h->nnz / 256 + 1), 0);
    int32_t l = 0;
    for (size_t c = 0; c < lfchunk.size(); ++c) {
      const int64_t e = (int64_t)c * 256;
      while (l + 1 < ld && lfoff[(size_t)l + 1] <= e) ++l;
      lfchunk[c] = l;
    }
    // one bit per entry: set where a link's entries start, and past the end
    lfhead.assign((size_t)((h->nnz + 256) / 64 + 1), ~0ull);
    for (int64_t e = 0; e < h->nnz; ++e) lfhead[(size_t)(e >> 6)] &= ~(1ull << (e & 63));
    for (int64_t k = 0; k < ld; ++k) {
      const int64_t e = lfoff[(size_t)k];
      if (e < h->nnz) lfhead[(size_t)(e >> 6)] |= 1ull << (e & 63);
    }
  }
  h->h_lfoff = lfoff;
  // initial dynamic state
  h->h_cnt0 = ndeps;
  h->h_rel0.assign((size_t)std::max<int64_t>(F, 1), 0.0);
  h->h_pend0.assign((size_t)std::max<int64_t>(F, 1), 0);
  for (int32_t k = 0; k < NP; ++k) {
    ScenCtl& c = ctl[(size_t)k];
    int32_t np = 0;
    for (int32_t d = c.f0; d < c.f1; ++d)
      if (ndeps[(size_t)d] == 0) {
        h->h_pend0[(size_t)(c.f0 + np)] = d;
        h->h_rel0[(size_t)d] = start[(size_t)d];
        ++np;
      }
    c.n_pend0 = np;
  }
  // rollback history: 1/16 of it for event records, the rest for undo
  // records, shared among the parts in proportion to their flows
  size_t hist_bytes = 0;
  if (h->opt.history_mb > 0 && !exact && F > 0) {
    const size_t total = (size_t)h->opt.history_mb << 20;
    const int64_t ev_total = (int64_t)(total / 16 / sizeof(netsim_dev::HistEv));
    const int64_t un_total = (int64_t)((total - (size_t)ev_total * sizeof(netsim_dev::HistEv)) /
                                       sizeof(netsim_dev::HistUndo));
    int64_t hb = 0, eb = 0;
    for (int32_t k = 0; k < NP; ++k) {
      ScenCtl& c = ctl[(size_t)k];
      const double share = (double)(c.f1 - c.f0) / (double)F;
      c.hbase = hb;
      // undo offsets within a part are 32-bit (history.hip)
      c.hcap = std::min<int64_t>(std::max<int64_t>(1, (int64_t)((double)un_total * share)),
                                 std::numeric_limits<int32_t>::max());
      c.ebase = eb;
      c.ecap = std::max<int64_t>(1, (int64_t)((double)ev_total * share));
      hb += c.hcap;
      eb += c.ecap;
    }
    hist_bytes = (size_t)hb * sizeof(netsim_dev::HistUndo) + (size_t)eb * sizeof(netsim_dev::HistEv);
  }
  h->h_ctl0 = ctl;
  // one device allocation, carved into aligned arrays
  const size_t Fz = (size_t)std::max<int64_t>(F, 1), Lz = (size_t)std::max<int64_t>(ld, 1);
  const size_t XL = h->opt.exact ? Lz : 1;
  struct Part { void** dst; size_t bytes; };
  Params& P = h->prm;
  P = Params{};
  std::vector<Part> parts = {
      {(void**)&P.poff, sizeof(int32_t) * (Fz + 1)},
      {(void**)&P.plink, sizeof(int32_t) * plink.size()},
      {(void**)&P.nbytes, sizeof(double) * Fz},
      {(void**)&P.start, sizeof(double) * Fz},
      {(void**)&P.soff, sizeof(int32_t) * (Fz + 1)},
      {(void**)&P.succ, sizeof(int32_t) * succ.size()},
      {(void**)&P.R0, sizeof(int64_t) * Lz},
      // persistent dynamic state (contiguous: one copy makes a checkpoint)
      {(void**)&P.rem, sizeof(double) * Fz},
      {(void**)&P.tref, sizeof(double) * Fz},
      {(void**)&P.rate, sizeof(double) * Fz},
      {(void**)&P.finish, sizeof(double) * Fz},
      {(void**)&P.rel, sizeof(double) * Fz},
      {(void**)&P.base, sizeof(double) * Fz},
      {(void**)&P.cnt, sizeof(int32_t) * Fz},
      {(void**)&P.evr, sizeof(int32_t) * Fz},
      {(void**)&P.eva, sizeof(int32_t) * Fz},
      {(void**)&P.evd, sizeof(int32_t) * Fz},
      {(void**)&P.act0, sizeof(int32_t) * Fz},
      {(void**)&P.act1, sizeof(int32_t) * Fz},
      {(void**)&P.tau0, sizeof(double) * Fz},
      {(void**)&P.tau1, sizeof(double) * Fz},
      {(void**)&P.srate0, sizeof(double) * Fz},
      {(void**)&P.srate1, sizeof(double) * Fz},
      {(void**)&P.pend0, sizeof(int32_t) * Fz},
      {(void**)&P.pend1, sizeof(int32_t) * Fz},
      {(void**)&P.ctl, sizeof(ScenCtl) * (size_t)std::max<int32_t>(NP, 1)},
      // scratch
      {(void**)&P.mf, sizeof(double) * Fz},
      {(void**)&P.arrslot, sizeof(int32_t) * Fz},
      {(void**)&P.comp, sizeof(int32_t) * Fz},
      {(void**)&P.theta, sizeof(uint64_t) * (size_t)std::max<int32_t>(ncomp_total, 1)},
      {(void**)&P.arr, sizeof(int32_t) * Fz},
      {(void**)&P.lst, sizeof(int64_t) * 2 * Lz},
      {(void**)&P.nact, sizeof(int32_t) * Lz},
      {(void**)&P.fl, sizeof(uint32_t) * Lz},
      {(void**)&P.path16, 16 * Fz},
      {(void**)&P.stage, 16 * Fz},
      {(void**)&P.lat, sizeof(double) * Fz},
      {(void**)&P.comp0, sizeof(int32_t) * Fz},
      {(void**)&P.comp1, sizeof(int32_t) * Fz},
      {(void**)&P.comp2, sizeof(int32_t) * Fz},
      {(void**)&P.unf0, sizeof(int32_t) * Fz},
      {(void**)&P.unf1, sizeof(int32_t) * Fz},
      {(void**)&P.bar, sizeof(uint32_t) * netsim_dev::BAR_WORDS},
      {(void**)&P.slots, sizeof(uint64_t) * 8},
      // exact mode: link state in fp64 (one element each otherwise)
      {(void**)&P.capf, sizeof(double) * XL},
      {(void**)&P.xR, sizeof(double) * XL},
      {(void**)&P.xs, sizeof(double) * XL},
      {(void**)&P.xn, sizeof(int32_t) * XL},
      {(void**)&P.xk, sizeof(int32_t) * XL},
      {(void**)&P.xlive0, sizeof(int32_t) * XL},
      {(void**)&P.xlive1, sizeof(int32_t) * XL},
      {(void**)&P.lfoff, sizeof(int32_t) * (XL + 1)},
      {(void**)&P.lfid, sizeof(int32_t) * (exact ? lfid.size() : 1)},
      {(void**)&P.lfchunk, sizeof(int32_t) * (exact ? lfchunk.size() : 1)},
      {(void**)&P.lfhead, sizeof(uint64_t) * (exact ? lfhead.size() : 1)},
      {(void**)&P.xmask, sizeof(uint32_t) * (exact ? Fz / 32 + 8 : 1)},  // +8: 16-byte reads past the end
      {(void**)&P.xfz, XL},
      {(void**)&P.xgrid, sizeof(netsim_dev::XGrid)},
  };
  size_t total = 0;
  for (auto& p : parts) total += (p.bytes + 255) & ~size_t(255);
  hipError_t he = hipSetDevice(h->opt.device);
  if (he != hipSuccess) return hip_fail(h, he, "hipSetDevice");
  he = hipMalloc(&h->d_block, total);
  if (he != hipSuccess) {
    h->d_block = nullptr;
    return fail(h, NETSIM_E_NOMEM, "hipMalloc of " + std::to_string(total) + " bytes failed");
  }
  char* base = (char*)h->d_block;
  for (auto& p : parts) {
    *p.dst = base;
    base += (p.bytes + 255) & ~size_t(255);
  }
  h->persist = (char*)P.rem;
  h->persist_bytes = (size_t)((char*)P.ctl - (char*)P.rem) + sizeof(ScenCtl) * (size_t)std::max<int32_t>(NP, 1);
  if (hist_bytes > 0) {
    he = hipMalloc(&h->d_hist, hist_bytes);
    if (he != hipSuccess) {
      (void)hipGetLastError();
      h->d_hist = nullptr;
      return fail(h, NETSIM_E_NOMEM, "hipMalloc of " + std::to_string(hist_bytes) +
                                         " bytes for the rollback history failed");
    }
    int64_t hb = 0;
    for (const ScenCtl& c : h->h_ctl0) hb += c.hcap;
    P.hist = (netsim_dev::HistUndo*)h->d_hist;
    P.hev = (netsim_dev::HistEv*)((char*)h->d_hist + (size_t)hb * sizeof(netsim_dev::HistUndo));
  }
  struct Up { const void* src; const void* dst; size_t bytes; };
  const Up ups[] = {
      {poff.data(), P.poff, sizeof(int32_t) * (size_t)(F + 1)},
      {plink.data(), P.plink, sizeof(int32_t) * plink.size()},
      {nbytes.data(), P.nbytes, sizeof(double) * nbytes.size()},
      {start.data(), P.start, sizeof(double) * start.size()},
      {soff.data(), P.soff, sizeof(int32_t) * (size_t)(F + 1)},
      {succ.data(), P.succ, sizeof(int32_t) * succ.size()},
      {R0.data(), P.R0, sizeof(int64_t) * R0.size()},
      {comp_of_dev.data(), P.comp, sizeof(int32_t) * comp_of_dev.size()},
      {path16.data(), P.path16, sizeof(uint16_t) * path16.size()},
      {lat.data(), P.lat, any_lat ? sizeof(double) * lat.size() : 0},
      {capf.data(), P.capf, h->opt.exact ? sizeof(double) * capf.size() : 0},
      {lfoff.data(), P.lfoff, sizeof(int32_t) * lfoff.size()},
      {lfid.data(), P.lfid, sizeof(int32_t) * lfid.size()},
      {lfchunk.data(), P.lfchunk, sizeof(int32_t) * lfchunk.size()},
      {lfhead.data(), P.lfhead, sizeof(uint64_t) * lfhead.size()},
  };
  for (const Up& u : ups) {
    if (u.bytes == 0) continue;
    he = hipMemcpy((void*)u.dst, u.src, u.bytes, hipMemcpyHostToDevice);
    if (he != hipSuccess) return hip_fail(h, he, "hipMemcpy (upload)");
  }
  if (!any_lat) P.lat = nullptr;  // no latency anywhere: arrival = last byte
  P.num_scen = NP;
  P.scale = h->scale;
  P.inv_scale = 1.0 / h->scale;
  h->prepared = true;
  return NETSIM_OK;
}

// Resets the dynamic state for a run from t = 0 (on `stream`).
netsim_status reset_state(netsim_t* h, hipStream_t st) {
  Params& P = h->prm;
  const size_t Fz = (size_t)std::max<int64_t>(h->F, 1), Lz = (size_t)std::max<int64_t>(h->L, 1);
  hipError_t he;
  std::vector<double> nan((size_t)Fz, std::numeric_limits<double>::quiet_NaN());
  const uint64_t inf_bits = 0x7FF0000000000000ull;
  uint64_t slots[8];
  for (auto& x : slots) x = inf_bits;
  struct Up { const void* src; void* dst; size_t bytes; };
  const Up ups[] = {
      {h->h_cnt0.data(), P.cnt, sizeof(int32_t) * Fz},
      {h->h_rel0.data(), P.rel, sizeof(double) * Fz},
      {h->h_pend0.data(), P.pend0, sizeof(int32_t) * Fz},
      {nan.data(), P.finish, sizeof(double) * Fz},
      {h->h_ctl0.data(), P.ctl, sizeof(ScenCtl) * h->h_ctl0.size()},
      {slots, P.slots, sizeof(slots)},
  };
  for (const Up& u : ups) {
    if (u.bytes == 0) continue;
    he = hipMemcpyAsync(u.dst, u.src, u.bytes, hipMemcpyHostToDevice, st);
    if (he != hipSuccess) return hip_fail(h, he, "hipMemcpyAsync (reset)");
  }
  h->hist_ok = P.hist != nullptr;
  he = hipMemsetAsync(P.nact, 0, sizeof(int32_t) * Lz, st);
  // per-flow event indices: EV_NEVER, every byte 0x7F
  for (int32_t* a : {P.evr, P.eva, P.evd})
    if (he == hipSuccess) he = hipMemsetAsync(a, 0x7F, sizeof(int32_t) * Fz, st);
  if (he == hipSuccess) he = hipMemsetAsync(P.base, 0, sizeof(double) * Fz, st);
  if (he == hipSuccess) he = hipMemsetAsync(P.rate, 0, sizeof(double) * Fz, st);
  if (he == hipSuccess) he = hipMemsetAsync(P.bar, 0, sizeof(uint32_t) * netsim_dev::BAR_WORDS, st);
  if (he != hipSuccess) return hip_fail(h, he, "hipMemsetAsync (reset)");
  he = hipStreamSynchronize(st);
  if (he != hipSuccess) return hip_fail(h, he, "hipStreamSynchronize (reset)");
  return NETSIM_OK;
}

// One kernel launch: a rate solve per part (solve_only), or the event loop of
// every part from t = 0 or, with resume, from where the last launch stopped,
// processing events up to `until` and at most max_events more per part.
netsim_status launch(netsim_t* h, hipStream_t st, bool solve_only, float* ms, bool resume = false,
                     int64_t max_events = -1, double until = std::numeric_limits<double>::quiet_NaN()) {
  Params P = h->prm;
  P.mode = solve_only ? 1 : 0;
  P.resume = resume ? 1 : 0;
  if (max_events < 0) max_events = h->opt.max_events;
  if (std::isnan(until)) until = h->opt.until;
  P.max_events = solve_only ? 0 : max_events;
  P.until = std::isnan(until) ? std::numeric_limits<double>::infinity() : until;
  P.debug = h->opt.debug;
  P.max_rounds = h->opt.max_rounds > 0 ? h->opt.max_rounds
                                       : (int32_t)std::min<int64_t>(h->F + 1, std::numeric_limits<int32_t>::max());
  P.assist_min = h->opt.assist_min_flows > 0 ? h->opt.assist_min_flows : kAssistMinFlows;
  P.assist_helpers = h->opt.assist_helpers > 0 ? h->opt.assist_helpers : kAssistHelpers;
  const int32_t S = h->num_parts;
  int exec = h->opt.exec;
  // flows without predecessors in the widest part (a part whose flows chain
  // through dependencies keeps few of them active at once, however many it has)
  int64_t widest = 0;
  for (const ScenCtl& c : h->h_ctl0) {
    int64_t roots = 0;
    for (int32_t d = c.f0; d < c.f1; ++d) roots += h->h_cnt0[(size_t)d] == 0;
    widest = std::max(widest, roots);
  }
  if (exec == NETSIM_EXEC_AUTO) {
    // the whole GPU on one part when its first solve alone exceeds what one
    // workgroup solves in shared memory (more than 64 x 1024 flows); the
    // cluster layout when there are no more parts than XCDs (one leader
    // each) and some part starts wide enough for re-solves the helpers
    // speed up; otherwise one workgroup per part
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, h->opt.device) != hipSuccess)
      cus = 0;
    const int xcds = cus / kCusPerXcd;
    if (S == 1 && widest > 65536) exec = NETSIM_EXEC_GRID;
    // (not with the rollback history, which the cluster kernel does not keep)
    else if (!solve_only && S <= kMaxClustersPerXcd * xcds && widest > 16384 && h->opt.history_mb <= 0)
      exec = NETSIM_EXEC_CLUSTER;
    else exec = NETSIM_EXEC_BLOCK;
  }
  if (exec == NETSIM_EXEC_CLUSTER && solve_only) exec = NETSIM_EXEC_BLOCK;
  if (h->opt.exact) exec = NETSIM_EXEC_EXACT;
  h->layout = exec;
  if (!solve_only && (exec == NETSIM_EXEC_CLUSTER || exec == NETSIM_EXEC_EXACT)) h->hist_ok = false;
  // grid-barrier words and min-reduction slots start fresh in every launch
  // (a launch that continues a run must not see the last launch's counts)
  uint64_t inf_slots[8];
  for (auto& x : inf_slots) x = 0x7FF0000000000000ull;
  hipError_t he = hipMemsetAsync(P.bar, 0, sizeof(uint32_t) * netsim_dev::BAR_WORDS, st);
  if (he == hipSuccess) he = hipMemcpyAsync(P.slots, inf_slots, sizeof(inf_slots), hipMemcpyHostToDevice, st);
  if (he != hipSuccess) return hip_fail(h, he, "reset of the grid synchronisation words");
  hipEvent_t e0, e1;
  he = hipEventCreate(&e0);
  if (he == hipSuccess) he = hipEventCreate(&e1);
  if (he != hipSuccess) return hip_fail(h, he, "hipEventCreate");
  he = hipEventRecord(e0, st);
  if (he == hipSuccess) {
    if (exec == NETSIM_EXEC_EXACT) {
      // link state in shared memory for every part whose links fit the pool
      // (sized by the largest such part, so small parts leave room for more
      // workgroups per CU); larger parts keep theirs in global memory
      const int64_t per = netsim_dev::exact_link_bytes();
      int64_t lds = 0;
      for (const ScenCtl& c : h->h_ctl0) {
        const int64_t b = (int64_t)(c.l1 - c.l0) * per;
        if (b <= kExactLdsBytes) lds = std::max(lds, b);
      }
      P.exact_lds_bytes = (int32_t)((lds + 15) & ~int64_t(15));
      int threads = h->opt.block_threads > 0 ? h->opt.block_threads : kExactThreads;
      threads = std::max(64, std::min(1024, threads / 64 * 64));
      const int blocks = std::max(1, std::min<int32_t>(S, 1 << 20));
      he = netsim_dev::launch_exact(P, blocks, threads, st);
    } else if (exec == NETSIM_EXEC_CLUSTER) {
      int blocks = 0;
      he = netsim_dev::cluster_capacity(h->opt.device, &blocks);
      if (he == hipSuccess && blocks < 1) he = hipErrorInvalidConfiguration;
      // as many leaders as parts (up to kMaxClustersPerXcd per XCD), so that
      // every part runs at once with the helpers that leaves it
      int cus = 0;
      if (he == hipSuccess) he = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, h->opt.device);
      const int xcds = std::max(1, cus / kCusPerXcd);
      P.clusters_per_xcd = std::max(1, std::min(kMaxClustersPerXcd, (S + xcds - 1) / xcds));
      if (he == hipSuccess) he = netsim_dev::launch_cluster(P, blocks, st);
    } else if (exec == NETSIM_EXEC_GRID) {
      const int threads = 1024;
      int cap = 0;
      he = netsim_dev::grid_capacity(h->opt.device, threads, &cap);
      hipDeviceProp_t prop;
      if (he == hipSuccess) he = hipGetDeviceProperties(&prop, h->opt.device);
      if (he == hipSuccess) {
        int blocks = std::min(cap, prop.multiProcessorCount);
        if (blocks < 1) blocks = 1;
        he = netsim_dev::launch_grid(P, blocks, threads, st);
      }
    } else {
      // 1024 threads when some part starts with more than 16384 flows
      // without predecessors (its solves may need more than the 64 x 512
      // items one 512-thread workgroup solves in shared memory); otherwise
      // 512, which spills no registers and has cheaper barriers
      int threads = h->opt.block_threads > 0 ? h->opt.block_threads : widest > 16384 ? 1024 : 512;
      threads = std::max(64, std::min(1024, threads / 64 * 64));
      const int blocks = std::max(1, std::min<int32_t>(S, 1 << 20));
      he = netsim_dev::launch_block(P, blocks, threads, st);
    }
  }
  if (he == hipSuccess) he = hipEventRecord(e1, st);
  if (he == hipSuccess) he = hipEventSynchronize(e1);
  if (he == hipSuccess) he = hipEventElapsedTime(ms, e0, e1);
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  if (he != hipSuccess) return hip_fail(h, he, "kernel launch");
  return NETSIM_OK;
}

netsim_status collect(netsim_t* h, std::vector<ScenCtl>* ctl_out) {
  const int32_t S = h->num_parts;
  std::vector<ScenCtl> ctl((size_t)S);
  hipError_t he = hipMemcpy(ctl.data(), h->prm.ctl, sizeof(ScenCtl) * (size_t)S, hipMemcpyDeviceToHost);
  if (he != hipSuccess) return hip_fail(h, he, "hipMemcpy (control blocks)");
  *ctl_out = ctl;
  for (int32_t s = 0; s < S; ++s) {
    const int32_t st = ctl[(size_t)s].status;
    if (st < 0) {
      if (st == -8)
        return fail(h, NETSIM_E_DEVICE, "debug check failed in scenario " + std::to_string(ctl[(size_t)s].scen) +
                                            ": event " + std::to_string(ctl[(size_t)s].dbg[0] - 1) +
                                            " link " + std::to_string(ctl[(size_t)s].dbg[1]) +
                                            " last solve path " + std::to_string(ctl[(size_t)s].dbg[2]));
      std::string why = st == netsim_dev::ST_ROUNDS ? "round watchdog fired"
                        : st == netsim_dev::ST_BARRIER ? "grid barrier timed out"
                        : st == netsim_dev::ST_OVERFLOW ? "work list fault"
                                                        : "non-positive fair share";
      return fail(h, st == netsim_dev::ST_ROUNDS ? NETSIM_E_LIMIT : NETSIM_E_DEVICE,
                  "device solver fault in scenario " + std::to_string(ctl[(size_t)s].scen) + ": " + why);
    }
  }
  return NETSIM_OK;
}


void drop_checkpoints(netsim_t* h) {
  for (auto& c : h->checkpoints)
    if (c.dev) (void)hipFree(c.dev);
  h->checkpoints.clear();
}

// A fresh run from t = 0 (resume = false) or a continuation of the current
// position (resume = true; from t = 0 if there is none), then the results.
netsim_status simulate(netsim_t* h, hipStream_t st, bool resume, int64_t max_events, double until) {
  const auto t0 = std::chrono::steady_clock::now();
  netsim_status rc;
  if (!h->prepared) {
    rc = prepare(h);
    if (rc) return rc;
  }
  hipError_t he = hipSetDevice(h->opt.device);
  if (he != hipSuccess) return hip_fail(h, he, "hipSetDevice");
  if (!resume || !h->has_state) {
    drop_checkpoints(h);
    rc = reset_state(h, st);
    if (rc) return rc;
  }
  const auto t1 = std::chrono::steady_clock::now();
  float ms = 0.0f;
  if (h->F > 0) {
    rc = launch(h, st, false, &ms, resume, max_events, until);
    if (rc) return rc;
  }
  h->has_state = true;
  std::vector<ScenCtl> ctl;
  rc = h->F > 0 ? collect(h, &ctl) : NETSIM_OK;
  if (h->F == 0) ctl = h->h_ctl0;
  // results, even on a device fault (partial), for inspection
  const int64_t F = h->F;
  std::vector<double> fin_dev((size_t)std::max<int64_t>(F, 1));
  if (F > 0) {
    he = hipMemcpy(fin_dev.data(), h->prm.finish, sizeof(double) * (size_t)F, hipMemcpyDeviceToHost);
    if (he != hipSuccess) return hip_fail(h, he, "hipMemcpy (finish)");
  }
  h->finish.assign((size_t)F, 0.0);
  for (int64_t id = 0; id < F; ++id) h->finish[(size_t)id] = fin_dev[(size_t)h->dev_of_flow[(size_t)id]];
  h->makespan.assign(h->scen.size(), 0.0);
  netsim_stats s{};
  s.complete = 1;
  s.parts = h->num_parts;
  const int32_t NP = h->num_parts;
  h->part_t.assign((size_t)NP, -std::numeric_limits<double>::infinity());
  for (int32_t k = 0; k < NP; ++k)
    if (ctl[(size_t)k].started) h->part_t[(size_t)k] = ctl[(size_t)k].t;
  for (int32_t k = 0; k < NP; ++k) {
    const ScenCtl& c = ctl[(size_t)k];
    double& m = h->makespan[(size_t)c.scen];
    for (int32_t d = c.f0; d < c.f1; ++d)
      if (!std::isnan(fin_dev[(size_t)d])) {
        m = std::max(m, fin_dev[(size_t)d]);
        s.completed_flows += 1;
      }
    s.events += c.events;
    s.solves += c.solves;
    s.rounds += c.rounds;
    s.flows_swept += c.flows_swept;
    s.incidences_swept += c.incidences_swept;
    s.active_swept += c.active_swept;
    s.pending_swept += c.pending_swept;
    s.reselected += c.reselected;
    s.wide_solves += c.wide_solves;
    s.assisted_solves += c.assisted;
    s.links_swept += c.links_swept;
    s.launch_events += c.launch_events;
    s.layout = h->layout;
    s.sim_time = std::max(s.sim_time, c.t);
    if (c.status != 0) s.complete = 0;
  }
  int khz = 0;
  if (hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, h->opt.device) != hipSuccess || khz <= 0)
    khz = 100000;
  for (int32_t k = 0; k < NP; ++k)
    for (int j = 0; j < 8; ++j) s.phase_seconds[j] += (double)ctl[(size_t)k].ticks[j] / (1e3 * khz);
  s.device_seconds = ms * 1e-3;
  s.upload_seconds = std::chrono::duration<double>(t1 - t0).count();
  h->stats = s;
  h->has_result = true;
  return rc;
}


// A wide exact solve of the n flows of part p listed in its act0 slice, on
// the whole GPU (sweep.hip).  Levels are enqueued in batches; the host reads
// the unfrozen count after each batch.  Adds the solve's statistics to *out.
struct GridStats {
  unsigned long long levels = 0, fsw = 0, isw = 0, lsw = 0;
};

netsim_status grid_solve(netsim_t* h, hipStream_t st, int32_t p, int32_t n, GridStats* out) {
  const Params& P = h->prm;
  const ScenCtl& C = h->h_ctl0[(size_t)p];
  hipError_t he = netsim_dev::grid_solve_begin(P, C, n, st);
  if (he == hipSuccess)
    he = netsim_dev::grid_solve_count(P, C, h->h_lfoff[(size_t)C.l0], h->h_lfoff[(size_t)C.l1], st);
  const int64_t limit = h->opt.max_rounds > 0 ? h->opt.max_rounds : (int64_t)n + 1;
  netsim_dev::XGridHead g{};  // the counters the host reads
  // levels 0 and 1 directly; then batches of kGridLevelBatch levels replayed
  // from one captured graph (the kernels use only the parity of the level
  // and whether it is the first, so the batch captured as levels 2, 3, ...
  // serves for every later batch)
  hipGraphExec_t batch = nullptr;
  for (int j = 0; j < 2 && he == hipSuccess; ++j) {
    he = netsim_dev::grid_solve_links(P, C, j, st);
    if (he == hipSuccess) he = netsim_dev::grid_solve_freeze(P, C, n, j, st);
  }
  if (he == hipSuccess) {
    hipStream_t cs = nullptr;
    hipGraph_t graph = nullptr;
    he = hipStreamCreateWithFlags(&cs, hipStreamNonBlocking);
    if (he == hipSuccess) he = hipStreamBeginCapture(cs, hipStreamCaptureModeThreadLocal);
    if (he == hipSuccess) {
      for (int b = 0; b < kGridLevelBatch && he == hipSuccess; ++b) {
        he = netsim_dev::grid_solve_links(P, C, 2 + b, cs);
        if (he == hipSuccess) he = netsim_dev::grid_solve_freeze(P, C, n, 2 + b, cs);
      }
      const hipError_t he2 = hipStreamEndCapture(cs, &graph);
      if (he == hipSuccess) he = he2;
    }
    if (he == hipSuccess) he = hipGraphInstantiate(&batch, graph, nullptr, nullptr, 0);
    if (graph) (void)hipGraphDestroy(graph);
    if (cs) (void)hipStreamDestroy(cs);
  }
  for (int rep = 0; he == hipSuccess; ++rep) {
    if (rep > 0) he = hipGraphLaunch(batch, st);
    if (he == hipSuccess) he = hipMemcpyAsync(&g, P.xgrid, sizeof g, hipMemcpyDeviceToHost, st);
    if (he == hipSuccess) he = hipStreamSynchronize(st);
    if (he != hipSuccess) break;
    if (g.fault) {
      (void)hipGraphExecDestroy(batch);
      return fail(h, NETSIM_E_DEVICE, "device solver fault: non-positive fair share");
    }
    if (g.done) break;
    if ((int64_t)g.levels > limit) {
      (void)hipGraphExecDestroy(batch);
      return fail(h, NETSIM_E_LIMIT, "device solver fault: round watchdog fired");
    }
  }
  if (batch) (void)hipGraphExecDestroy(batch);
  if (he != hipSuccess) return hip_fail(h, he, "wide exact solve");
  // per-workgroup statistics
  std::vector<unsigned long long> isw((size_t)g.ublocks), lsw((size_t)g.lblocks);
  const netsim_dev::XGrid* dg = P.xgrid;
  he = hipMemcpy(isw.data(), dg->isw, sizeof(unsigned long long) * isw.size(), hipMemcpyDeviceToHost);
  if (he == hipSuccess)
    he = hipMemcpy(lsw.data(), dg->lsw, sizeof(unsigned long long) * lsw.size(), hipMemcpyDeviceToHost);
  if (he != hipSuccess) return hip_fail(h, he, "wide exact solve statistics");
  out->levels += g.levels;
  out->fsw += g.fsw;
  for (unsigned long long v : isw) out->isw += v;
  for (unsigned long long v : lsw) out->lsw += v;
  return NETSIM_OK;
}

// Part of device flow d (parts hold consecutive device flows).
int32_t part_of_dev(const netsim_t* h, int32_t d) {
  int32_t lo = 0, hi = h->num_parts - 1;
  while (lo < hi) {
    const int32_t mid = (lo + hi) / 2;
    if (h->h_ctl0[(size_t)mid].f1 <= d) lo = mid + 1; else hi = mid;
  }
  return lo;
}

// Keeps a copy of the persistent state (best effort: without device memory
// for it, later rollbacks go back to an older checkpoint or to t = 0).
netsim_status push_checkpoint(netsim_t* h, hipStream_t st) {
  netsim_t::Checkpoint c;
  if (hipMalloc(&c.dev, h->persist_bytes) != hipSuccess) {
    (void)hipGetLastError();
    return NETSIM_OK;
  }
  hipError_t he = hipMemcpyAsync(c.dev, h->persist, h->persist_bytes, hipMemcpyDeviceToDevice, st);
  if (he == hipSuccess) he = hipStreamSynchronize(st);
  if (he != hipSuccess) {
    (void)hipFree(c.dev);
    return hip_fail(h, he, "checkpoint copy");
  }
  c.t = h->part_t;
  c.valid.assign((size_t)h->num_parts, 1);
  h->checkpoints.push_back(std::move(c));
  return NETSIM_OK;
}

// Restores part p to checkpoint k (k < 0: its state at t = 0) and marks the
// later checkpoints as off its history.
netsim_status restore_part(netsim_t* h, int32_t p, int k) {
  const Params& P = h->prm;
  const ScenCtl& c0 = h->h_ctl0[(size_t)p];
  const size_t f0 = (size_t)c0.f0, n = (size_t)(c0.f1 - c0.f0);
  hipError_t he = hipSuccess;
  if (k >= 0) {
    const char* src = (const char*)h->checkpoints[(size_t)k].dev;
    struct A { void* a; size_t z; };
    const A arrays[] = {{P.rem, 8}, {P.tref, 8}, {P.rate, 8}, {P.finish, 8}, {P.rel, 8}, {P.base, 8},
                        {P.cnt, 4}, {P.evr, 4}, {P.eva, 4}, {P.evd, 4},
                        {P.act0, 4}, {P.act1, 4}, {P.tau0, 8}, {P.tau1, 8},
                        {P.srate0, 8}, {P.srate1, 8}, {P.pend0, 4}, {P.pend1, 4}};
    for (const A& a : arrays) {
      const size_t off = (size_t)((char*)a.a - h->persist) + f0 * a.z;
      if (he == hipSuccess && n > 0) he = hipMemcpy((char*)a.a + f0 * a.z, src + off, n * a.z, hipMemcpyDeviceToDevice);
    }
    const size_t coff = (size_t)((char*)P.ctl - h->persist) + sizeof(ScenCtl) * (size_t)p;
    if (he == hipSuccess) he = hipMemcpy(P.ctl + p, src + coff, sizeof(ScenCtl), hipMemcpyDeviceToDevice);
  } else {
    std::vector<double> nan(n, std::numeric_limits<double>::quiet_NaN()), zero(n, 0.0);
    if (n > 0) {
      he = hipMemcpy(P.cnt + f0, h->h_cnt0.data() + f0, 4 * n, hipMemcpyHostToDevice);
      if (he == hipSuccess) he = hipMemcpy(P.rel + f0, h->h_rel0.data() + f0, 8 * n, hipMemcpyHostToDevice);
      if (he == hipSuccess) he = hipMemcpy(P.pend0 + f0, h->h_pend0.data() + f0, 4 * n, hipMemcpyHostToDevice);
      if (he == hipSuccess) he = hipMemcpy(P.finish + f0, nan.data(), 8 * n, hipMemcpyHostToDevice);
      if (he == hipSuccess) he = hipMemcpy(P.base + f0, zero.data(), 8 * n, hipMemcpyHostToDevice);
      if (he == hipSuccess) he = hipMemcpy(P.rate + f0, zero.data(), 8 * n, hipMemcpyHostToDevice);
      for (int32_t* a : {P.evr, P.eva, P.evd})
        if (he == hipSuccess) he = hipMemset(a + f0, 0x7F, 4 * n);
    }
    if (he == hipSuccess) he = hipMemcpy(P.ctl + p, &c0, sizeof(ScenCtl), hipMemcpyHostToDevice);
  }
  if (he != hipSuccess) return hip_fail(h, he, "rollback copy");
  for (size_t j = (size_t)std::max(k + 1, 0); j < h->checkpoints.size(); ++j)
    h->checkpoints[j].valid[(size_t)p] = 0;
  h->part_t[(size_t)p] = k >= 0 ? h->checkpoints[(size_t)k].t[(size_t)p]
                                : -std::numeric_limits<double>::infinity();
  return NETSIM_OK;
}

// Part p back to the end of its last event before `before` from the
// rollback history (Section 4.2).  *done = false when the history cannot do
// it (none, or its rings no longer hold every record since): nothing has
// changed then.
netsim_status history_rollback(netsim_t* h, int32_t p, double before, bool* done) {
  *done = false;
  const Params& P = h->prm;
  if (!P.hist || !h->hist_ok) return NETSIM_OK;
  ScenCtl c;
  hipError_t he = hipMemcpy(&c, P.ctl + p, sizeof c, hipMemcpyDeviceToHost);
  if (he != hipSuccess) return hip_fail(h, he, "hipMemcpy (control block)");
  if (c.hcap <= 0 || c.ecap <= 0) return NETSIM_OK;
  const int64_t E = c.started ? (int64_t)c.e : 0;  // events processed so far
  const int64_t lo = std::max<int64_t>(0, E - c.ecap);  // oldest event still recorded
  netsim_dev::HistEv rec{};
  auto read = [&](int64_t e) {
    return hipMemcpy(&rec, P.hev + c.ebase + e % c.ecap, sizeof rec, hipMemcpyDeviceToHost);
  };
  // first recorded event at or after `before` (event times increase)
  int64_t a = lo, b = E;
  while (a < b && he == hipSuccess) {
    const int64_t m = a + (b - a) / 2;
    he = read(m);
    if (rec.t < before) a = m + 1; else b = m;
  }
  if (he != hipSuccess) return hip_fail(h, he, "hipMemcpy (event record)");
  const int64_t es = a - 1;  // the last event before `before`
  if (es < lo) {
    if (lo > 0) return NETSIM_OK;  // older than the ring holds
    netsim_status rc = restore_part(h, p, -1);  // no event before it: t = 0
    if (rc == NETSIM_OK) *done = true;
    return rc;
  }
  he = read(es);
  if (he != hipSuccess) return hip_fail(h, he, "hipMemcpy (event record)");
  if (c.hpos - rec.hpos > c.hcap) return NETSIM_OK;  // undo records overwritten
  const ScenCtl& c0 = h->h_ctl0[(size_t)p];
  const int32_t f0 = c0.f0, f1 = c0.f1;
  const size_t n = (size_t)(f1 - f0);
  if (n > 0) {
    he = hipMemcpy(P.unf0 + f0, h->h_cnt0.data() + f0, 4 * n, hipMemcpyHostToDevice);
    if (he == hipSuccess) he = hipMemcpy(P.mf + f0, h->h_rel0.data() + f0, 8 * n, hipMemcpyHostToDevice);
  }
  if (he == hipSuccess)
    he = netsim_dev::history_restore(P, p, f0, f1, c.hbase, c.hcap, (int32_t)es, rec, c.hpos, P.unf0 + f0,
                                     P.mf + f0, P.arr + f0, P.bar, nullptr);
  if (he == hipSuccess) he = hipStreamSynchronize(nullptr);
  if (he != hipSuccess) return hip_fail(h, he, "rollback from the history");
  for (auto& ck : h->checkpoints)
    if (ck.t[(size_t)p] > rec.t) ck.valid[(size_t)p] = 0;
  h->part_t[(size_t)p] = rec.t;
  *done = true;
  return NETSIM_OK;
}

// Latest checkpoint on part p's history whose last event precedes `before`
// (-1: none, i.e. t = 0).
int latest_checkpoint(const netsim_t* h, int32_t p, double before) {
  for (int k = (int)h->checkpoints.size() - 1; k >= 0; --k) {
    const auto& c = h->checkpoints[(size_t)k];
    if (c.valid[(size_t)p] && c.t[(size_t)p] < before) return k;
  }
  return -1;
}

}  // namespace

extern "C" {

void netsim_default_options(netsim_options* opt) {
  if (!opt) return;
  std::memset(opt, 0, sizeof *opt);
  opt->until = std::numeric_limits<double>::infinity();
}

netsim_status netsim_create(netsim_t** out, int32_t num_scenarios, const int64_t* link_off,
                            const double* capacity_Bps, const netsim_options* opt) {
  if (!out) return fail(nullptr, NETSIM_E_INVALID, "create: out is NULL");
  *out = nullptr;
  if (num_scenarios < 1 || !link_off) return fail(nullptr, NETSIM_E_INVALID, "create: need >= 1 scenario and link_off");
  if (link_off[0] != 0) return fail(nullptr, NETSIM_E_INVALID, "create: link_off[0] must be 0");
  for (int32_t s = 0; s < num_scenarios; ++s)
    if (link_off[s + 1] < link_off[s]) return fail(nullptr, NETSIM_E_INVALID, "create: link_off must not decrease");
  const int64_t L = link_off[num_scenarios];
  if (L > 0 && !capacity_Bps) return fail(nullptr, NETSIM_E_INVALID, "create: capacity_Bps is NULL");
  for (int64_t l = 0; l < L; ++l)
    if (!(std::isfinite(capacity_Bps[l]) && capacity_Bps[l] > 0.0))
      return fail(nullptr, NETSIM_E_INVALID, "create: capacities must be finite and > 0 (link " + std::to_string(l) + ")");
  netsim_t* h = new (std::nothrow) netsim_t();
  if (!h) return fail(nullptr, NETSIM_E_NOMEM, "create: out of memory");
  if (opt) h->opt = *opt;
  else netsim_default_options(&h->opt);
  if (h->opt.history_mb < 0) {
    delete h;
    return fail(nullptr, NETSIM_E_INVALID, "create: history_mb must be >= 0");
  }
  h->scen.resize((size_t)num_scenarios);
  for (int32_t s = 0; s < num_scenarios; ++s)
    h->scen[(size_t)s].cap.assign(capacity_Bps + link_off[s], capacity_Bps + link_off[s + 1]);
  *out = h;
  return NETSIM_OK;
}

netsim_status netsim_create_topology(netsim_t** out, int32_t num_scenarios,
                                     const netsim_topology* topos, const netsim_options* opt) {
  if (!out) return fail(nullptr, NETSIM_E_INVALID, "create_topology: out is NULL");
  *out = nullptr;
  if (num_scenarios < 1 || !topos) return fail(nullptr, NETSIM_E_INVALID, "create_topology: need >= 1 topology");
  netsim_t* h = new (std::nothrow) netsim_t();
  if (!h) return fail(nullptr, NETSIM_E_NOMEM, "create_topology: out of memory");
  if (opt) h->opt = *opt;
  else netsim_default_options(&h->opt);
  if (h->opt.history_mb < 0) {
    delete h;
    return fail(nullptr, NETSIM_E_INVALID, "create: history_mb must be >= 0");
  }
  h->scen.resize((size_t)num_scenarios);
  for (int32_t s = 0; s < num_scenarios; ++s) {
    Scen& sc = h->scen[(size_t)s];
    std::string err;
    if (!sc.fab.init(topos[s], &err)) {
      delete h;
      return fail(nullptr, NETSIM_E_INVALID, "scenario " + std::to_string(s) + ": " + err);
    }
    sc.has_fabric = true;
    sc.fab.capacities(&sc.cap);
    sc.fab.latencies(&sc.lat);
  }
  *out = h;
  return NETSIM_OK;
}

netsim_status netsim_get_links(const netsim_t* h, int32_t scen, int64_t* num_links, double* cap_out) {
  if (!h) return fail(nullptr, NETSIM_E_INVALID, "get_links: handle is NULL");
  if (scen < 0 || scen >= (int32_t)h->scen.size()) return fail(h, NETSIM_E_INVALID, "get_links: bad scenario");
  const auto& c = h->scen[(size_t)scen].cap;
  if (num_links) *num_links = (int64_t)c.size();
  if (cap_out) std::copy(c.begin(), c.end(), cap_out);
  return NETSIM_OK;
}

netsim_status netsim_add_flows(netsim_t* h, int32_t scen, int64_t n, const int32_t* src,
                               const int32_t* dst, const double* nbytes, const double* start,
                               const int64_t* path_off, const int32_t* path_link,
                               const int64_t* dep_off, const int64_t* dep_ids, int64_t* first_id) {
  if (!h) return fail(nullptr, NETSIM_E_INVALID, "add_flows: handle is NULL");
  const int64_t first = (int64_t)h->f_bytes.size();
  const netsim_status st =
      add_flows_impl(h, scen, n, src, dst, nbytes, start, path_off, path_link, dep_off, dep_ids, first_id);
  if (st == NETSIM_OK) set_exits(h, first, first + n);  // every flow of the batch
  return st;
}

netsim_status netsim_add_ring(netsim_t* h, int32_t scen, int32_t kind, int32_t mode, int32_t p,
                              const int32_t* ranks, double nbytes, double lag, int64_t n_after,
                              const int64_t* after, int64_t* first_id, int64_t* count) {
  if (!h) return fail(nullptr, NETSIM_E_INVALID, "add_ring: handle is NULL");
  if (h->prepared) return fail(h, NETSIM_E_STATE, "add_ring: flows cannot be added after a run");
  if (kind < NETSIM_RING_ALLREDUCE || kind > NETSIM_RING_ALL_GATHER) return fail(h, NETSIM_E_INVALID, "add_ring: bad kind");
  if (mode < NETSIM_MODE_CHAINED || mode > NETSIM_MODE_AGGREGATED) return fail(h, NETSIM_E_INVALID, "add_ring: bad mode");
  if (p < 2) return fail(h, NETSIM_E_INVALID, "add_ring: need p >= 2");
  if (!finite_nonneg(nbytes) || !finite_nonneg(lag)) return fail(h, NETSIM_E_INVALID, "add_ring: bytes and lag must be finite and >= 0");
  netsim_status st = check_ranks(h, scen, p, ranks);
  if (st) return st;
  st = check_after(h, scen, n_after, after);
  if (st) return st;
  const int64_t steps = kind == NETSIM_RING_ALLREDUCE ? 2 * (int64_t)(p - 1) : (int64_t)(p - 1);
  const double chunk = nbytes / (double)p;
  const int64_t first = (int64_t)h->f_bytes.size();
  const int64_t n = mode == NETSIM_MODE_AGGREGATED ? p : steps * p;
  std::vector<int32_t> src((size_t)n), dst((size_t)n);
  std::vector<double> b((size_t)n), t0((size_t)n);
  std::vector<int64_t> doff((size_t)n + 1, 0), dids;
  for (int64_t k = 0; k < n / p; ++k)
    for (int32_t i = 0; i < p; ++i) {
      const int64_t f = k * p + i;
      src[(size_t)f] = ranks[i];
      dst[(size_t)f] = ranks[(i + 1) % p];
      b[(size_t)f] = mode == NETSIM_MODE_AGGREGATED ? (double)steps * chunk : chunk;
      const bool entry = mode != NETSIM_MODE_CHAINED || k == 0;
      t0[(size_t)f] = entry ? lag : 0.0;
      if (entry) {
        dids.insert(dids.end(), after, after + n_after);
      } else {
        dids.push_back(first + (k - 1) * p + (i + p - 1) % p);  // the step-(k-1) flow into rank i
      }
      doff[(size_t)f + 1] = (int64_t)dids.size();
    }
  st = add_flows_impl(h, scen, n, src.data(), dst.data(), b.data(), t0.data(), nullptr, nullptr,
                      doff.data(), dids.data(), nullptr);
  if (st) return st;
  // exits: a chained ring's last step, every flow otherwise
  const int64_t e0 = mode == NETSIM_MODE_CHAINED ? first + (steps - 1) * p : first;
  set_exits(h, e0, first + n);
  if (first_id) *first_id = first;
  if (count) *count = n;
  return NETSIM_OK;
}

netsim_status netsim_add_all_to_all(netsim_t* h, int32_t scen, int32_t p, const int32_t* ranks,
                                    const double* nbytes, double lag, int64_t n_after,
                                    const int64_t* after, int64_t* first_id, int64_t* count) {
  if (!h) return fail(nullptr, NETSIM_E_INVALID, "add_all_to_all: handle is NULL");
  if (h->prepared) return fail(h, NETSIM_E_STATE, "add_all_to_all: flows cannot be added after a run");
  if (p < 1) return fail(h, NETSIM_E_INVALID, "add_all_to_all: need p >= 1");
  if (!nbytes) return fail(h, NETSIM_E_INVALID, "add_all_to_all: nbytes is NULL");
  if (!finite_nonneg(lag)) return fail(h, NETSIM_E_INVALID, "add_all_to_all: lag must be finite and >= 0");
  netsim_status st = check_ranks(h, scen, p, ranks);
  if (st) return st;
  st = check_after(h, scen, n_after, after);
  if (st) return st;
  const int64_t first = (int64_t)h->f_bytes.size();
  const int64_t n = (int64_t)p * (p - 1);
  std::vector<int32_t> src, dst;
  std::vector<double> b, t0;
  std::vector<int64_t> doff(1, 0), dids;
  src.reserve((size_t)n);
  for (int32_t i = 0; i < p; ++i)
    for (int32_t j = 0; j < p; ++j) {
      if (i == j) continue;
      src.push_back(ranks[i]);
      dst.push_back(ranks[j]);
      b.push_back(nbytes[(size_t)i * p + j]);
      t0.push_back(lag);
      dids.insert(dids.end(), after, after + n_after);
      doff.push_back((int64_t)dids.size());
    }
  st = add_flows_impl(h, scen, n, src.data(), dst.data(), b.data(), t0.data(), nullptr, nullptr,
                      doff.data(), dids.data(), nullptr);
  if (st) return st;
  set_exits(h, first, first + n);  // every flow
  if (first_id) *first_id = first;
  if (count) *count = n;
  return NETSIM_OK;
}


netsim_status netsim_set_link_latency(netsim_t* h, int32_t scen, int64_t num_links,
                                      const double* latency_s) {
  if (!h) return fail(nullptr, NETSIM_E_INVALID, "set_link_latency: handle is NULL");
  if (h->prepared) return fail(h, NETSIM_E_STATE, "set_link_latency: latencies cannot change after a run");
  if (scen < 0 || scen >= (int32_t)h->scen.size()) return fail(h, NETSIM_E_INVALID, "set_link_latency: bad scenario");
  Scen& sc = h->scen[(size_t)scen];
  if (num_links != (int64_t)sc.cap.size()) return fail(h, NETSIM_E_INVALID, "set_link_latency: need one value per link");
  if (num_links > 0 && !latency_s) return fail(h, NETSIM_E_INVALID, "set_link_latency: latency_s is NULL");
  for (int64_t l = 0; l < num_links; ++l)
    if (!finite_nonneg(latency_s[l])) return fail(h, NETSIM_E_INVALID, "set_link_latency: latencies must be finite and >= 0");
  sc.lat.assign(latency_s, latency_s + num_links);
  return NETSIM_OK;
}

}  // extern "C"

namespace {

// In-order binary tree over nodes 1..p: node u of level l = ctz(u) >= 1 has
// children u - 2^(l-1) and u + 2^j for the largest j < l with u + 2^j <= p.
int32_t tree_level(int32_t u) { return __builtin_ctz((unsigned)u); }

struct TreeShape {
  int32_t root = 0;
  std::vector<int32_t> parent;                  // [p+1], 0 for the root
  std::vector<std::vector<int32_t>> kids;       // [p+1]
  std::vector<int32_t> up, down;                // children ordered for reduce / broadcast
};

TreeShape tree_shape(int32_t p) {
  TreeShape t;
  t.parent.assign((size_t)p + 1, 0);
  t.kids.assign((size_t)p + 1, {});
  for (int32_t u = 2; u <= p; u += 2) {
    const int32_t l = tree_level(u);
    t.kids[(size_t)u].push_back(u - (1 << (l - 1)));
    for (int32_t j = l - 1; j >= 0; --j)
      if (u + (1 << j) <= p) {
        t.kids[(size_t)u].push_back(u + (1 << j));
        break;
      }
  }
  for (int32_t u = 1; u <= p; ++u)
    for (int32_t c : t.kids[(size_t)u]) t.parent[(size_t)c] = u;
  t.root = 1;
  while (t.root * 2 <= p) t.root *= 2;
  for (int32_t u = 1; u <= p; ++u)
    if (u != t.root) t.up.push_back(u);
  t.down = t.up;
  // reduce: children before parents (lower level first); broadcast: the reverse
  std::stable_sort(t.up.begin(), t.up.end(), [](int32_t a, int32_t b) {
    return tree_level(a) != tree_level(b) ? tree_level(a) < tree_level(b) : a < b;
  });
  std::stable_sort(t.down.begin(), t.down.end(), [](int32_t a, int32_t b) {
    return tree_level(a) != tree_level(b) ? tree_level(a) > tree_level(b) : a < b;
  });
  return t;
}

// Flows of a rank set laid out as appended rows (src, dst, bytes, lag, deps).
struct FlowRows {
  std::vector<int32_t> src, dst;
  std::vector<double> b, t0;
  std::vector<int64_t> doff{0}, dids;
  void add(int32_t s, int32_t d, double bytes, double lag, const int64_t* deps, size_t nd) {
    src.push_back(s);
    dst.push_back(d);
    b.push_back(bytes);
    t0.push_back(lag);
    dids.insert(dids.end(), deps, deps + nd);
    doff.push_back((int64_t)dids.size());
  }
  int64_t size() const { return (int64_t)b.size(); }
};

netsim_status commit_rows(netsim_t* h, int32_t scen, const FlowRows& r, int64_t first,
                          int64_t* first_id, int64_t* count) {
  netsim_status st = add_flows_impl(h, scen, r.size(), r.src.data(), r.dst.data(), r.b.data(),
                                    r.t0.data(), nullptr, nullptr, r.doff.data(),
                                    r.dids.empty() ? nullptr : r.dids.data(), nullptr);
  if (st) return st;
  if (first_id) *first_id = first;
  if (count) *count = r.size();
  return NETSIM_OK;
}

// Per tree (A: position u-1 at node u; B: position p-u), reduce flows then
// broadcast flows; rank i's completion flows (the broadcasts into and out
// of it in both trees) go to done_of[i] when given.
void tree_rows(int32_t p, const int32_t* ranks, double nbytes, double lag, int64_t n_after,
               const int64_t* after, int64_t first, FlowRows* r,
               std::vector<std::vector<int64_t>>* done_of) {
  const TreeShape t = tree_shape(p);
  std::vector<int64_t> rslot((size_t)p + 1), bslot((size_t)p + 1);
  for (size_t k = 0; k < t.up.size(); ++k) rslot[(size_t)t.up[k]] = (int64_t)k;
  for (size_t k = 0; k < t.down.size(); ++k) bslot[(size_t)t.down[k]] = (int64_t)k;
  const double half = nbytes / 2.0;
  for (int32_t tr = 0; tr < 2; ++tr) {
    auto pos = [&](int32_t u) { return tr == 0 ? u - 1 : p - u; };
    const int64_t red0 = first + (int64_t)tr * 2 * (p - 1);
    const int64_t bc0 = red0 + (p - 1);
    for (int32_t c : t.up) {
      std::vector<int64_t> into;
      for (int32_t x : t.kids[(size_t)c]) into.push_back(red0 + rslot[(size_t)x]);
      if (into.empty())
        r->add(ranks[pos(c)], ranks[pos(t.parent[(size_t)c])], half, lag, after, (size_t)n_after);
      else
        r->add(ranks[pos(c)], ranks[pos(t.parent[(size_t)c])], half, 0.0, into.data(), into.size());
    }
    for (int32_t c : t.down) {
      const int32_t q = t.parent[(size_t)c];
      std::vector<int64_t> dep;
      if (q == t.root)
        for (int32_t x : t.kids[(size_t)q]) dep.push_back(red0 + rslot[(size_t)x]);
      else
        dep.push_back(bc0 + bslot[(size_t)q]);
      r->add(ranks[pos(q)], ranks[pos(c)], half, 0.0, dep.data(), dep.size());
      if (done_of) {
        const int64_t f = bc0 + bslot[(size_t)c];
        (*done_of)[(size_t)pos(q)].push_back(f);
        (*done_of)[(size_t)pos(c)].push_back(f);
      }
    }
  }
}

// Hierarchical all-reduce over an m x g rank array (row = server): per
// server a chained ring reduce-scatter (chunks S/g), per local position a
// chained ring all-reduce across the servers (chunks S/(g m)), per server a
// chained ring all-gather (chunks S/g); a rank's first step of a phase waits
// for its previous phase's last-step flows out of and into it.  done_of
// (row-major rank index) receives each rank's last-phase flows.
void hier_rows(int32_t m, int32_t g, const int32_t* R, double nbytes, double lag, int64_t n_after,
               const int64_t* after, int64_t first, FlowRows* r,
               std::vector<std::vector<int64_t>>* done_of) {
  std::vector<std::vector<int64_t>> done((size_t)m * g);  // previous phase, per rank
  bool started = false;
  auto rk = [&](int32_t a, int32_t i) { return R[(size_t)a * g + i]; };
  auto entry = [&](int32_t a, int32_t i, double bytes, int32_t s, int32_t d) {
    if (started)
      r->add(s, d, bytes, 0.0, done[(size_t)a * g + i].data(), done[(size_t)a * g + i].size());
    else
      r->add(s, d, bytes, lag, after, (size_t)n_after);
  };
  int64_t next = first;
  auto server_rings = [&]() {
    std::vector<std::vector<int64_t>> nd((size_t)m * g);
    for (int32_t a = 0; a < m; ++a) {
      const int64_t base = next;
      for (int32_t k = 0; k < g - 1; ++k)
        for (int32_t i = 0; i < g; ++i) {
          if (k == 0) {
            entry(a, i, nbytes / (double)g, rk(a, i), rk(a, (i + 1) % g));
          } else {
            const int64_t prev = base + (int64_t)(k - 1) * g + (i + g - 1) % g;
            r->add(rk(a, i), rk(a, (i + 1) % g), nbytes / (double)g, 0.0, &prev, 1);
          }
        }
      const int64_t last = base + (int64_t)(g - 2) * g;
      for (int32_t i = 0; i < g; ++i) nd[(size_t)a * g + i] = {last + i, last + (i + g - 1) % g};
      next += (int64_t)(g - 1) * g;
    }
    done.swap(nd);
    started = true;
  };
  if (g > 1) server_rings();
  if (m > 1) {
    std::vector<std::vector<int64_t>> nd((size_t)m * g);
    const int32_t steps = 2 * (m - 1);
    const double chunk = nbytes / ((double)g * (double)m);
    for (int32_t j = 0; j < g; ++j) {
      const int64_t base = next;
      for (int32_t k = 0; k < steps; ++k)
        for (int32_t a = 0; a < m; ++a) {
          if (k == 0) {
            entry(a, j, chunk, rk(a, j), rk((a + 1) % m, j));
          } else {
            const int64_t prev = base + (int64_t)(k - 1) * m + (a + m - 1) % m;
            r->add(rk(a, j), rk((a + 1) % m, j), chunk, 0.0, &prev, 1);
          }
        }
      const int64_t last = base + (int64_t)(steps - 1) * m;
      for (int32_t a = 0; a < m; ++a) nd[(size_t)a * g + j] = {last + a, last + (a + m - 1) % m};
      next += (int64_t)steps * m;
    }
    done.swap(nd);
    started = true;
  }
  if (g > 1) server_rings();
  if (done_of) *done_of = done;
}

netsim_status check_tree_args(netsim_t* h, const char* what, int32_t scen, int32_t p,
                              const int32_t* ranks, double nbytes, double lag, int64_t n_after,
                              const int64_t* after) {
  if (h->prepared) return fail(h, NETSIM_E_STATE, std::string(what) + ": flows cannot be added after a run");
  if (p < 2) return fail(h, NETSIM_E_INVALID, std::string(what) + ": need at least 2 ranks");
  if (!finite_nonneg(nbytes) || !finite_nonneg(lag))
    return fail(h, NETSIM_E_INVALID, std::string(what) + ": bytes and lag must be finite and >= 0");
  netsim_status st = check_ranks(h, scen, p, ranks);
  if (st) return st;
  return check_after(h, scen, n_after, after);
}

}  // namespace

extern "C" {

netsim_status netsim_add_tree_allreduce(netsim_t* h, int32_t scen, int32_t p, const int32_t* ranks,
                                        double nbytes, double lag, int64_t n_after,
                                        const int64_t* after, int64_t* first_id, int64_t* count) {
  if (!h) return fail(nullptr, NETSIM_E_INVALID, "add_tree_allreduce: handle is NULL");
  netsim_status st = check_tree_args(h, "add_tree_allreduce", scen, p, ranks, nbytes, lag, n_after, after);
  if (st) return st;
  const int64_t first = (int64_t)h->f_bytes.size();
  FlowRows r;
  std::vector<std::vector<int64_t>> done((size_t)p);
  tree_rows(p, ranks, nbytes, lag, n_after, after, first, &r, &done);
  st = commit_rows(h, scen, r, first, first_id, count);
  if (st == NETSIM_OK) set_exits(h, done);  // the broadcast flows of both trees
  return st;
}

netsim_status netsim_add_hier_allreduce(netsim_t* h, int32_t scen, int32_t m, int32_t g,
                                        const int32_t* ranks, double nbytes, double lag,
                                        int64_t n_after, const int64_t* after, int64_t* first_id,
                                        int64_t* count) {
  if (!h) return fail(nullptr, NETSIM_E_INVALID, "add_hier_allreduce: handle is NULL");
  if (m < 1 || g < 1 || (int64_t)m * g > std::numeric_limits<int32_t>::max())
    return fail(h, NETSIM_E_INVALID, "add_hier_allreduce: bad m x g");
  netsim_status st = check_tree_args(h, "add_hier_allreduce", scen, m * g, ranks, nbytes, lag, n_after, after);
  if (st) return st;
  const int64_t first = (int64_t)h->f_bytes.size();
  FlowRows r;
  std::vector<std::vector<int64_t>> done;
  hier_rows(m, g, ranks, nbytes, lag, n_after, after, first, &r, &done);
  st = commit_rows(h, scen, r, first, first_id, count);
  if (st == NETSIM_OK) set_exits(h, done);  // the last step of the last phase
  return st;
}

}  // extern "C"

// ------------------------------------------------------- event-queue front end
// A computation is a zero-byte flow whose release lags its dependencies by
// its duration; a rendezvous is a zero-byte flow after the tails of every
// participating stream; an operation's completion on a stream is the flow
// that becomes the stream's tail.

namespace {

netsim_status check_stream_scen(netsim_t* h, int32_t s) {
  if (h->prepared) return fail(h, NETSIM_E_STATE, "stream: operations cannot be added after a run");
  if (s < 0 || s >= (int32_t)h->scen.size()) return fail(h, NETSIM_E_INVALID, "stream: bad scenario");
  return NETSIM_OK;
}

int64_t stream_tail(netsim_t* h, int32_t s, int64_t stream) {
  auto it = h->scen[(size_t)s].tails.find(stream);
  return it == h->scen[(size_t)s].tails.end() ? -1 : it->second;
}

// One zero-byte flow after `deps` (negative entries ignored) and `lag`.
netsim_status zero_flow(netsim_t* h, int32_t s, std::vector<int64_t> deps, double lag, int64_t* id) {
  deps.erase(std::remove_if(deps.begin(), deps.end(), [](int64_t d) { return d < 0; }), deps.end());
  std::sort(deps.begin(), deps.end());
  deps.erase(std::unique(deps.begin(), deps.end()), deps.end());
  const int64_t poff[2] = {0, 0};
  const int64_t doff[2] = {0, (int64_t)deps.size()};
  const double zero = 0.0;
  const int32_t none = -1;
  return add_flows_impl(h, s, 1, &none, &none, &zero, &lag, poff, nullptr, doff,
                        deps.empty() ? nullptr : deps.data(), id);
}

netsim_status check_streams(netsim_t* h, int32_t p, const int64_t* streams, int64_t* done) {
  if (!streams || !done) return fail(h, NETSIM_E_INVALID, "stream collective: streams and done are required");
  std::vector<int64_t> v(streams, streams + p);
  std::sort(v.begin(), v.end());
  if (std::adjacent_find(v.begin(), v.end()) != v.end())
    return fail(h, NETSIM_E_INVALID, "stream collective: a stream appears twice");
  return NETSIM_OK;
}

// Rendezvous of the streams, the collective after it (added by `add` with
// the rendezvous as its only predecessor), and one completion flow per rank
// after the collective flows that rank i still waits for (deps_of(i)).
template <class Add, class DepsOf>
netsim_status stream_collective(netsim_t* h, int32_t s, int32_t p, const int64_t* streams,
                                int64_t* done, Add add, DepsOf deps_of) {
  netsim_status st = check_streams(h, p, streams, done);
  if (st) return st;
  const size_t mark = h->f_bytes.size();
  std::vector<int64_t> tails((size_t)p);
  for (int32_t i = 0; i < p; ++i) tails[(size_t)i] = stream_tail(h, s, streams[i]);
  int64_t rv = -1;
  st = zero_flow(h, s, tails, 0.0, &rv);
  int64_t first = -1;
  if (!st) st = add(rv, &first);
  std::vector<int64_t> ids((size_t)p);
  for (int32_t i = 0; i < p && !st; ++i) st = zero_flow(h, s, deps_of(first, i), 0.0, &ids[(size_t)i]);
  if (st) {
    // all or nothing: drop what this call appended
    while (h->f_bytes.size() > mark) {
      h->f_scen.pop_back(); h->f_src.pop_back(); h->f_dst.pop_back();
      h->f_bytes.pop_back(); h->f_start.pop_back();
      h->p_link.resize((size_t)h->p_off[h->p_off.size() - 2]);
      h->p_off.pop_back();
      h->d_ids.resize((size_t)h->d_off[h->d_off.size() - 2]);
      h->d_off.pop_back();
      h->scen[(size_t)s].flows.pop_back();
    }
    return st;
  }
  for (int32_t i = 0; i < p; ++i) {
    h->scen[(size_t)s].tails[streams[i]] = ids[(size_t)i];
    done[i] = ids[(size_t)i];
  }
  return NETSIM_OK;
}

}  // namespace

extern "C" {

netsim_status netsim_stream_compute(netsim_t* h, int32_t scen, int64_t stream, double duration,
                                    int64_t n_wait, const int64_t* wait, int64_t* done) {
  if (!h) return fail(nullptr, NETSIM_E_INVALID, "stream_compute: handle is NULL");
  netsim_status st = check_stream_scen(h, scen);
  if (st) return st;
  if (!finite_nonneg(duration)) return fail(h, NETSIM_E_INVALID, "stream_compute: duration must be finite and >= 0");
  if (n_wait < 0 || (n_wait > 0 && !wait)) return fail(h, NETSIM_E_INVALID, "stream_compute: bad wait list");
  std::vector<int64_t> deps(wait, wait + n_wait);
  deps.push_back(stream_tail(h, scen, stream));
  int64_t id = -1;
  st = zero_flow(h, scen, deps, duration, &id);
  if (st) return st;
  h->scen[(size_t)scen].tails[stream] = id;
  if (done) *done = id;
  return NETSIM_OK;
}

netsim_status netsim_stream_wait(netsim_t* h, int32_t scen, int64_t stream, int64_t n_wait,
                                 const int64_t* wait) {
  return netsim_stream_compute(h, scen, stream, 0.0, n_wait, wait, nullptr);
}

netsim_status netsim_stream_tail(const netsim_t* h, int32_t scen, int64_t stream, int64_t* flow) {
  if (!h || !flow) return fail(h, NETSIM_E_INVALID, "stream_tail: NULL argument");
  if (scen < 0 || scen >= (int32_t)h->scen.size()) return fail(h, NETSIM_E_INVALID, "stream_tail: bad scenario");
  *flow = stream_tail(const_cast<netsim_t*>(h), scen, stream);
  return NETSIM_OK;
}

netsim_status netsim_stream_ring(netsim_t* h, int32_t scen, int32_t kind, int32_t mode, int32_t p,
                                 const int32_t* ranks, const int64_t* streams, double nbytes,
                                 int64_t* done) {
  if (!h) return fail(nullptr, NETSIM_E_INVALID, "stream_ring: handle is NULL");
  netsim_status st = check_stream_scen(h, scen);
  if (st) return st;
  if (p < 2) return fail(h, NETSIM_E_INVALID, "stream_ring: need p >= 2");
  if (mode < NETSIM_MODE_CHAINED || mode > NETSIM_MODE_AGGREGATED) return fail(h, NETSIM_E_INVALID, "stream_ring: bad mode");
  const int64_t steps = kind == NETSIM_RING_ALLREDUCE ? 2 * (int64_t)(p - 1) : (int64_t)(p - 1);
  return stream_collective(
      h, scen, p, streams, done,
      [&](int64_t rv, int64_t* first) {
        return netsim_add_ring(h, scen, kind, mode, p, ranks, nbytes, 0.0, 1, &rv, first, nullptr);
      },
      [&](int64_t first, int32_t i) {
        // rank i is done when the flows out of it and into it are
        const int64_t in = (i + p - 1) % p;
        std::vector<int64_t> d;
        if (mode == NETSIM_MODE_AGGREGATED) {
          d = {first + i, first + in};
        } else if (mode == NETSIM_MODE_CHAINED) {
          d = {first + (steps - 1) * p + i, first + (steps - 1) * p + in};
        } else {
          for (int64_t k = 0; k < steps; ++k) {
            d.push_back(first + k * p + i);
            d.push_back(first + k * p + in);
          }
        }
        return d;
      });
}

netsim_status netsim_stream_all_to_all(netsim_t* h, int32_t scen, int32_t p, const int32_t* ranks,
                                       const int64_t* streams, const double* nbytes, int64_t* done) {
  if (!h) return fail(nullptr, NETSIM_E_INVALID, "stream_all_to_all: handle is NULL");
  netsim_status st = check_stream_scen(h, scen);
  if (st) return st;
  if (p < 2) return fail(h, NETSIM_E_INVALID, "stream_all_to_all: need p >= 2");
  return stream_collective(
      h, scen, p, streams, done,
      [&](int64_t rv, int64_t* first) {
        return netsim_add_all_to_all(h, scen, p, ranks, nbytes, 0.0, 1, &rv, first, nullptr);
      },
      [&](int64_t first, int32_t i) {
        std::vector<int64_t> d;
        auto id = [&](int32_t a, int32_t b) { return first + (int64_t)a * (p - 1) + (b < a ? b : b - 1); };
        for (int32_t j = 0; j < p; ++j)
          if (j != i) {
            d.push_back(id(i, j));
            d.push_back(id(j, i));
          }
        return d;
      });
}

netsim_status netsim_stream_send(netsim_t* h, int32_t scen, int32_t src, int64_t src_stream,
                                 int32_t dst, int64_t dst_stream, double nbytes, int64_t* done) {
  if (!h) return fail(nullptr, NETSIM_E_INVALID, "stream_send: handle is NULL");
  netsim_status st = check_stream_scen(h, scen);
  if (st) return st;
  if (src_stream == dst_stream) return fail(h, NETSIM_E_INVALID, "stream_send: the two ends need two streams");
  const int64_t streams[2] = {src_stream, dst_stream};
  int64_t d2[2];
  st = stream_collective(
      h, scen, 2, streams, d2,
      [&](int64_t rv, int64_t* first) {
        const int64_t doff[2] = {0, 1};
        const double lag = 0.0;
        return add_flows_impl(h, scen, 1, &src, &dst, &nbytes, &lag, nullptr, nullptr, doff, &rv, first);
      },
      [&](int64_t first, int32_t) { return std::vector<int64_t>{first}; });
  if (st) return st;
  if (done) *done = d2[0];
  return NETSIM_OK;
}

netsim_status netsim_stream_tree_allreduce(netsim_t* h, int32_t scen, int32_t p,
                                           const int32_t* ranks, const int64_t* streams,
                                           double nbytes, int64_t* done) {
  if (!h) return fail(nullptr, NETSIM_E_INVALID, "stream_tree_allreduce: handle is NULL");
  netsim_status st = check_stream_scen(h, scen);
  if (st) return st;
  if (p < 2) return fail(h, NETSIM_E_INVALID, "stream_tree_allreduce: need p >= 2");
  std::vector<std::vector<int64_t>> per_rank;
  return stream_collective(
      h, scen, p, streams, done,
      [&](int64_t rv, int64_t* first) {
        netsim_status s2 = netsim_add_tree_allreduce(h, scen, p, ranks, nbytes, 0.0, 1, &rv, first, nullptr);
        if (s2) return s2;
        FlowRows scratch;
        per_rank.assign((size_t)p, {});
        tree_rows(p, ranks, nbytes, 0.0, 1, &rv, *first, &scratch, &per_rank);
        return (netsim_status)NETSIM_OK;
      },
      [&](int64_t, int32_t i) { return per_rank[(size_t)i]; });
}

netsim_status netsim_stream_hier_allreduce(netsim_t* h, int32_t scen, int32_t m, int32_t g,
                                           const int32_t* ranks, const int64_t* streams,
                                           double nbytes, int64_t* done) {
  if (!h) return fail(nullptr, NETSIM_E_INVALID, "stream_hier_allreduce: handle is NULL");
  netsim_status st = check_stream_scen(h, scen);
  if (st) return st;
  if (m < 1 || g < 1 || (int64_t)m * g < 2 || (int64_t)m * g > std::numeric_limits<int32_t>::max())
    return fail(h, NETSIM_E_INVALID, "stream_hier_allreduce: bad m x g");
  std::vector<std::vector<int64_t>> per_rank;
  return stream_collective(
      h, scen, m * g, streams, done,
      [&](int64_t rv, int64_t* first) {
        netsim_status s2 = netsim_add_hier_allreduce(h, scen, m, g, ranks, nbytes, 0.0, 1, &rv, first, nullptr);
        if (s2) return s2;
        FlowRows scratch;
        hier_rows(m, g, ranks, nbytes, 0.0, 1, &rv, *first, &scratch, &per_rank);
        return (netsim_status)NETSIM_OK;
      },
      [&](int64_t, int32_t i) { return per_rank[(size_t)i]; });
}

netsim_status netsim_last_exits(const netsim_t* h, int64_t* n, int64_t* ids) {
  if (!h || !n) return fail(h, NETSIM_E_INVALID, "last_exits: NULL argument");
  if (!h->has_exits) return fail(h, NETSIM_E_STATE, "last_exits: no operation appended yet");
  *n = (int64_t)h->last_exits.size();
  if (ids) std::copy(h->last_exits.begin(), h->last_exits.end(), ids);
  return NETSIM_OK;
}

netsim_status netsim_counts(const netsim_t* h, int64_t* num_flows, int64_t* num_incidences,
                            int64_t* num_deps) {
  if (!h) return fail(nullptr, NETSIM_E_INVALID, "counts: handle is NULL");
  if (num_flows) *num_flows = (int64_t)h->f_bytes.size();
  if (num_incidences) *num_incidences = (int64_t)h->p_link.size();
  if (num_deps) *num_deps = (int64_t)h->d_ids.size();
  return NETSIM_OK;
}

netsim_status netsim_export_flows(const netsim_t* h, int32_t* scen, int32_t* src, int32_t* dst,
                                  double* nbytes, double* start, int64_t* path_off,
                                  int32_t* path_link, int64_t* dep_off, int64_t* dep_ids) {
  if (!h) return fail(nullptr, NETSIM_E_INVALID, "export_flows: handle is NULL");
  if (scen) std::copy(h->f_scen.begin(), h->f_scen.end(), scen);
  if (src) std::copy(h->f_src.begin(), h->f_src.end(), src);
  if (dst) std::copy(h->f_dst.begin(), h->f_dst.end(), dst);
  if (nbytes) std::copy(h->f_bytes.begin(), h->f_bytes.end(), nbytes);
  if (start) std::copy(h->f_start.begin(), h->f_start.end(), start);
  if (path_off) std::copy(h->p_off.begin(), h->p_off.end(), path_off);
  if (path_link) std::copy(h->p_link.begin(), h->p_link.end(), path_link);
  if (dep_off) std::copy(h->d_off.begin(), h->d_off.end(), dep_off);
  if (dep_ids) std::copy(h->d_ids.begin(), h->d_ids.end(), dep_ids);
  return NETSIM_OK;
}

netsim_status netsim_set_limits(netsim_t* h, int64_t max_events, double until) {
  if (!h) return fail(nullptr, NETSIM_E_INVALID, "set_limits: handle is NULL");
  if (max_events < 0 || std::isnan(until)) return fail(h, NETSIM_E_INVALID, "set_limits: bad limit");
  h->opt.max_events = max_events;
  h->opt.until = until;
  return NETSIM_OK;
}

netsim_status netsim_run(netsim_t* h, void* hip_stream) {
  if (!h) return fail(nullptr, NETSIM_E_INVALID, "run: handle is NULL");
  return simulate(h, (hipStream_t)hip_stream, false, -1, std::numeric_limits<double>::quiet_NaN());
}

netsim_status netsim_advance(netsim_t* h, double until, int64_t max_events, void* hip_stream) {
  if (!h) return fail(nullptr, NETSIM_E_INVALID, "advance: handle is NULL");
  if (std::isnan(until) || max_events < 0) return fail(h, NETSIM_E_INVALID, "advance: bad limit");
  hipStream_t st = (hipStream_t)hip_stream;
  netsim_status rc = simulate(h, st, true, max_events, until);
  if (rc) return rc;
  return h->F > 0 ? push_checkpoint(h, st) : NETSIM_OK;
}

netsim_status netsim_update_start(netsim_t* h, int64_t id, double start) {
  if (!h) return fail(nullptr, NETSIM_E_INVALID, "update_start: handle is NULL");
  const int64_t F = (int64_t)h->f_bytes.size();
  if (id < 0 || id >= F) return fail(h, NETSIM_E_INVALID, "update_start: no such flow");
  if (!finite_nonneg(start)) return fail(h, NETSIM_E_INVALID, "update_start: start must be finite and >= 0");
  h->f_start[(size_t)id] = start;
  if (!h->prepared) return NETSIM_OK;  // uploaded by the first run
  hipError_t he = hipSetDevice(h->opt.device);
  if (he != hipSuccess) return hip_fail(h, he, "hipSetDevice");
  const Params& P = h->prm;
  const int32_t d = h->dev_of_flow[(size_t)id];
  he = hipMemcpy(const_cast<double*>(P.start) + d, &start, sizeof(double), hipMemcpyHostToDevice);
  if (he != hipSuccess) return hip_fail(h, he, "hipMemcpy (start)");
  if (!h->has_state) return NETSIM_OK;  // the next run starts from t = 0 with it
  const int32_t p = part_of_dev(h, d);
  int32_t cnt = 0;
  double rel_old = 0.0, base = 0.0;
  he = hipMemcpy(&cnt, P.cnt + d, sizeof(int32_t), hipMemcpyDeviceToHost);
  if (he == hipSuccess) he = hipMemcpy(&rel_old, P.rel + d, sizeof(double), hipMemcpyDeviceToHost);
  if (he == hipSuccess) he = hipMemcpy(&base, P.base + d, sizeof(double), hipMemcpyDeviceToHost);
  if (he != hipSuccess) return hip_fail(h, he, "hipMemcpy (flow state)");
  if (cnt > 0) return NETSIM_OK;  // waiting for predecessors: applies when they finish
  const double t_part = h->part_t[(size_t)p];
  const double rel_new = start + base;
  const bool released = rel_old <= t_part;
  if (!released && rel_new >= t_part) {
    // still pending and the new release is not in the part's past
    he = hipMemcpy(P.rel + d, &rel_new, sizeof(double), hipMemcpyHostToDevice);
    return he == hipSuccess ? NETSIM_OK : hip_fail(h, he, "hipMemcpy (release)");
  }
  // time rollback (Section 4.2): the part goes back to the latest state in
  // which the flow was not yet released and that precedes its new release
  const double before = released ? std::min(rel_old, rel_new) : rel_new;
  bool done = false;
  netsim_status rc = history_rollback(h, p, before, &done);
  if (rc) return rc;
  if (!done) {
    rc = restore_part(h, p, latest_checkpoint(h, p, before));
    if (rc) return rc;
  }
  he = hipMemcpy(&cnt, P.cnt + d, sizeof(int32_t), hipMemcpyDeviceToHost);
  if (he != hipSuccess) return hip_fail(h, he, "hipMemcpy (flow state)");
  if (cnt == 0) {
    he = hipMemcpy(P.rel + d, &rel_new, sizeof(double), hipMemcpyHostToDevice);
    if (he != hipSuccess) return hip_fail(h, he, "hipMemcpy (release)");
  }
  return NETSIM_OK;
}

netsim_status netsim_gc(netsim_t* h, double t_min) {
  if (!h) return fail(nullptr, NETSIM_E_INVALID, "gc: handle is NULL");
  if (std::isnan(t_min)) return fail(h, NETSIM_E_INVALID, "gc: bad time");
  auto& cps = h->checkpoints;
  std::vector<char> keep(cps.size(), 1);
  for (size_t k = 0; k < cps.size(); ++k) {
    bool covered = true;  // every part that may use k has a later checkpoint before t_min
    for (int32_t p = 0; p < h->num_parts && covered; ++p) {
      if (!cps[k].valid[(size_t)p]) continue;
      bool later = false;
      for (size_t j = k + 1; j < cps.size() && !later; ++j)
        later = cps[j].valid[(size_t)p] && cps[j].t[(size_t)p] < t_min;
      covered = later;
    }
    if (covered) keep[k] = 0;
  }
  std::vector<netsim_t::Checkpoint> out;
  for (size_t k = 0; k < cps.size(); ++k) {
    if (keep[k]) out.push_back(std::move(cps[k]));
    else (void)hipFree(cps[k].dev);
  }
  cps = std::move(out);
  return NETSIM_OK;
}

netsim_status netsim_num_checkpoints(const netsim_t* h, int64_t* n) {
  if (!h || !n) return fail(h, NETSIM_E_INVALID, "num_checkpoints: NULL argument");
  *n = (int64_t)h->checkpoints.size();
  return NETSIM_OK;
}

netsim_status netsim_get_finish(const netsim_t* h, double* finish, double* makespan) {
  if (!h) return fail(nullptr, NETSIM_E_INVALID, "get_finish: handle is NULL");
  if (!h->has_result) return fail(h, NETSIM_E_STATE, "get_finish: no run yet");
  if (!finish && h->F > 0) return fail(h, NETSIM_E_INVALID, "get_finish: finish is NULL");
  std::copy(h->finish.begin(), h->finish.end(), finish);
  if (makespan) std::copy(h->makespan.begin(), h->makespan.end(), makespan);
  return NETSIM_OK;
}

netsim_status netsim_get_finish_device(const netsim_t* h, double* d_finish) {
  if (!h) return fail(nullptr, NETSIM_E_INVALID, "get_finish_device: handle is NULL");
  if (!h->has_result) return fail(h, NETSIM_E_STATE, "get_finish_device: no run yet");
  if (h->F == 0) return NETSIM_OK;
  if (!d_finish) return fail(h, NETSIM_E_INVALID, "get_finish_device: pointer is NULL");
  hipError_t he = hipMemcpy(d_finish, h->finish.data(), sizeof(double) * (size_t)h->F, hipMemcpyHostToDevice);
  if (he != hipSuccess) return hip_fail(h, he, "hipMemcpy (finish to device)");
  return NETSIM_OK;
}

netsim_status netsim_get_stats(const netsim_t* h, netsim_stats* stats) {
  if (!h || !stats) return fail(h, NETSIM_E_INVALID, "get_stats: NULL argument");
  *stats = h->stats;
  return NETSIM_OK;
}

netsim_status netsim_solve_once(netsim_t* h, int32_t scen, int64_t n_active, const int64_t* active_ids,
                                double* rates_out) {
  if (!h) return fail(nullptr, NETSIM_E_INVALID, "solve_once: handle is NULL");
  if (scen < 0 || scen >= (int32_t)h->scen.size()) return fail(h, NETSIM_E_INVALID, "solve_once: bad scenario");
  if (n_active < 0 || (n_active > 0 && (!active_ids || !rates_out)))
    return fail(h, NETSIM_E_INVALID, "solve_once: bad arguments");
  const int64_t F = (int64_t)h->f_bytes.size();
  std::vector<char> seen((size_t)F, 0);
  for (int64_t k = 0; k < n_active; ++k) {
    const int64_t id = active_ids[k];
    if (id < 0 || id >= F || h->f_scen[(size_t)id] != scen) return fail(h, NETSIM_E_INVALID, "solve_once: id not in the scenario");
    if (seen[(size_t)id]) return fail(h, NETSIM_E_INVALID, "solve_once: repeated id");
    if (h->p_off[(size_t)id + 1] == h->p_off[(size_t)id]) return fail(h, NETSIM_E_INVALID, "solve_once: flow without a path");
    seen[(size_t)id] = 1;
  }
  netsim_status rc;
  if (!h->prepared) {
    rc = prepare(h);
    if (rc) return rc;
  }
  hipError_t he = hipSetDevice(h->opt.device);
  if (he != hipSuccess) return hip_fail(h, he, "hipSetDevice");
  rc = reset_state(h, nullptr);
  if (rc) return rc;
  const Params& P = h->prm;
  std::vector<ScenCtl> ctl = h->h_ctl0;
  for (auto& c : ctl) c.n_solve = 0;
  // the active flows of each part, listed in that part's act0 slice (parts
  // share no link, so the allocation splits into one solve per part)
  std::vector<int32_t> part_of((size_t)std::max<int64_t>(n_active, 1));
  for (int64_t k = 0; k < n_active; ++k) {
    const int32_t d = h->dev_of_flow[(size_t)active_ids[k]];
    int32_t lo = 0, hi = h->num_parts - 1;
    while (lo < hi) {
      const int32_t mid = (lo + hi) / 2;
      if (ctl[(size_t)mid].f1 <= d) lo = mid + 1; else hi = mid;
    }
    part_of[(size_t)k] = lo;
    ctl[(size_t)lo].n_solve += 1;
  }
  std::vector<int32_t> list((size_t)std::max<int64_t>(h->F, 1));
  std::vector<int32_t> dev((size_t)std::max<int64_t>(n_active, 1));
  std::vector<int32_t> fill((size_t)std::max<int32_t>(h->num_parts, 1), 0);
  std::vector<int32_t> nact((size_t)std::max<int64_t>(h->L, 1), 0);
  for (int64_t k = 0; k < n_active; ++k) {
    const int64_t id = active_ids[k];
    const int32_t d = h->dev_of_flow[(size_t)id];
    const int32_t pk = part_of[(size_t)k];
    dev[(size_t)k] = d;
    list[(size_t)(ctl[(size_t)pk].f0 + fill[(size_t)pk]++)] = d;
    for (int64_t e = h->p_off[(size_t)id]; e < h->p_off[(size_t)id + 1]; ++e)
      nact[(size_t)h->dev_link[(size_t)scen][(size_t)h->p_link[(size_t)e]]] += 1;
  }
  // exact mode: wide solves on the whole GPU, the others one workgroup each
  std::vector<std::pair<int32_t, int32_t>> wide;
  if (h->opt.exact)
    for (int32_t k = 0; k < h->num_parts; ++k) {
      ScenCtl& c = ctl[(size_t)k];
      if (c.n_solve > 0 && (c.n_solve >= kExactGridMin || (h->opt.debug & DEBUG_EXACT_GRID))) {
        wide.emplace_back(k, c.n_solve);
        c.n_solve = 0;
      }
    }
  he = hipMemcpy(P.ctl, ctl.data(), sizeof(ScenCtl) * ctl.size(), hipMemcpyHostToDevice);
  if (he == hipSuccess && h->F > 0)
    he = hipMemcpy(P.act0, list.data(), sizeof(int32_t) * (size_t)h->F, hipMemcpyHostToDevice);
  if (he == hipSuccess) he = hipMemcpy(P.nact, nact.data(), sizeof(int32_t) * nact.size(), hipMemcpyHostToDevice);
  if (he != hipSuccess) return hip_fail(h, he, "hipMemcpy (solve_once setup)");
  float ms = 0.0f;
  rc = launch(h, nullptr, true, &ms);
  if (rc) return rc;
  std::vector<ScenCtl> out;
  rc = collect(h, &out);
  if (rc) return rc;
  GridStats gs;
  if (!wide.empty()) {
    hipEvent_t e0, e1;
    he = hipEventCreate(&e0);
    if (he == hipSuccess) he = hipEventCreate(&e1);
    if (he != hipSuccess) return hip_fail(h, he, "hipEventCreate");
    he = hipEventRecord(e0, nullptr);
    for (const auto& w : wide) {
      if (he != hipSuccess) break;
      rc = grid_solve(h, nullptr, w.first, w.second, &gs);
      if (rc) break;
      out[(size_t)w.first].solves += 1;
    }
    float gms = 0.0f;
    if (he == hipSuccess && !rc) he = hipEventRecord(e1, nullptr);
    if (he == hipSuccess && !rc) he = hipEventSynchronize(e1);
    if (he == hipSuccess && !rc) he = hipEventElapsedTime(&gms, e0, e1);
    (void)hipEventDestroy(e0);
    (void)hipEventDestroy(e1);
    if (rc) return rc;
    if (he != hipSuccess) return hip_fail(h, he, "wide exact solve timing");
    ms += gms;
  }
  std::vector<double> rate((size_t)std::max<int64_t>(h->F, 1));
  he = hipMemcpy(rate.data(), P.rate, sizeof(double) * (size_t)std::max<int64_t>(h->F, 1), hipMemcpyDeviceToHost);
  if (he != hipSuccess) return hip_fail(h, he, "hipMemcpy (rates)");
  for (int64_t k = 0; k < n_active; ++k) rates_out[k] = rate[(size_t)dev[(size_t)k]];
  h->stats = netsim_stats{};
  h->stats.complete = 1;
  h->stats.parts = h->num_parts;
  h->stats.device_seconds = ms * 1e-3;
  int khz = 0;
  if (hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, h->opt.device) != hipSuccess || khz <= 0)
    khz = 100000;
  for (int32_t k = 0; k < h->num_parts; ++k) {
    const ScenCtl& c = out[(size_t)k];
    if (c.scen != scen) continue;
    h->stats.solves += c.solves;
    h->stats.rounds += c.rounds;
    h->stats.flows_swept += c.flows_swept;
    h->stats.incidences_swept += c.incidences_swept;
    h->stats.links_swept += c.links_swept;
    for (int j = 0; j < 8; ++j) h->stats.phase_seconds[j] += (double)c.ticks[j] / (1e3 * khz);
  }
  h->stats.rounds += (int64_t)gs.levels;
  h->stats.flows_swept += (int64_t)gs.fsw;
  h->stats.incidences_swept += (int64_t)gs.isw;
  h->stats.links_swept += (int64_t)gs.lsw;
  h->stats.layout = h->opt.exact ? NETSIM_EXEC_EXACT : h->layout;
  return NETSIM_OK;
}

netsim_status netsim_bench_sweeps(netsim_t* h, int32_t scen, int64_t n_active, const int64_t* active_ids,
                                  int32_t reps, int64_t flush_bytes, void* hip_stream, double* count_ms,
                                  double* freeze_ms, double* count_kernel_ms, double* freeze_kernel_ms) {
  if (!h) return fail(nullptr, NETSIM_E_INVALID, "bench_sweeps: handle is NULL");
  if (!h->opt.exact) return fail(h, NETSIM_E_STATE, "bench_sweeps: needs a handle in exact mode");
  if (scen < 0 || scen >= (int32_t)h->scen.size()) return fail(h, NETSIM_E_INVALID, "bench_sweeps: bad scenario");
  if (n_active < 1 || n_active > std::numeric_limits<int32_t>::max() || !active_ids || reps < 1 ||
      flush_bytes < 0 || !count_ms || !freeze_ms)
    return fail(h, NETSIM_E_INVALID, "bench_sweeps: bad arguments");
  const int64_t F = (int64_t)h->f_bytes.size();
  std::vector<char> seen((size_t)F, 0);
  for (int64_t k = 0; k < n_active; ++k) {
    const int64_t id = active_ids[k];
    if (id < 0 || id >= F || h->f_scen[(size_t)id] != scen) return fail(h, NETSIM_E_INVALID, "bench_sweeps: id not in the scenario");
    if (seen[(size_t)id]) return fail(h, NETSIM_E_INVALID, "bench_sweeps: repeated id");
    if (h->p_off[(size_t)id + 1] == h->p_off[(size_t)id]) return fail(h, NETSIM_E_INVALID, "bench_sweeps: flow without a path");
    seen[(size_t)id] = 1;
  }
  netsim_status rc;
  if (!h->prepared) {
    rc = prepare(h);
    if (rc) return rc;
  }
  hipError_t he = hipSetDevice(h->opt.device);
  if (he != hipSuccess) return hip_fail(h, he, "hipSetDevice");
  hipStream_t st = static_cast<hipStream_t>(hip_stream);
  rc = reset_state(h, st);
  if (rc) return rc;
  int32_t p = -1;  // exact mode: one part per scenario
  for (int32_t k = 0; k < h->num_parts; ++k)
    if (h->h_ctl0[(size_t)k].scen == scen) p = k;
  if (p < 0) return fail(h, NETSIM_E_INVALID, "bench_sweeps: the scenario has no flows");
  const ScenCtl& C = h->h_ctl0[(size_t)p];
  std::vector<int32_t> list((size_t)n_active);
  for (int64_t k = 0; k < n_active; ++k) list[(size_t)k] = h->dev_of_flow[(size_t)active_ids[k]];
  const Params& P = h->prm;
  he = hipMemcpy(P.act0 + C.f0, list.data(), sizeof(int32_t) * list.size(), hipMemcpyHostToDevice);
  if (he != hipSuccess) return hip_fail(h, he, "hipMemcpy (bench_sweeps setup)");
  void* buf = nullptr;
  const size_t fb = (size_t)flush_bytes / 16 * 16;
  if (fb > 0 && hipMalloc(&buf, fb) != hipSuccess) {
    (void)hipGetLastError();
    return fail(h, NETSIM_E_NOMEM, "bench_sweeps: no memory for the flush buffer");
  }
  // per-workgroup wall-clock stamps of the two sweeps
  const int e0 = h->h_lfoff[(size_t)C.l0], e1 = h->h_lfoff[(size_t)C.l1];
  const int cb = netsim_dev::count_blocks(e0, e1), fbk = netsim_dev::freeze_blocks((int)n_active);
  unsigned long long* stamps = nullptr;
  if (hipMalloc(&stamps, sizeof(unsigned long long) * 2 * (size_t)(cb + fbk)) != hipSuccess) {
    (void)hipGetLastError();
    if (buf) (void)hipFree(buf);
    return fail(h, NETSIM_E_NOMEM, "bench_sweeps: no memory for the time stamps");
  }
  std::vector<unsigned long long> hs((size_t)2 * (cb + fbk));
  int khz = 0;
  if (hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, h->opt.device) != hipSuccess || khz <= 0)
    khz = 100000;
  auto span_ms = [&](const unsigned long long* a, int blocks) {
    unsigned long long lo = ~0ull, hi = 0;
    for (int b = 0; b < blocks; ++b) {
      lo = std::min(lo, a[2 * b]);
      hi = std::max(hi, a[2 * b + 1]);
    }
    return hi > lo ? (double)(hi - lo) / (double)khz : 0.0;
  };
  hipEvent_t ev[4] = {};
  for (auto& e : ev)
    if (he == hipSuccess) he = hipEventCreate(&e);
  const int n = (int)n_active;
  for (int32_t r = 0; r < reps && he == hipSuccess; ++r) {
    // cold caches before each sweep: a streaming write larger than the L2s
    // and the Infinity Cache together
    if (fb > 0) he = netsim_dev::launch_flush(buf, fb, (uint32_t)(2 * r), st);
    if (he == hipSuccess) he = netsim_dev::grid_solve_begin(P, C, n, st);
    if (he == hipSuccess) he = hipEventRecord(ev[0], st);
    if (he == hipSuccess) he = netsim_dev::grid_solve_count(P, C, e0, e1, st, stamps);
    if (he == hipSuccess) he = hipEventRecord(ev[1], st);
    if (he == hipSuccess && fb > 0) he = netsim_dev::launch_flush(buf, fb, (uint32_t)(2 * r + 1), st);
    if (he == hipSuccess) he = netsim_dev::grid_solve_links(P, C, 0, st);
    if (he == hipSuccess) he = hipEventRecord(ev[2], st);
    if (he == hipSuccess) he = netsim_dev::grid_solve_freeze(P, C, n, 0, st, stamps + 2 * cb);
    if (he == hipSuccess) he = hipEventRecord(ev[3], st);
    if (he == hipSuccess) he = hipEventSynchronize(ev[3]);
    float a = 0.0f, b = 0.0f;
    if (he == hipSuccess) he = hipEventElapsedTime(&a, ev[0], ev[1]);
    if (he == hipSuccess) he = hipEventElapsedTime(&b, ev[2], ev[3]);
    count_ms[r] = a;
    freeze_ms[r] = b;
    if (he == hipSuccess)
      he = hipMemcpy(hs.data(), stamps, sizeof(unsigned long long) * hs.size(), hipMemcpyDeviceToHost);
    if (he == hipSuccess) {
      if (count_kernel_ms) count_kernel_ms[r] = span_ms(hs.data(), cb);
      if (freeze_kernel_ms) freeze_kernel_ms[r] = span_ms(hs.data() + 2 * cb, fbk);
    }
  }
  for (auto& e : ev)
    if (e) (void)hipEventDestroy(e);
  if (buf) (void)hipFree(buf);
  (void)hipFree(stamps);
  if (he != hipSuccess) return hip_fail(h, he, "bench_sweeps");
  h->has_state = false;  // the device holds no simulation position now
  return NETSIM_OK;
}

const char* netsim_last_error(const netsim_t* h) {
  return h ? h->err.c_str() : g_thread_err.c_str();
}

void netsim_destroy(netsim_t* h) {
  if (!h) return;
  if (h->d_block) {
    (void)hipSetDevice(h->opt.device);
    drop_checkpoints(h);
    (void)hipFree(h->d_block);
    if (h->d_hist) (void)hipFree(h->d_hist);
  }
  delete h;
}

}  // extern "C"
