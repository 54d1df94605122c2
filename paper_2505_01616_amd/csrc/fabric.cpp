#include "fabric.h"

#include <cmath>
#include <limits>

namespace netsim_host {

namespace {
bool good_rate(double x) { return std::isfinite(x) && x > 0.0; }
}  // namespace

bool Fabric::init(const netsim_topology& t, std::string* err) {
  kind_ = t.kind;
  S_ = t.servers;
  G_ = t.gpus_per_server;
  spl_ = t.servers_per_leaf;
  spines_ = t.spines;
  P_ = t.pods;
  E_ = t.edges_per_pod;
  A_ = t.aggs_per_pod;
  U_ = t.agg_uplinks;
  if (S_ <= 0 || G_ <= 0 || spl_ <= 0 || S_ % spl_ != 0) {
    *err = "topology: need servers > 0, gpus_per_server > 0 and servers_per_leaf dividing servers";
    return false;
  }
  N_ = S_ * G_;
  NV_ = S_ * G_ * (G_ - 1);
  if (kind_ == NETSIM_TOPO_LEAF_SPINE || kind_ == NETSIM_TOPO_RAIL) {
    if (spines_ <= 0) {
      *err = "topology: spines must be > 0";
      return false;
    }
    groups_ = S_ / spl_;
    leaves_ = kind_ == NETSIM_TOPO_LEAF_SPINE ? groups_ : G_ * groups_;
    ncab_ = N_ + leaves_ * spines_;
  } else if (kind_ == NETSIM_TOPO_FAT_TREE) {
    if (P_ <= 0 || E_ <= 0 || A_ <= 0 || U_ <= 0 || P_ * E_ * spl_ != S_) {
      *err = "topology: fat tree needs pods, edges, aggs, uplinks > 0 and servers = pods*edges*servers_per_leaf";
      return false;
    }
    ncab_ = N_ + P_ * E_ * A_ + P_ * A_ * U_;
  } else {
    *err = "topology: unknown kind";
    return false;
  }
  L_ = NV_ + 2 * ncab_;
  if (L_ > std::numeric_limits<int32_t>::max() || N_ > std::numeric_limits<int32_t>::max()) {
    *err = "topology: more than 2^31-1 links or endpoints";
    return false;
  }
  if ((G_ > 1 && !good_rate(t.nvlink_Bps)) || !good_rate(t.nic_Bps) || !good_rate(t.fabric_Bps)) {
    *err = "topology: link rates must be finite and > 0";
    return false;
  }
  nv_bps_ = t.nvlink_Bps;
  nic_bps_ = t.nic_Bps;
  fab_bps_ = t.fabric_Bps;
  if (t.num_degraded < 0 || (t.num_degraded > 0 && (!t.degraded_cables || !good_rate(t.degraded_Bps)))) {
    *err = "topology: degraded cables need a list and a finite rate > 0";
    return false;
  }
  degraded_.assign(t.degraded_cables, t.degraded_cables + t.num_degraded);
  for (int64_t c : degraded_)
    if (c < 0 || c >= ncab_) {
      *err = "topology: degraded cable id out of range";
      return false;
    }
  deg_bps_ = t.degraded_Bps;
  if (!(t.fabric_latency_s >= 0.0) || !std::isfinite(t.fabric_latency_s) ||
      !(t.nvlink_latency_s >= 0.0) || !std::isfinite(t.nvlink_latency_s)) {
    *err = "topology: latencies must be finite and >= 0";
    return false;
  }
  nv_lat_ = t.nvlink_latency_s;
  fab_lat_ = t.fabric_latency_s;
  key_ = splitmix64(t.ecmp_seed);
  return true;
}

void Fabric::latencies(std::vector<double>* lat) const {
  lat->assign((size_t)L_, fab_lat_);
  for (int64_t l = 0; l < NV_; ++l) (*lat)[(size_t)l] = nv_lat_;
}

void Fabric::capacities(std::vector<double>* cap) const {
  cap->assign((size_t)L_, 0.0);
  for (int64_t l = 0; l < NV_; ++l) (*cap)[l] = nv_bps_;
  for (int64_t c = 0; c < ncab_; ++c) {
    const double r = c < N_ ? nic_bps_ : fab_bps_;
    (*cap)[up(c)] = r;
    (*cap)[down(c)] = r;
  }
  for (int64_t c : degraded_) {
    (*cap)[up(c)] = deg_bps_;
    (*cap)[down(c)] = deg_bps_;
  }
}

int Fabric::route(int64_t src, int64_t dst, int32_t* out) const {
  const int64_t ss = src / G_, sd = dst / G_;
  if (ss == sd) {
    const int64_t i = src % G_, j = dst % G_;
    out[0] = (int32_t)(ss * G_ * (G_ - 1) + i * (G_ - 1) + (j < i ? j : j - 1));
    return 1;
  }
  const uint64_t h = splitmix64(key_ ^ (((uint64_t)src << 32) | (uint64_t)dst));
  if (kind_ == NETSIM_TOPO_LEAF_SPINE || kind_ == NETSIM_TOPO_RAIL) {
    int64_t ls, ld;
    if (kind_ == NETSIM_TOPO_LEAF_SPINE) {
      ls = ss / spl_;
      ld = sd / spl_;
    } else {
      ls = (src % G_) * groups_ + ss / spl_;
      ld = (dst % G_) * groups_ + sd / spl_;
    }
    if (ls == ld) {
      out[0] = (int32_t)up(src);
      out[1] = (int32_t)down(dst);
      return 2;
    }
    const int64_t sp = (int64_t)(h % (uint64_t)spines_);
    out[0] = (int32_t)up(src);
    out[1] = (int32_t)up(N_ + ls * spines_ + sp);
    out[2] = (int32_t)down(N_ + ld * spines_ + sp);
    out[3] = (int32_t)down(dst);
    return 4;
  }
  // fat tree
  const int64_t es = ss / spl_, ed = sd / spl_;  // global edge ids (pod*E + e)
  if (es == ed) {
    out[0] = (int32_t)up(src);
    out[1] = (int32_t)down(dst);
    return 2;
  }
  const int64_t ps = es / E_, pd = ed / E_;
  const int64_t a = (int64_t)(h % (uint64_t)A_);
  const int64_t ea_s = N_ + es * A_ + a;
  const int64_t ea_d = N_ + ed * A_ + a;
  if (ps == pd) {
    out[0] = (int32_t)up(src);
    out[1] = (int32_t)up(ea_s);
    out[2] = (int32_t)down(ea_d);
    out[3] = (int32_t)down(dst);
    return 4;
  }
  const int64_t u = (int64_t)((h / (uint64_t)A_) % (uint64_t)U_);
  const int64_t base = N_ + P_ * E_ * A_;
  out[0] = (int32_t)up(src);
  out[1] = (int32_t)up(ea_s);
  out[2] = (int32_t)up(base + (ps * A_ + a) * U_ + u);
  out[3] = (int32_t)down(base + (pd * A_ + a) * U_ + u);
  out[4] = (int32_t)down(ea_d);
  out[5] = (int32_t)down(dst);
  return 6;
}

}  // namespace netsim_host
