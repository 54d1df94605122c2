// Built-in cluster fabrics and their ECMP router (host side of libnetsim).
//
// The paper's simulator is configured with switch port bandwidths, the
// interconnect and its multipath routing / load-balancing rule (Section
// 4.1, netsim description).  This file implements the three fabrics and the
// link numbering, routes and hash documented in include/netsim.h.
#pragma once

#include <stdint.h>

#include <string>
#include <vector>

#include "netsim.h"

namespace netsim_host {

inline uint64_t splitmix64(uint64_t x) {
  uint64_t z = x + 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

class Fabric {
 public:
  // Validates the description; on failure returns false with a message.
  bool init(const netsim_topology& t, std::string* err);
  int64_t num_links() const { return L_; }
  int64_t endpoints() const { return N_; }
  int64_t num_cables() const { return ncab_; }
  void capacities(std::vector<double>* cap) const;
  // Per link: nvlink latency for intra-server links, fabric latency for cables.
  void latencies(std::vector<double>* lat) const;
  // Writes the route of src -> dst (src != dst, both in [0, N)) into out[0..6)
  // and returns its length.
  int route(int64_t src, int64_t dst, int32_t* out) const;
  static constexpr int kMaxHops = 6;

 private:
  int64_t up(int64_t cable) const { return NV_ + 2 * cable; }
  int64_t down(int64_t cable) const { return NV_ + 2 * cable + 1; }
  int32_t kind_ = 0;
  int64_t S_ = 0, G_ = 0, N_ = 0, NV_ = 0, spl_ = 1, spines_ = 0;
  int64_t P_ = 0, E_ = 0, A_ = 0, U_ = 0, groups_ = 0, leaves_ = 0, ncab_ = 0, L_ = 0;
  uint64_t key_ = 0;
  double nv_bps_ = 0, nic_bps_ = 0, fab_bps_ = 0, deg_bps_ = 0;
  double nv_lat_ = 0, fab_lat_ = 0;
  std::vector<int64_t> degraded_;
};

}  // namespace netsim_host
