// Host model of the index arithmetic of the default solver's one-workgroup
// rate solve (kernels.hip: solve_mask and for_items -- the gather of ids and
// path records into the shared-memory cache or the staging buffer, the two
// phases of every freezing round over the items of a thread's unfrozen mask,
// the write-back of rates and slots), templated on the number of path
// records a thread keeps in flight (D; the kernel uses 4), with every array
// access bounds-checked.  One workgroup of T threads is run thread by thread
// per phase; link ids, masks and cache sizes follow the kernel's rules.  Run
// under AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/test_native_checks.py over re-solve sizes of the 4096-GPU workload.
#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

static long g_checks = 0;
template <class V>
struct Checked {
  std::vector<V> v;
  const char* name;
  Checked(size_t n, const char* nm) : v(n), name(nm) {}
  V& operator[](long i) {
    ++g_checks;
    if (i < 0 || (size_t)i >= v.size()) {
      std::fprintf(stderr, "OUT OF BOUNDS %s[%ld] size %zu\n", name, i, v.size());
      std::abort();
    }
    return v[(size_t)i];
  }
};
struct U4 { uint32_t x, y, z, w; };

static uint64_t low_items(int n, int T, int t) {
  const int c = n > t ? (n - t - 1) / T + 1 : 0;
  return c >= 64 ? ~0ull : (1ull << c) - 1ull;
}
static int ffsll(uint64_t m) { return m ? __builtin_ctzll(m) + 1 : 0; }

// for_items of the kernel, depth D
template <int D, class Body>
static void for_items(int t, uint64_t mask, uint64_t cmask, Checked<U4>& cache, Checked<U4>& stg, int T, Body body) {
  for (uint64_t m = mask & cmask; m;) {
    int k[D]; U4 r[D];
    for (int u = 0; u < D; ++u) {
      k[u] = m ? ffsll(m) - 1 : -1;
      m &= m - 1;
      if (k[u] >= 0) r[u] = cache[t + k[u] * T];
    }
    for (int u = 0; u < D; ++u) if (k[u] >= 0) body(k[u], t + k[u] * T, true, r[u]);
  }
  for (uint64_t m = mask & ~cmask; m;) {
    int k[D]; U4 r[D];
    for (int u = 0; u < D; ++u) {
      k[u] = m ? ffsll(m) - 1 : -1;
      m &= m - 1;
      if (k[u] >= 0) r[u] = stg[t + k[u] * T];
    }
    for (int u = 0; u < D; ++u) if (k[u] >= 0) body(k[u], t + k[u] * T, false, r[u]);
  }
}

static int unpack(const U4& rec, int l0, int* lv) {
  const uint32_t w[3] = {rec.x, rec.y, rec.z};
  int deg = 0;
  for (int k = 0; k < 6; ++k) {
    const uint32_t u = (w[k >> 1] >> (16 * (k & 1))) & 0xFFFFu;
    lv[k] = l0 + (int)u;
    deg += u != 0xFFFFu;
  }
  return deg;
}

template <int D>
static void run(int T, int n, int ccap, int nl, int cap, uint32_t seed) {
  std::mt19937 rng(seed);
  const int f0 = 0, l0 = 0, lsent = l0 + nl;
  // part: cap flows, nl links (+ sentinel); a re-solve of n flows in slots
  Checked<int32_t> list(cap, "list"), at(cap, "rs.at"), slot_id(cap, "slot.id");
  Checked<U4> path16(cap, "path16"), stage(cap, "stage"), cache(ccap > 0 ? ccap : 1, "fc.path");
  Checked<int32_t> fid(ccap > 0 ? ccap : 1, "fc.fid");
  Checked<double> mf(cap, "mf"), rem(cap, "rem"), tref(cap, "tref"), rate(cap, "rate"), srate(cap, "slot.rate"), tau(cap, "slot.tau");
  Checked<double> table(nl + 2, "share table");
  Checked<uint32_t> stamp(nl + 2, "stamp");
  Checked<int64_t> R(nl + 2, "R"), N(nl + 2, "n");
  std::vector<int> perm(cap);
  for (int i = 0; i < cap; ++i) perm[i] = i;
  std::shuffle(perm.begin(), perm.end(), rng);
  for (int i = 0; i < cap; ++i) {
    // a path of 1..6 distinct part-local links, packed first, 0xFFFF after
    uint16_t ids[6];
    const int deg = 1 + (int)(rng() % 6);
    for (int k = 0; k < 6; ++k) ids[k] = k < deg ? (uint16_t)(rng() % nl) : 0xFFFF;
    path16[i] = U4{ids[0] | (uint32_t)ids[1] << 16, ids[2] | (uint32_t)ids[3] << 16, ids[4] | (uint32_t)ids[5] << 16, 0};
  }
  for (int i = 0; i < n; ++i) { list[i] = perm[i]; at[i] = (int)(rng() % cap); }
  const int nc = n < ccap ? n : ccap;
  // gather (depth D)
  for (int t = 0; t < T; ++t)
    for (int j0 = 0; j0 * T < n; j0 += D)
      for (int u = 0; u < D; ++u) {
        const int i = t + (j0 + u) * T;
        if (i >= n) continue;
        const int f = list[i];
        const U4 rv = path16[f - f0 >= 0 && f - f0 < cap ? f : f0];
        (void)at[i];
        if (i < nc) { fid[i] = f; cache[i] = rv; } else { stage[i] = rv; }
        int lv[6];
        const int deg = unpack(rv, l0, lv);
        for (int j = 0; j < 6; ++j) if (j < deg) { R[lv[j] - l0] += 1; N[lv[j] - l0] += 1; }
      }
  table[nl] = 1e300; stamp[nl] = 0;
  // rounds: random freezing until everything is frozen
  std::vector<uint64_t> alive(T);
  for (int t = 0; t < T; ++t) alive[t] = low_items(n, T, t);
  for (int r = 0; r < 200; ++r) {
    bool any = false;
    for (int t = 0; t < T; ++t) {
      const uint64_t cmask = low_items(nc, T, t);
      // phase B
      for_items<D>(t, alive[t], cmask, cache, stage, T, [&](int, int i, bool cached, U4 rec) {
        int lv[6];
        unpack(rec, l0, lv);
        for (int k = 0; k < 6; ++k) { lv[k] = lv[k] < lsent ? lv[k] : lsent; (void)table[lv[k] - l0]; }
        stamp[lv[0] - l0] = (uint32_t)r;
        if (cached) cache[i].w = 1; else stage[i].w = 1;
      });
      // phase C: freeze a random subset
      uint64_t frozen = 0;
      for_items<D>(t, alive[t], cmask, cache, stage, T, [&](int k, int i, bool, U4 rec) {
        if (rng() % 3) return;
        int lv[6];
        const int deg = unpack(rec, l0, lv);
        for (int j = 0; j < 6; ++j) if (j < deg) { (void)stamp[lv[j] - l0]; (void)table[lv[j] - l0]; R[lv[j] - l0] -= 1; N[lv[j] - l0] -= 1; }
        mf[i] = 1.0;
        frozen |= 1ull << k;
      });
      alive[t] &= ~frozen;
      any |= alive[t] != 0;
    }
    if (!any) break;
  }
  // write-back (depth D): rates by flow, slots
  for (int t = 0; t < T; ++t)
    for (int j0 = 0; j0 * T < n; j0 += D)
      for (int u = 0; u < D; ++u) {
        const int i = t + (j0 + u) * T;
        if (i >= n) continue;
        const int f = i < nc ? fid[i] : list[i];
        const double mv = mf[i];
        const int s = at[i];
        rate[f] = mv; srate[s] = mv; tau[s] = 1.0 / (mv + rem[f] + tref[f]);
      }
}

template <int D>
static void sweep_sizes() {
  long cases = 0;
  for (int T : {512, 1024})
    for (int ccap : {4195, 7782, 0})
      for (int n : {1, 2, 63, 64, 65, T - 1, T, T + 1, 4 * T - 1, 4 * T, 4 * T + 1, 5 * T + 3, 4195, 4196,
                    7782, 7783, 16383, 16384, 32256, 32767, 63 * T + 17, 64 * T}) {
        if (n > 64 * T) continue;
        const int cap = n + 17;  // the part's flows (>= the re-solve)
        run<D>(T, n, ccap, 2560, cap, (uint32_t)(n * 131 + T + ccap + D));
        ++cases;
      }
  std::printf("depth %d: %ld cases, in bounds\n", D, cases);
}

int main() {
  sweep_sizes<1>(); sweep_sizes<2>(); sweep_sizes<3>(); sweep_sizes<4>();
  sweep_sizes<5>(); sweep_sizes<6>(); sweep_sizes<7>(); sweep_sizes<8>();
  std::printf("%ld bounds-checked accesses\n", g_checks);
  return 0;
}
