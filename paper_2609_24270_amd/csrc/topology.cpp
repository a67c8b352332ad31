// Topology map: compute-unit identity records -> dense CU map, invariants,
// CU sets.
//
// Section 5.1 recovers which logical units share a physical cluster and
// Section 5.2 shows the layout differs per chip, so the map is measured on
// every chip rather than looked up.  On gfx950 a workgroup can read its own
// XCC id and the SE / shader-array / CU fields of the HW_ID register, so the
// map is the set of distinct (xcc, se, sh, cu) tuples the hardware reports,
// in sorted order.  Appendix G groups XCDs by memory affinity; the groups are
// filled in by the latency probe.
#include <algorithm>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <set>
#include <tuple>

#include "internal.h"

namespace asym {

int build_topology(const int32_t* rec, int n, int n_cus_expected,
                   int n_xccs_expected, const int32_t* mask_bit_record,
                   Topology& out) {
  if (!rec || n < 1) return fail(ASYM_EINVAL, "topology: no records");
  if (n_cus_expected < 1 || n_cus_expected > ASYM_MAX_CUS)
    return fail(ASYM_EINVAL, "topology: bad expected CU count");
  if (n_xccs_expected < 1 || n_xccs_expected > ASYM_MAX_XCDS)
    return fail(ASYM_EINVAL, "topology: bad expected XCC count");
  using Key = std::tuple<int, int, int, int>;
  std::set<Key> seen;
  std::vector<Key> keyof(n);
  for (int i = 0; i < n; ++i) {
    const uint32_t x = (uint32_t)rec[4 * i + 0], h = (uint32_t)rec[4 * i + 1];
    keyof[i] = Key(xccid(x), hwid_se(h), hwid_sh(h), hwid_cu(h));
    seen.insert(keyof[i]);
  }
  Topology t;
  t.n_xccs = n_xccs_expected;
  t.n_cus = (int)seen.size();
  std::map<Key, int> dense;
  for (const Key& k : seen) {
    const int idx = (int)t.cus.size();
    dense[k] = idx;
    t.cus.push_back(CuRecord{std::get<0>(k), std::get<1>(k), std::get<2>(k),
                             std::get<3>(k), -1});
  }
  t.cus_per_xcd.assign(n_xccs_expected, 0);
  for (const CuRecord& c : t.cus) {
    if (c.xcc >= n_xccs_expected)
      return fail(ASYM_EINVARIANT, "topology: XCC id " + std::to_string(c.xcc) +
                                       " >= device XCC count " +
                                       std::to_string(n_xccs_expected));
    t.cus_per_xcd[c.xcc] += 1;
  }
  t.bit_to_cu.assign(n_cus_expected, -1);
  if (mask_bit_record) {
    t.has_maskmap = true;
    for (int b = 0; b < n_cus_expected; ++b) {
      const int r = mask_bit_record[b];
      if (r < 0 || r >= n) {
        t.has_maskmap = false;
        continue;
      }
      const int cu = dense[keyof[r]];
      t.bit_to_cu[b] = cu;
      t.cus[cu].mask_bit = b;
    }
  }
  // dispatch: how consistently each residue class of block indices (mod the
  // XCD count) sits on one XCD
  {
    std::vector<int> blk(n), xs(n);
    for (int i = 0; i < n; ++i) {
      blk[i] = rec[4 * i + 2];
      xs[i] = xccid((uint32_t)rec[4 * i]);
    }
    int rot = 0;
    dispatch_stats(blk.data(), xs.data(), n, n_xccs_expected, &t.rr_fraction, &rot);
  }
  // invariants against the device's own counts
  if (t.n_cus != n_cus_expected)
    return fail(ASYM_EINVARIANT, "topology: found " + std::to_string(t.n_cus) +
                                     " distinct CUs, device reports " +
                                     std::to_string(n_cus_expected));
  int rc = check_invariants(t);
  if (rc != ASYM_OK) return rc;
  out = std::move(t);
  return ASYM_OK;
}

int check_invariants(const Topology& t) {
  if (t.n_cus != (int)t.cus.size()) return fail(ASYM_EINVARIANT, "topology: CU count mismatch");
  std::set<std::tuple<int, int, int, int>> s;
  int sum = 0;
  for (const CuRecord& c : t.cus)
    if (!s.insert(std::make_tuple(c.xcc, c.se, c.sh, c.cu)).second)
      return fail(ASYM_EINVARIANT, "topology: duplicate CU record");
  for (int x = 0; x < t.n_xccs; ++x) {
    if (t.cus_per_xcd[x] < 1)
      return fail(ASYM_EINVARIANT, "topology: XCC " + std::to_string(x) + " has no CU");
    sum += t.cus_per_xcd[x];
  }
  if (sum != t.n_cus) return fail(ASYM_EINVARIANT, "topology: per-XCD counts do not sum to the CU count");
  if (t.has_maskmap) {
    std::vector<int> hit(t.n_cus, 0);
    for (int b = 0; b < t.n_cus; ++b) {
      const int cu = t.bit_to_cu[b];
      if (cu < 0 || cu >= t.n_cus || hit[cu]++)
        return fail(ASYM_EINVARIANT, "topology: mask-bit map is not a bijection");
    }
  }
  return ASYM_OK;
}

int mask_counts(const Topology& t, const uint32_t* mask, std::vector<int>& per) {
  per.assign(t.n_xccs, 0);
  int pop = 0;
  for (int b = 0; b < ASYM_MAX_CUS; ++b) {
    if (!((mask[b >> 5] >> (b & 31)) & 1u)) continue;
    if (b >= t.n_cus) return fail(ASYM_EINVAL, "mask: bit " + std::to_string(b) + " beyond the CU count");
    ++pop;
  }
  if (pop == t.n_cus) {
    per = t.cus_per_xcd;
    return ASYM_OK;
  }
  if (!t.has_maskmap)
    return fail(ASYM_EUNSUPPORTED, "mask: a partial CU mask needs a topology probed with ASYM_PROBE_MASKMAP");
  for (int b = 0; b < t.n_cus; ++b)
    if ((mask[b >> 5] >> (b & 31)) & 1u) per[t.cus[t.bit_to_cu[b]].xcc] += 1;
  return ASYM_OK;
}

// splitmix64 (Steele, Lea, Flood 2014), for seeded CU choices
static uint64_t splitmix64(uint64_t& s) {
  uint64_t z = (s += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

static int cuset_make(const Topology& t, int n, int policy, uint64_t seed,
                      const uint32_t* exclude, uint32_t* mask_out) {
  if (!t.has_maskmap) return fail(ASYM_EUNSUPPORTED, "cuset: needs a topology probed with ASYM_PROBE_MASKMAP");
  if (n < 1 || n > t.n_cus) return fail(ASYM_EINVAL, "cuset: bad CU count");
  std::vector<char> freecu(t.n_cus, 1);
  if (exclude)
    for (int b = 0; b < t.n_cus; ++b)
      if ((exclude[b >> 5] >> (b & 31)) & 1u) freecu[t.bit_to_cu[b]] = 0;
  std::vector<int> chosen;
  if (policy == ASYM_CUSET_XCD_ALIGNED || policy == ASYM_CUSET_AFFINITY_ALIGNED) {
    std::vector<int> xorder;
    for (int x = 0; x < t.n_xccs; ++x) xorder.push_back(x);
    if (policy == ASYM_CUSET_AFFINITY_ALIGNED && t.has_latency) {
      std::stable_sort(xorder.begin(), xorder.end(), [&](int a, int b) {
        return t.lat.group_of_xcd[a] < t.lat.group_of_xcd[b];
      });
    }
    int got = 0;
    for (int x : xorder) {
      if (got >= n) break;
      bool whole = true;
      for (int c = 0; c < t.n_cus; ++c)
        if (t.cus[c].xcc == x && !freecu[c]) whole = false;
      if (!whole) continue;
      if (got + t.cus_per_xcd[x] > n) continue;
      for (int c = 0; c < t.n_cus; ++c)
        if (t.cus[c].xcc == x) chosen.push_back(c);
      got += t.cus_per_xcd[x];
    }
    if (got != n) return fail(ASYM_EINVAL, "cuset: " + std::to_string(n) + " CUs are not a union of free whole XCDs");
  } else if (policy == ASYM_CUSET_STRIPED) {
    // the same share of every XCD (remainder to the lower XCDs), and within
    // an XCD round-robin over shader engines, lowest CU first
    std::vector<int> share = largest_remainder_quotas(n, t.cus_per_xcd);
    for (int x = 0; x < t.n_xccs; ++x) {
      std::map<int, std::vector<int>> by_se;
      for (int c = 0; c < t.n_cus; ++c)
        if (t.cus[c].xcc == x && freecu[c]) by_se[t.cus[c].se * 2 + t.cus[c].sh].push_back(c);
      int need = share[x];
      size_t depth = 0;
      bool progress = true;
      while (need > 0 && progress) {
        progress = false;
        for (auto& kv : by_se) {
          if (need == 0) break;
          if (depth < kv.second.size()) {
            chosen.push_back(kv.second[depth]);
            --need;
            progress = true;
          }
        }
        ++depth;
      }
      if (need > 0) return fail(ASYM_EINVAL, "cuset: not enough free CUs on XCC " + std::to_string(x));
    }
  } else if (policy == ASYM_CUSET_RANDOM) {
    std::vector<int> pool;
    for (int c = 0; c < t.n_cus; ++c)
      if (freecu[c]) pool.push_back(c);
    if ((int)pool.size() < n) return fail(ASYM_EINVAL, "cuset: not enough free CUs");
    uint64_t st = seed;
    for (int i = (int)pool.size() - 1; i > 0; --i) {
      const int j = (int)(splitmix64(st) % (uint64_t)(i + 1));
      std::swap(pool[i], pool[j]);
    }
    chosen.assign(pool.begin(), pool.begin() + n);
  } else {
    return fail(ASYM_EINVAL, "cuset: unknown policy");
  }
  std::memset(mask_out, 0, sizeof(uint32_t) * ASYM_MASK_WORDS);
  for (int c : chosen) {
    const int b = t.cus[c].mask_bit;
    mask_out[b >> 5] |= 1u << (b & 31);
  }
  return ASYM_OK;
}

static std::string topology_json(const Topology& t) {
  std::string s = "{";
  char buf[256];
  std::snprintf(buf, sizeof buf, "\"device\": %d, \"n_cus\": %d, \"n_xccs\": %d, \"rr_fraction\": %.6f, ",
                t.device, t.n_cus, t.n_xccs, t.rr_fraction);
  s += buf;
  s += "\"cus_per_xcd\": [";
  for (int x = 0; x < t.n_xccs; ++x) s += (x ? ", " : "") + std::to_string(t.cus_per_xcd[x]);
  s += "], \"has_maskmap\": ";
  s += t.has_maskmap ? "true" : "false";
  s += ", \"probes\": " + std::to_string(t.flags);
  s += ", \"compute_partition\": \"" + t.compute_partition + "\", \"memory_partition\": \"" +
       t.memory_partition + "\"";
  std::string k;  // the key as a JSON string (it holds no quote or backslash, but escape anyway)
  for (char c : t.key) {
    if (c == '"' || c == '\\') k += '\\';
    k += c;
  }
  s += ", \"key\": \"" + k + "\"";
  s += ", \"cus\": [";
  for (size_t i = 0; i < t.cus.size(); ++i) {
    const CuRecord& c = t.cus[i];
    std::snprintf(buf, sizeof buf, "%s[%d, %d, %d, %d, %d]", i ? ", " : "", c.xcc, c.se, c.sh, c.cu, c.mask_bit);
    s += buf;
  }
  s += "]";
  if (t.has_latency) {
    const asym_latency_summary& L = t.lat;
    auto arr = [&](const double* v) {
      std::string a = "[";
      for (int x = 0; x < L.n_xcds; ++x) {
        std::snprintf(buf, sizeof buf, "%s%.2f", x ? ", " : "", v[x]);
        a += buf;
      }
      return a + "]";
    };
    s += ", \"latency\": {\"n_samples\": " + std::to_string(L.n_samples) +
         ", \"passes\": " + std::to_string(L.passes) + ", \"l2_samples\": " + std::to_string(L.l2_samples);
    std::snprintf(buf, sizeof buf, ", \"timer_overhead\": %.1f, \"clock_mhz\": %.1f, \"unclassified_share\": %.4f",
                  L.timer_overhead, L.clock_mhz, L.unclassified_share);
    s += buf;
    s += ", \"l2_hit\": " + arr(L.l2_hit) + ", \"mall_hit\": " + arr(L.mall_hit) + ", \"hbm\": " + arr(L.hbm);
    s += ", \"group_of_xcd\": [";
    for (int x = 0; x < L.n_xcds; ++x) s += (x ? ", " : "") + std::to_string(L.group_of_xcd[x]);
    s += "], \"n_groups\": " + std::to_string(L.n_groups);
    s += ", \"home_share\": [";
    for (int g = 0; g < L.n_groups; ++g) {
      std::snprintf(buf, sizeof buf, "%s%.4f", g ? ", " : "", L.home_share[g]);
      s += buf;
    }
    s += "], \"hbm_by_home\": [";
    for (int x = 0; x < L.n_xcds; ++x) {
      s += x ? ", [" : "[";
      for (int g = 0; g < L.n_groups; ++g) {
        std::snprintf(buf, sizeof buf, "%s%.2f", g ? ", " : "", L.hbm_by_home[x][g]);
        s += buf;
      }
      s += "]";
    }
    s += "]}";
  }
  s += "}";
  return s;
}

void dispatch_stats(const int* block, const int* xcc, int n, int n_x, double* class_fraction, int* rotation) {
  if (n < 1 || n_x < 1) {
    *class_fraction = 0.0;
    *rotation = 0;
    return;
  }
  std::vector<std::vector<int>> cnt(n_x, std::vector<int>(ASYM_MAX_XCDS, 0));
  std::vector<int> rot(n_x, 0);
  for (int i = 0; i < n; ++i) {
    const int x = xcc[i], b = block[i];
    if (x < 0 || x >= ASYM_MAX_XCDS || b < 0) continue;
    cnt[b % n_x][x] += 1;
    if (x < n_x) rot[((x - b % n_x) % n_x + n_x) % n_x] += 1;
  }
  int best = 0;
  for (int r = 0; r < n_x; ++r) best += *std::max_element(cnt[r].begin(), cnt[r].end());
  *class_fraction = (double)best / n;
  *rotation = (int)(std::max_element(rot.begin(), rot.end()) - rot.begin());
}

}  // namespace asym

struct asym_topology {
  asym::Topology t;
};

using asym::fail;

extern "C" int asym_topology_from_records(const int32_t* records, int n_records,
                                          int n_cus_expected, int n_xccs_expected,
                                          const int32_t* mask_bit_record,
                                          asym_topology** out) {
  if (!out) return fail(ASYM_EINVAL, "null out");
  *out = nullptr;
  asym::Topology t;
  int rc = asym::build_topology(records, n_records, n_cus_expected, n_xccs_expected,
                                mask_bit_record, t);
  if (rc != ASYM_OK) return rc;
  t.flags = ASYM_PROBE_IDENTITY | (mask_bit_record ? ASYM_PROBE_MASKMAP : 0u);
  t.key = "records";
  *out = new asym_topology{std::move(t)};
  return ASYM_OK;
}

namespace asym {
asym_topology* wrap_topology(Topology&& t) { return new asym_topology{std::move(t)}; }
const Topology* unwrap(const asym_topology* p) { return p ? &p->t : nullptr; }
}  // namespace asym

extern "C" void asym_topology_free(asym_topology* topo) { delete topo; }

extern "C" int asym_topology_info(const asym_topology* topo, int* n_cus, int* n_xcds,
                                  int* cus_per_xcd, int* group_of_xcd) {
  if (!topo) return fail(ASYM_EINVAL, "null topology");
  const asym::Topology& t = topo->t;
  if (n_cus) *n_cus = t.n_cus;
  if (n_xcds) *n_xcds = t.n_xccs;
  for (int x = 0; x < ASYM_MAX_XCDS; ++x) {
    if (cus_per_xcd) cus_per_xcd[x] = x < t.n_xccs ? t.cus_per_xcd[x] : 0;
    if (group_of_xcd) group_of_xcd[x] = (t.has_latency && x < t.n_xccs) ? t.lat.group_of_xcd[x] : -1;
  }
  return ASYM_OK;
}

extern "C" int asym_topology_cu(const asym_topology* topo, int cu_index, int* xcc,
                                int* se, int* sh, int* cu, int* mask_bit) {
  if (!topo) return fail(ASYM_EINVAL, "null topology");
  const asym::Topology& t = topo->t;
  if (cu_index < 0 || cu_index >= t.n_cus) return fail(ASYM_EINVAL, "CU index out of range");
  const asym::CuRecord& c = t.cus[cu_index];
  if (xcc) *xcc = c.xcc;
  if (se) *se = c.se;
  if (sh) *sh = c.sh;
  if (cu) *cu = c.cu;
  if (mask_bit) *mask_bit = c.mask_bit;
  return ASYM_OK;
}

extern "C" int asym_topology_dispatch(const asym_topology* topo, double* rr_fraction) {
  if (!topo || !rr_fraction) return fail(ASYM_EINVAL, "null argument");
  *rr_fraction = topo->t.rr_fraction;
  return ASYM_OK;
}

extern "C" int asym_topology_latency(const asym_topology* topo, asym_latency_summary* out) {
  if (!topo || !out) return fail(ASYM_EINVAL, "null argument");
  if (!topo->t.has_latency) return fail(ASYM_EUNSUPPORTED, "topology was probed without ASYM_PROBE_LATENCY");
  *out = topo->t.lat;
  return ASYM_OK;
}

extern "C" int asym_topology_json(const asym_topology* topo, char* buf, size_t len,
                                  size_t* needed) {
  if (!topo) return fail(ASYM_EINVAL, "null topology");
  const std::string s = asym::topology_json(topo->t);
  if (needed) *needed = s.size() + 1;
  if (!buf || len < s.size() + 1) return fail(ASYM_EINVAL, "buffer too small");
  std::memcpy(buf, s.c_str(), s.size() + 1);
  return ASYM_OK;
}

extern "C" int asym_cuset_make(const asym_topology* topo, int n_cus, int policy,
                               uint64_t seed, const uint32_t* exclude, uint32_t* mask_out) {
  if (!topo || !mask_out) return fail(ASYM_EINVAL, "null argument");
  return asym::cuset_make(topo->t, n_cus, policy, seed, exclude, mask_out);
}

extern "C" int asym_cuset_counts(const asym_topology* topo, const uint32_t* mask, int* per_xcd) {
  if (!topo || !mask || !per_xcd) return fail(ASYM_EINVAL, "null argument");
  std::vector<int> per;
  int rc = asym::mask_counts(topo->t, mask, per);
  if (rc != ASYM_OK) return rc;
  for (int x = 0; x < ASYM_MAX_XCDS; ++x) per_xcd[x] = x < (int)per.size() ? per[x] : 0;
  return ASYM_OK;
}

// Two tenants on disjoint whole-XCD sides.  Workgroups are dealt to every XCD
// in turn whatever the stream's CU mask, so a tenant whose mask left an XCD
// empty could never run the workgroups dealt there, and a tenant whose
// workgroups had to wait for a CU held by the other side's persistent kernel
// would stall its own dispatch.  So each side gives the other one CU (its
// lowest) on each of its XCDs: the other tenant's workgroups that land there
// find a free CU and leave at once (xcd_mask restricts the work to the
// tenant's own XCDs).
extern "C" int asym_cuset_split_xcds(const asym_topology* topo, uint32_t xcd_mask_a,
                                     uint32_t* mask_a, uint32_t* mask_b) {
  using namespace asym;
  if (!topo || !mask_a || !mask_b) return fail(ASYM_EINVAL, "null argument");
  const Topology& t = topo->t;
  if (!t.has_maskmap) return fail(ASYM_EUNSUPPORTED, "cuset split: needs a topology with a mask map");
  const uint32_t all = t.n_xccs >= 32 ? 0xFFFFFFFFu : ((1u << t.n_xccs) - 1u);
  if ((xcd_mask_a & ~all) || (xcd_mask_a & all) == 0 || (xcd_mask_a & all) == all)
    return fail(ASYM_EINVAL, "cuset split: side A must name some but not all XCDs");
  std::memset(mask_a, 0, sizeof(uint32_t) * ASYM_MASK_WORDS);
  std::memset(mask_b, 0, sizeof(uint32_t) * ASYM_MASK_WORDS);
  std::vector<int> bit_of(t.n_cus, -1);
  for (int b = 0; b < (int)t.bit_to_cu.size(); ++b)
    if (t.bit_to_cu[b] >= 0) bit_of[t.bit_to_cu[b]] = b;
  std::vector<bool> first_seen(t.n_xccs, false);
  for (int c = 0; c < t.n_cus; ++c) {  // dense order: each XCD's lowest CU comes first
    const int x = t.cus[c].xcc, b = bit_of[c];
    if (b < 0) return fail(ASYM_EINVAL, "cuset split: mask map incomplete");
    const bool side_a = (xcd_mask_a >> x) & 1u;
    const bool give = !first_seen[x];
    first_seen[x] = true;
    uint32_t* m = (side_a != give) ? mask_a : mask_b;
    m[b >> 5] |= 1u << (b & 31);
  }
  return ASYM_OK;
}
