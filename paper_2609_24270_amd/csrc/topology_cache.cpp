// Per-chip topology cache.  Section 5.2 finds that the unit-to-partition map
// differs between chips of one product, so a probe result belongs to one chip
// in one configuration: the cache key names the PCI function, the device UUID,
// the runtime and driver versions, the architecture, the compute and memory
// partition modes and the CU / XCD counts, and a cached map is used only under
// the same key.  The file is plain text:
//
//   asym-topology 1
//   key <one line>
//   flags <probes made>
//   counts <n_cus> <n_xccs> <has_maskmap> <rr_fraction>
//   partitions <compute> <memory>
//   cu <xcc> <se> <sh> <cu> <mask_bit>          (n_cus lines, dense order)
//   latency <values>                            (only with a latency probe)
//   end
//
// Loading rebuilds the per-XCD counts and the mask map from the CU lines and
// checks the exact invariants again, so a damaged file is rejected, not used.
#include <hip/hip_runtime.h>

#include <cctype>
#include <cstdio>
#include <cstring>
#include <fstream>
#include <sstream>

#include "internal.h"

struct asym_topology;
namespace asym {
asym_topology* wrap_topology(Topology&& t);
const Topology* unwrap(const asym_topology* p);

namespace {

constexpr const char* kMagic = "asym-topology 1";

// The latency summary as a flat list of numbers, in declaration order.
std::vector<double> latency_values(const asym_latency_summary& L) {
  std::vector<double> v = {(double)L.n_xcds, (double)L.n_samples, (double)L.passes, (double)L.l2_samples,
                           L.timer_overhead, L.clock_mhz};
  for (int x = 0; x < ASYM_MAX_XCDS; ++x) v.push_back(L.l2_hit[x]);
  for (int x = 0; x < ASYM_MAX_XCDS; ++x) v.push_back(L.mall_hit[x]);
  for (int x = 0; x < ASYM_MAX_XCDS; ++x) v.push_back(L.hbm[x]);
  for (int x = 0; x < ASYM_MAX_XCDS; ++x) v.push_back((double)L.group_of_xcd[x]);
  v.push_back((double)L.n_groups);
  for (int x = 0; x < ASYM_MAX_XCDS; ++x) v.push_back(L.home_share[x]);
  v.push_back(L.unclassified_share);
  for (int x = 0; x < ASYM_MAX_XCDS; ++x)
    for (int y = 0; y < ASYM_MAX_XCDS; ++y) v.push_back(L.corr[x][y]);
  for (int x = 0; x < ASYM_MAX_XCDS; ++x)
    for (int y = 0; y < ASYM_MAX_XCDS; ++y) v.push_back(L.hbm_by_home[x][y]);
  return v;
}

bool latency_from_values(const std::vector<double>& v, asym_latency_summary& L) {
  const size_t want = latency_values(asym_latency_summary{}).size();
  if (v.size() != want) return false;
  size_t i = 0;
  L = asym_latency_summary{};
  L.n_xcds = (int)v[i++];
  L.n_samples = (int)v[i++];
  L.passes = (int)v[i++];
  L.l2_samples = (int)v[i++];
  L.timer_overhead = v[i++];
  L.clock_mhz = v[i++];
  for (int x = 0; x < ASYM_MAX_XCDS; ++x) L.l2_hit[x] = v[i++];
  for (int x = 0; x < ASYM_MAX_XCDS; ++x) L.mall_hit[x] = v[i++];
  for (int x = 0; x < ASYM_MAX_XCDS; ++x) L.hbm[x] = v[i++];
  for (int x = 0; x < ASYM_MAX_XCDS; ++x) L.group_of_xcd[x] = (int)v[i++];
  L.n_groups = (int)v[i++];
  for (int x = 0; x < ASYM_MAX_XCDS; ++x) L.home_share[x] = v[i++];
  L.unclassified_share = v[i++];
  for (int x = 0; x < ASYM_MAX_XCDS; ++x)
    for (int y = 0; y < ASYM_MAX_XCDS; ++y) L.corr[x][y] = v[i++];
  for (int x = 0; x < ASYM_MAX_XCDS; ++x)
    for (int y = 0; y < ASYM_MAX_XCDS; ++y) L.hbm_by_home[x][y] = v[i++];
  return L.n_xcds >= 1 && L.n_xcds <= ASYM_MAX_XCDS && L.n_groups >= 0 && L.n_groups <= ASYM_MAX_XCDS;
}

bool one_word(const std::string& s) {
  if (s.empty() || s.size() > 15) return false;
  for (char c : s)
    if (!std::isgraph((unsigned char)c)) return false;
  return true;
}

std::string sysfs_word(const std::string& path) {
  std::ifstream f(path);
  std::string w;
  if (!(f >> w) || !one_word(w)) return "unknown";
  return w;
}

int nocache(const std::string& why) { return fail(ASYM_ENOCACHE, "topology cache: " + why); }

}  // namespace

int device_key(int device, std::string* key, asym_device_info* info_out) {
  asym_device_info info;
  int rc = asym_device_query(device, &info);
  if (rc != ASYM_OK) return rc;
  std::ostringstream k;
  k << "pci=" << info.pci_bus_id << " uuid=" << info.uuid << " hip=" << info.runtime_version
    << " driver=" << info.driver_version << " arch=" << info.arch << " compute=" << info.compute_partition
    << " memory=" << info.memory_partition << " cus=" << info.n_cus << " xccs=" << info.n_xccs;
  if (key) *key = k.str();
  if (info_out) *info_out = info;
  return ASYM_OK;
}

int read_partition_modes(const char* pci_bus_id, char* compute, char* memory, size_t len) {
  const std::string dir = std::string("/sys/bus/pci/devices/") + pci_bus_id + "/";
  const std::string c = sysfs_word(dir + "current_compute_partition");
  const std::string m = sysfs_word(dir + "current_memory_partition");
  std::snprintf(compute, len, "%s", c.c_str());
  std::snprintf(memory, len, "%s", m.c_str());
  return ASYM_OK;
}

int topology_save(const Topology& t, const char* path) {
  if (!path || !*path) return fail(ASYM_EINVAL, "topology cache: empty path");
  if (t.key.find('\n') != std::string::npos) return fail(ASYM_EINVAL, "topology cache: key holds a newline");
  std::ostringstream o;
  o.precision(17);
  o << kMagic << "\n";
  o << "key " << t.key << "\n";
  o << "flags " << t.flags << "\n";
  o << "counts " << t.n_cus << " " << t.n_xccs << " " << (t.has_maskmap ? 1 : 0) << " " << t.rr_fraction << "\n";
  o << "partitions " << (one_word(t.compute_partition) ? t.compute_partition : "unknown") << " "
    << (one_word(t.memory_partition) ? t.memory_partition : "unknown") << "\n";
  for (const CuRecord& c : t.cus)
    o << "cu " << c.xcc << " " << c.se << " " << c.sh << " " << c.cu << " " << c.mask_bit << "\n";
  if (t.has_latency) {
    o << "latency";
    for (double v : latency_values(t.lat)) o << " " << v;
    o << "\n";
  }
  o << "end\n";
  const std::string tmp = std::string(path) + ".tmp";
  {
    std::ofstream f(tmp, std::ios::trunc);
    if (!f) return fail(ASYM_EINVAL, std::string("topology cache: cannot write ") + tmp);
    f << o.str();
    if (!f.flush()) return fail(ASYM_EINVAL, std::string("topology cache: write failed: ") + tmp);
  }
  if (std::rename(tmp.c_str(), path) != 0) {
    std::remove(tmp.c_str());
    return fail(ASYM_EINVAL, std::string("topology cache: cannot replace ") + path);
  }
  return ASYM_OK;
}

int topology_load(const char* path, const std::string& key, unsigned flags, Topology* out) {
  if (!path || !out) return fail(ASYM_EINVAL, "topology cache: null argument");
  std::ifstream f(path);
  if (!f) return nocache(std::string("no file ") + path);
  std::string line;
  if (!std::getline(f, line) || line != kMagic) return nocache("not a topology cache file");
  if (!std::getline(f, line) || line.compare(0, 4, "key ") != 0) return nocache("no key line");
  if (line.substr(4) != key) return nocache("made under another key (" + line.substr(4) + ")");
  Topology t;
  t.key = key;
  bool have_counts = false, have_end = false;
  int maskmap = 0;
  while (std::getline(f, line)) {
    std::istringstream in(line);
    std::string tag;
    in >> tag;
    if (tag == "flags") {
      if (!(in >> t.flags)) return nocache("bad flags line");
    } else if (tag == "counts") {
      if (!(in >> t.n_cus >> t.n_xccs >> maskmap >> t.rr_fraction)) return nocache("bad counts line");
      if (t.n_cus < 1 || t.n_cus > ASYM_MAX_CUS || t.n_xccs < 1 || t.n_xccs > ASYM_MAX_XCDS)
        return nocache("counts out of range");
      have_counts = true;
    } else if (tag == "partitions") {
      if (!(in >> t.compute_partition >> t.memory_partition)) return nocache("bad partitions line");
    } else if (tag == "cu") {
      CuRecord c;
      if (!(in >> c.xcc >> c.se >> c.sh >> c.cu >> c.mask_bit)) return nocache("bad cu line");
      t.cus.push_back(c);
    } else if (tag == "latency") {
      std::vector<double> v;
      double d;
      while (in >> d) v.push_back(d);
      if (!latency_from_values(v, t.lat)) return nocache("bad latency line");
      t.has_latency = true;
    } else if (tag == "end") {
      have_end = true;
      break;
    } else {
      return nocache("unknown line '" + tag + "'");
    }
  }
  if (!have_counts || !have_end) return nocache("truncated file");
  if ((int)t.cus.size() != t.n_cus) return nocache("CU record count differs from the CU count");
  if ((flags & t.flags) != flags) return nocache("the cached map lacks a requested probe");
  t.has_maskmap = maskmap != 0;
  if (t.has_maskmap != ((t.flags & ASYM_PROBE_MASKMAP) != 0)) return nocache("mask map flag disagrees with the probes");
  if (t.has_latency != ((t.flags & ASYM_PROBE_LATENCY) != 0)) return nocache("latency line disagrees with the probes");
  t.cus_per_xcd.assign(t.n_xccs, 0);
  t.bit_to_cu.assign(t.n_cus, -1);
  for (int i = 0; i < t.n_cus; ++i) {
    const CuRecord& c = t.cus[i];
    if (c.xcc < 0 || c.xcc >= t.n_xccs) return nocache("a CU record names an XCC beyond the count");
    t.cus_per_xcd[c.xcc] += 1;
    if (t.has_maskmap) {
      if (c.mask_bit < 0 || c.mask_bit >= t.n_cus || t.bit_to_cu[c.mask_bit] != -1)
        return nocache("mask bits are not a bijection");
      t.bit_to_cu[c.mask_bit] = i;
    }
  }
  if (check_invariants(t) != ASYM_OK) return nocache("the cached map breaks an invariant");
  *out = std::move(t);
  return ASYM_OK;
}

}  // namespace asym

using asym::fail;

extern "C" int asym_topology_cache_key(int device, char* buf, size_t len, size_t* needed) {
  std::string k;
  int rc = asym::device_key(device, &k, nullptr);
  if (rc != ASYM_OK) return rc;
  if (needed) *needed = k.size() + 1;
  if (!buf || len < k.size() + 1) return fail(ASYM_EINVAL, "cache key: buffer too small");
  std::memcpy(buf, k.c_str(), k.size() + 1);
  return ASYM_OK;
}

extern "C" int asym_topology_save(const asym_topology* topo, const char* path, const char* key) {
  const asym::Topology* t = asym::unwrap(topo);
  if (!t || !path) return fail(ASYM_EINVAL, "topology save: null argument");
  if (key) {
    asym::Topology c = *t;
    c.key = key;
    return asym::topology_save(c, path);
  }
  return asym::topology_save(*t, path);
}

extern "C" int asym_topology_load(const char* path, const char* key, unsigned flags, asym_topology** out) {
  if (!path || !key || !out) return fail(ASYM_EINVAL, "topology load: null argument");
  *out = nullptr;
  if (flags & ~(unsigned)(ASYM_PROBE_IDENTITY | ASYM_PROBE_MASKMAP | ASYM_PROBE_LATENCY))
    return fail(ASYM_EINVAL, "topology load: unknown flags");
  asym::Topology t;
  int rc = asym::topology_load(path, key, flags, &t);
  if (rc != ASYM_OK) return rc;
  *out = asym::wrap_topology(std::move(t));
  return ASYM_OK;
}
