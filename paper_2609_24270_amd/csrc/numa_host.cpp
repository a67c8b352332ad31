// Host analysis of the home map and the per-XCD chunk lists (Section 6.1's
// page classification; the appendix on NUMA-aware address remapping places
// data by it).  No GPU: the device side (timing the lines, reading chunks) is
// in numa.hip.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <string>
#include <vector>

#include "internal.h"

namespace asym {
namespace {

constexpr uint64_t kPage = 2ull << 20;

int parity64(uint64_t v) { return __builtin_popcountll(v) & 1; }

// Homes of lines [n_x][n] given the XCD groups (two): the group with the lower
// mean latency, -1 when the two means are closer than `tie`.
void homes_given_groups(const uint32_t* L, int n_x, int n, const int* grp, double tie, int8_t* home) {
  int cnt[2] = {0, 0};
  for (int x = 0; x < n_x; ++x) cnt[grp[x]] += 1;
  for (int i = 0; i < n; ++i) {
    double s[2] = {0.0, 0.0};
    for (int x = 0; x < n_x; ++x) s[grp[x]] += L[(size_t)x * n + i];
    const double m0 = s[0] / cnt[0], m1 = s[1] / cnt[1];
    home[i] = std::fabs(m0 - m1) < tie ? -1 : (m0 < m1 ? 0 : 1);
  }
}

}  // namespace

int home_map_analyze(const uint32_t* L, int n_x, int n_pages, const uint64_t* voffs, int n_verify,
                     const int* grp, uint64_t hash_mask, int chunk_log2, double tie, int8_t* chunk_home,
                     asym_home_map_info& info) {
  if (!L || !grp || !chunk_home || (n_verify > 0 && !voffs))
    return fail(ASYM_EINVAL, "home map: null pointer");
  if (n_x < 1 || n_x > ASYM_MAX_XCDS || n_pages < 1 || n_pages > (1 << 22) || n_verify < 0 ||
      n_verify > (1 << 20) || !(tie >= 0.0))
    return fail(ASYM_EINVAL, "home map: bad sizes or tie margin");
  if (chunk_log2 < 12 || chunk_log2 > 21) return fail(ASYM_EINVAL, "home map: chunk_log2 must be in [12, 21]");
  const uint64_t in_page = hash_mask & (kPage - 1);
  if (in_page & ((1ull << chunk_log2) - 1))
    return fail(ASYM_EINVAL, "home map: the hash has bits below the chunk size, a chunk would have two homes");
  for (int x = 0; x < n_x; ++x)
    if (grp[x] < 0 || grp[x] > 1) return fail(ASYM_EUNSUPPORTED, "home map: needs two XCD groups (0, 1)");
  if (std::count(grp, grp + n_x, 0) == 0 || std::count(grp, grp + n_x, 1) == 0)
    return fail(ASYM_EUNSUPPORTED, "home map: needs XCDs in both groups");
  const uint64_t bytes = (uint64_t)n_pages * kPage;
  for (int v = 0; v < n_verify; ++v)
    if (voffs[v] >= bytes) return fail(ASYM_EINVAL, "home map: verification offset beyond the range");
  const int n_s = n_pages + n_verify;
  std::vector<int8_t> home(n_s);
  homes_given_groups(L, n_x, n_s, grp, tie, home.data());

  std::memset(&info, 0, sizeof info);
  info.n_pages = n_pages;
  info.n_chunks = (int)(bytes >> chunk_log2);
  info.n_groups = 2;
  for (int x = 0; x < ASYM_MAX_XCDS; ++x) info.group_of_xcd[x] = x < n_x ? grp[x] : -1;
  long long c0 = 0, c1 = 0;
  const size_t per_page = kPage >> chunk_log2;
  for (int p = 0; p < n_pages; ++p) {
    if (home[p] < 0) info.unclassified_pages += 1;
    for (size_t c = 0; c < per_page; ++c) {
      const uint64_t q = (uint64_t)c << chunk_log2;
      const int8_t h = home[p] < 0 ? -1 : (int8_t)(home[p] ^ parity64(q & in_page));
      chunk_home[(size_t)p * per_page + c] = h;
      c0 += h == 0;
      c1 += h == 1;
    }
  }
  info.chunk_share[0] = (double)c0 / info.n_chunks;
  info.chunk_share[1] = (double)c1 / info.n_chunks;
  info.n_verify = n_verify;
  for (int v = 0; v < n_verify; ++v) {
    const int8_t got = home[n_pages + v];
    const int8_t want = chunk_home[voffs[v] >> chunk_log2];
    if (got < 0 || want < 0) continue;
    info.verify_classified += 1;
    info.verify_agree += got == want;
  }
  unsigned long long ls = 0, rs = 0, ln = 0, rn = 0;
  for (int x = 0; x < n_x; ++x)
    for (int p = 0; p < n_pages; ++p) {
      if (home[p] < 0) continue;
      const uint32_t v = L[(size_t)x * n_s + p];
      if (home[p] == grp[x]) {
        ls += v;
        ln += 1;
      } else {
        rs += v;
        rn += 1;
      }
    }
  info.local_cycles = ln ? (double)ls / ln : -1.0;
  info.remote_cycles = rn ? (double)rs / rn : -1.0;
  return ASYM_OK;
}

int chunk_lists(const int8_t* home, int n_chunks, int n_x, const int* grp, uint32_t xcd_mask, int mode,
                uint32_t* out, int* off, int* n_listed) {
  if (!home || !out || !off || !n_listed || n_chunks < 0 || n_x < 1 || n_x > ASYM_MAX_XCDS)
    return fail(ASYM_EINVAL, "chunk lists: bad arguments");
  if (mode < ASYM_CHUNKS_ALL || mode > ASYM_CHUNKS_REMOTE) return fail(ASYM_EINVAL, "chunk lists: unknown mode");
  if (mode != ASYM_CHUNKS_ALL && !grp) return fail(ASYM_EINVAL, "chunk lists: LOCAL and REMOTE need the groups");
  const uint32_t all = n_x >= 32 ? ~0u : ((1u << n_x) - 1);
  const uint32_t act = xcd_mask ? (xcd_mask & all) : all;
  if (!act) return fail(ASYM_EINVAL, "chunk lists: no active XCD");
  if (grp)
    for (int x = 0; x < n_x; ++x)
      if (grp[x] < 0 || grp[x] > 1) return fail(ASYM_EINVAL, "chunk lists: group ids must be 0 or 1");
  std::vector<std::vector<uint32_t>> per(n_x);
  if (mode == ASYM_CHUNKS_ALL) {
    std::vector<int> xs;
    for (int x = 0; x < n_x; ++x)
      if ((act >> x) & 1) xs.push_back(x);
    for (int c = 0; c < n_chunks; ++c) per[xs[c % xs.size()]].push_back((uint32_t)c);
  } else {
    std::vector<int> readers[2];
    for (int x = 0; x < n_x; ++x)
      if ((act >> x) & 1) readers[mode == ASYM_CHUNKS_LOCAL ? grp[x] : 1 - grp[x]].push_back(x);
    long long dealt[2] = {0, 0};
    for (int c = 0; c < n_chunks; ++c) {
      const int h = home[c];
      if (h < 0 || h > 1 || readers[h].empty()) continue;
      per[readers[h][dealt[h]++ % readers[h].size()]].push_back((uint32_t)c);
    }
  }
  int k = 0;
  for (int x = 0; x < n_x; ++x) {
    off[x] = k;
    for (uint32_t c : per[x]) out[k++] = c;
  }
  off[n_x] = k;
  *n_listed = k;
  return ASYM_OK;
}

}  // namespace asym

extern "C" int asym_home_map_analyze(const uint32_t* lat, int n_xcds, int n_pages,
                                     const uint64_t* verify_offs, int n_verify, const int* group_of_xcd,
                                     uint64_t hash_mask, int chunk_log2, double tie_cycles,
                                     int8_t* chunk_home, asym_home_map_info* info) {
  if (!info) return asym::fail(ASYM_EINVAL, "home map: null info");
  return asym::home_map_analyze(lat, n_xcds, n_pages, verify_offs, n_verify, group_of_xcd, hash_mask,
                                chunk_log2, tie_cycles, chunk_home, *info);
}

extern "C" int asym_chunk_lists(const int8_t* chunk_home, int n_chunks, int n_xcds, const int* group_of_xcd,
                                uint32_t xcd_mask, int mode, uint32_t* chunks_out, int* off_out,
                                int* n_listed) {
  return asym::chunk_lists(chunk_home, n_chunks, n_xcds, group_of_xcd, xcd_mask, mode, chunks_out, off_out,
                           n_listed);
}

