// Host-only library code under AddressSanitizer and UndefinedBehaviorSanitizer:
// the tile schedules, the topology map (records, JSON, CU sets, cache file),
// the latency / affinity and partition-hash analyses, the home map and chunk
// lists, and the page placement of the paged attention cache, each on
// synthetic inputs of several sizes and on its error paths.  Every call's
// result is checked for the property the header promises (every tile exactly
// once, groups found, homes matching the hash, ...).  Test infrastructure
// only: built with g++ by tests/test_host_sanitizers.py.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <string>
#include <vector>

#include "asym.h"

static int g_fail = 0;
#define CHECK(c)                                                    \
  do {                                                              \
    if (!(c)) {                                                     \
      std::printf("FAILED %s:%d: %s (%s)\n", __FILE__, __LINE__, #c, \
                  asym_last_error());                               \
      ++g_fail;                                                     \
    }                                                               \
  } while (0)

static bool each_once(const std::vector<int>& order, int n) {
  std::vector<int> seen(n, 0);
  for (int t : order) {
    if (t < 0 || t >= n) return false;
    seen[t] += 1;
  }
  for (int c : seen)
    if (c != 1) return false;
  return true;
}

static void schedules(std::mt19937& g) {
  const int maps[3] = {ASYM_MAP_AWARE, ASYM_MAP_OBLIVIOUS_GROUPED, ASYM_MAP_OBLIVIOUS_ROWMAJOR};
  for (int trial = 0; trial < 300; ++trial) {
    const int tm = 1 + g() % 40, tn = 1 + g() % 40, nx = 1 + g() % 8;
    std::vector<int> slots(nx);
    int any = 0;
    for (int& s : slots) any += (s = g() % 33);
    if (!any) slots[0] = 1;
    for (int m : maps) {
      std::vector<int> order(tm * tn, -1), off(nx + 1), quota(nx);
      const int band = trial % 3 == 0 ? 0 : 1 + g() % tm;
      CHECK(asym_schedule_build(tm, tn, nx, slots.data(), m, band, order.data(), off.data(), quota.data()) ==
            ASYM_OK);
      CHECK(each_once(order, tm * tn));
      CHECK(off[0] == 0 && off[nx] == tm * tn);
    }
    const int G = 1 + g() % 6;
    std::vector<int> tms(G);
    int rows = 0;
    for (int& t : tms) rows += (t = g() % 5);
    for (int m : maps) {
      std::vector<int> order(rows * tn + 1, -1), off(nx + 1), quota(nx);
      CHECK(asym_grouped_schedule_build(G, tms.data(), tn, nx, slots.data(), m, order.data(), off.data(),
                                        quota.data()) == ASYM_OK);
      order.resize(rows * tn);
      CHECK(each_once(order, rows * tn));
    }
  }
  std::vector<int> o(4), off(3), q(2), s2 = {1, 1};
  CHECK(asym_schedule_build(0, 2, 2, s2.data(), ASYM_MAP_AWARE, 0, o.data(), off.data(), q.data()) == ASYM_EINVAL);
  CHECK(asym_schedule_build(2, 2, 2, nullptr, ASYM_MAP_AWARE, 0, o.data(), off.data(), q.data()) == ASYM_EINVAL);
}

// identity records of a layout: 8 XCCs x 4 engines x 8 CUs, 3 records per CU
static std::vector<int32_t> records(int n_xcc, int per_se, int reps) {
  std::vector<int32_t> r;
  int b = 0;
  for (int rep = 0; rep < reps; ++rep)
    for (int cu = 0; cu < per_se; ++cu)
      for (int se = 0; se < 4; ++se)
        for (int x = 0; x < n_xcc; ++x) {
          r.push_back(x);
          r.push_back((cu << 8) | (se << 13));
          r.push_back(b++);
          r.push_back(0);
        }
  return r;
}

static void topology(const char* dir) {
  std::vector<int32_t> rec = records(8, 8, 3);
  const int n = (int)rec.size() / 4;
  std::vector<int32_t> bit(256);
  for (int b = 0; b < 256; ++b) bit[b] = b;  // record b: its XCD is b mod 8, as the mask map has it
  asym_topology* t = nullptr;
  CHECK(asym_topology_from_records(rec.data(), n, 256, 8, bit.data(), &t) == ASYM_OK);
  if (!t) return;
  int ncu = 0, nx = 0, per[ASYM_MAX_XCDS];
  CHECK(asym_topology_info(t, &ncu, &nx, per, nullptr) == ASYM_OK && ncu == 256 && nx == 8 && per[3] == 32);
  size_t need = 0;
  asym_topology_json(t, nullptr, 0, &need);
  std::vector<char> js(need + 1);
  CHECK(asym_topology_json(t, js.data(), js.size(), &need) == ASYM_OK && std::strstr(js.data(), "\"cus\""));
  uint32_t m[ASYM_MASK_WORDS], ma[ASYM_MASK_WORDS], mb[ASYM_MASK_WORDS];
  for (int pol = 0; pol < 4; ++pol)
    for (int k : {8, 64, 128, 192, 255}) {
      if (asym_cuset_make(t, k, pol, 7, nullptr, m) != ASYM_OK) continue;  // some policies need whole XCDs
      int cnt[ASYM_MAX_XCDS];
      CHECK(asym_cuset_counts(t, m, cnt) == ASYM_OK);
      int s = 0;
      for (int x = 0; x < 8; ++x) s += cnt[x];
      CHECK(s == k);
    }
  CHECK(asym_cuset_split_xcds(t, 0x3F, ma, mb) == ASYM_OK);
  CHECK(asym_cuset_split_xcds(t, 0xFF, ma, mb) == ASYM_EINVAL);
  const std::string path = std::string(dir) + "/topo.txt";
  CHECK(asym_topology_save(t, path.c_str(), "key-1") == ASYM_OK);
  asym_topology* u = nullptr;
  CHECK(asym_topology_load(path.c_str(), "key-1", 0, &u) == ASYM_OK && u);
  asym_topology* w = nullptr;
  CHECK(asym_topology_load(path.c_str(), "key-2", 0, &w) == ASYM_ENOCACHE && !w);
  CHECK(asym_topology_load((path + ".none").c_str(), "key-1", 0, &w) == ASYM_ENOCACHE);
  // a truncated file is refused, not read past its end
  FILE* f = std::fopen(path.c_str(), "rb");
  std::vector<char> buf(1 << 16);
  const size_t len = f ? std::fread(buf.data(), 1, buf.size(), f) : 0;
  if (f) std::fclose(f);
  for (size_t cut : {len / 3, len / 2, len - 5}) {
    FILE* h = std::fopen(path.c_str(), "wb");
    std::fwrite(buf.data(), 1, cut, h);
    std::fclose(h);
    CHECK(asym_topology_load(path.c_str(), "key-1", 0, &w) == ASYM_ENOCACHE);
  }
  if (u) asym_topology_free(u);
  asym_topology_free(t);
  // broken record sets
  CHECK(asym_topology_from_records(rec.data(), n, 250, 8, nullptr, &t) == ASYM_EINVARIANT);
  CHECK(asym_topology_from_records(rec.data(), 0, 256, 8, nullptr, &t) != ASYM_OK);
}

// latencies [n_x][n]: lines homed on group h(i) are fast from that group's XCDs
static std::vector<uint32_t> two_group_lat(int n_x, int n, const std::vector<int>& home, std::mt19937& g) {
  std::vector<uint32_t> L((size_t)n_x * n);
  for (int x = 0; x < n_x; ++x)
    for (int i = 0; i < n; ++i)
      L[(size_t)x * n + i] = (home[i] == (x < n_x / 2 ? 0 : 1) ? 740 : 970) + g() % 30;
  return L;
}

static void analyses(std::mt19937& g) {
  const int n_x = 8, n = 512;
  std::vector<int> home(n);
  for (int& h : home) h = g() % 2;
  std::vector<uint32_t> L = two_group_lat(n_x, n, home, g);
  asym_latency_summary s;
  CHECK(asym_latency_analyze(L.data(), n_x, n, 0.5, 20.0, &s) == ASYM_OK && s.n_groups == 2);
  CHECK(s.group_of_xcd[0] == s.group_of_xcd[3] && s.group_of_xcd[0] != s.group_of_xcd[4]);
  CHECK(asym_latency_analyze(nullptr, n_x, n, 0.5, 20.0, &s) == ASYM_EINVAL);

  // partition hash: blocks of (base, base ^ bit b for b in [lo, hi)), home = parity(offset & mask)
  const uint64_t mask = (1ull << 13) | (1ull << 21) | (1ull << 28);
  const int lo = 7, hi = 34, block = 1 + (hi - lo);
  const int n_blocks = 64;
  std::vector<uint64_t> offs;
  for (int k = 0; k < n_blocks; ++k) {
    const uint64_t base = ((uint64_t)g() << 20 ^ g()) & ((1ull << hi) - 1) & ~127ull;
    offs.push_back(base);
    for (int b = lo; b < hi; ++b) offs.push_back(base ^ (1ull << b));
  }
  const int na = (int)offs.size();
  std::vector<int> hh(na);
  for (int i = 0; i < na; ++i) hh[i] = __builtin_popcountll(offs[i] & mask) & 1;
  std::vector<uint32_t> LI = two_group_lat(n_x, na, hh, g);
  std::vector<int8_t> hv(na);
  asym_interleave_result ir;
  CHECK(asym_interleave_analyze(LI.data(), n_x, na, offs.data(), block, 0.5, 20.0, 0.1, hv.data(), &ir) ==
        ASYM_OK);
  CHECK(ir.hash_mask == mask);

  // home map: page homes from the first line of each page, chunks by bit 13
  const int n_pages = 64, n_verify = 256;
  std::vector<int> ph(n_pages + n_verify);
  std::vector<uint64_t> vo(n_verify);
  for (int p = 0; p < n_pages; ++p) ph[p] = g() % 2;
  for (int v = 0; v < n_verify; ++v) {
    vo[v] = (((uint64_t)g() << 16) ^ g()) % ((uint64_t)n_pages << 21) & ~127ull;
    ph[n_pages + v] = ph[vo[v] >> 21] ^ (int)((vo[v] >> 13) & 1);
  }
  std::vector<uint32_t> LH = two_group_lat(n_x, n_pages + n_verify, ph, g);
  const int grp[8] = {0, 0, 0, 0, 1, 1, 1, 1};
  std::vector<int8_t> ch((size_t)n_pages * 256);
  asym_home_map_info hi_;
  CHECK(asym_home_map_analyze(LH.data(), n_x, n_pages, vo.data(), n_verify, grp, mask, 13, 20.0, ch.data(),
                              &hi_) == ASYM_OK);
  CHECK(hi_.verify_agree == hi_.verify_classified && hi_.verify_classified == n_verify);
  // 16 KiB chunks would straddle the hash's bit 13: two homes per chunk, refused
  CHECK(asym_home_map_analyze(LH.data(), n_x, n_pages, vo.data(), n_verify, grp, mask, 14, 20.0, ch.data(),
                              &hi_) == ASYM_EINVAL);
  std::vector<uint32_t> lists(ch.size());
  std::vector<int> off(n_x + 1);
  int listed = 0;
  for (int mode : {ASYM_CHUNKS_ALL, ASYM_CHUNKS_LOCAL, ASYM_CHUNKS_REMOTE})
    for (uint32_t xm : {0u, 0x0Fu, 0x81u}) {
      CHECK(asym_chunk_lists(ch.data(), (int)ch.size(), n_x, grp, xm, mode, lists.data(), off.data(), &listed) ==
            ASYM_OK);
      // every chunk once, except chunks whose home has no active reader under LOCAL / REMOTE
      CHECK(off[n_x] == listed && listed <= (int)ch.size());
      if (mode == ASYM_CHUNKS_ALL || xm == 0 || xm == 0x81u) CHECK(listed == (int)ch.size());
      std::vector<int> seen(ch.size(), 0);
      for (int k = 0; k < listed; ++k) CHECK(lists[k] < ch.size() && ++seen[lists[k]] == 1);
      for (int x = 0; x < n_x; ++x)
        for (int k = off[x]; k < off[x + 1]; ++k) {
          CHECK(xm == 0 || ((xm >> x) & 1));
          if (mode != ASYM_CHUNKS_ALL) CHECK((ch[lists[k]] == grp[x]) == (mode == ASYM_CHUNKS_LOCAL));
        }
    }
}

static void placement(std::mt19937& g) {
  for (int trial = 0; trial < 50; ++trial) {
    const int B = 1 + g() % 3, H = 1 + g() % 8, S = 1 + g() % 5000;
    const int split = 16 * (1 + g() % 64);
    asym_attn_plan_info p;
    std::memset(&p, 0, sizeof p);
    p.split_tokens = split;
    p.n_splits = (S + split - 1) / split;
    p.tasks = B * H * p.n_splits;
    p.n_xcds = 8;
    for (int x = 0, left = p.tasks; x < 8; ++x) {
      p.tasks_per_xcd[x] = x == 7 ? left : (int)(g() % (left + 1));
      left -= p.tasks_per_xcd[x];
    }
    const int pph = (S + 31) / 32;
    const size_t pool = (size_t)3 * B * H * pph + 3;
    std::vector<int8_t> home(pool);
    for (auto& h : home) h = (int8_t)((int)(g() % 10) - 1 < 0 ? -1 : g() % 2);
    const int grp[8] = {0, 0, 0, 0, 1, 1, 1, 1};
    std::vector<int32_t> pages((size_t)B * H * pph);
    for (int pol : {ASYM_PAGES_IN_ORDER, ASYM_PAGES_LOCAL, ASYM_PAGES_REMOTE}) {
      const int rc = asym_attn_pages_place(&p, B, H, S, home.data(), pool, grp, pol, pages.data());
      CHECK(rc == ASYM_OK || rc == ASYM_EINVAL);
      if (rc != ASYM_OK) continue;
      std::vector<int> seen(pool, 0);
      for (int32_t q : pages) {
        CHECK(q >= 0 && (size_t)q < pool);
        if (q >= 0 && (size_t)q < pool) CHECK(++seen[q] == 1);
      }
    }
  }
}

int main(int argc, char** argv) {
  std::mt19937 g(12345);
  schedules(g);
  topology(argc > 1 ? argv[1] : ".");
  analyses(g);
  placement(g);
  if (g_fail) {
    std::printf("%d checks failed\n", g_fail);
    return 1;
  }
  std::printf("all checks passed\n");
  return 0;
}
