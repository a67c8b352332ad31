// Tile schedules for the persistent GEMM.
//
// The paper's full-GPU recipe (Section 7.1, "Integration with popular
// kernels") converts a kernel to persistent blocks, lets each block find the
// unit it runs on, and hands it the tasks whose data is local to that unit's
// partition, with work spread over partitions in proportion to their compute
// units (same section, last paragraph, and the full-GPU lesson of
// Section 7.4).  On MI355X the partition that matters for a GEMM is the XCD:
// each XCD has a private L2, so tiles that share A rows and B columns should
// run on the same XCD at the same time.
//
// Banded order: tile rows are cut into bands of `band` rows; a band is walked
// column by column, each column top to bottom.  A run of s consecutive tiles of
// this order covers about band rows x s/band columns, a near-square block when
// band ~ sqrt(s).
//   AWARE:             every band is shared out among the XCDs: the band's
//                      tiles, in the banded order, are cut into contiguous runs
//                      whose lengths are the largest-remainder apportionment of
//                      the band's tile count by the XCDs' persistent
//                      workgroups, and an XCD's list is its run of band 0, then
//                      of band 1, and so on.  Each XCD's concurrent tiles then
//                      form a compact block in its own L2, and all XCDs work in
//                      the same band at the same time, so the band's A rows are
//                      fetched from HBM once for all of them (memory-side cache).
//                      Where a band holds fewer tiles than one round of
//                      every XCD's workgroups (band * tiles_n < n * s, s the
//                      same on every XCD), a band's runs would be strips a few
//                      columns wide, taken from two bands at once.  The grid is
//                      then cut into band x (s / band) blocks instead, numbered
//                      band by band and left to right; block k goes to XCD
//                      k mod n (where the blocks divide the grid and come out
//                      even).  4096x4096 at 256^2 tiles: each XCD runs one
//                      8x4 block, not two 8x2 strips.
//   OBLIVIOUS_GROUPED: the banded order, tile i to workgroup i mod P; round-robin
//                      dispatch then puts neighbouring tiles on different XCDs.
//   OBLIVIOUS_ROWMAJOR: row-major order, tile i to workgroup i mod P.
#include <algorithm>
#include <cstdint>

#include "internal.h"

namespace asym {

std::vector<int> largest_remainder_quotas(int total, const std::vector<int>& w) {
  const int n = (int)w.size();
  std::vector<int> q(n, 0);
  int64_t W = 0;
  for (int x : w) W += x;
  if (W <= 0 || total <= 0) return q;
  std::vector<int64_t> rem(n, 0);
  int64_t assigned = 0;
  for (int i = 0; i < n; ++i) {
    const int64_t num = (int64_t)total * w[i];
    q[i] = (int)(num / W);
    rem[i] = num % W;
    assigned += q[i];
  }
  int left = (int)(total - assigned);
  // hand out the remaining units to the largest remainders, ties to lower index
  std::vector<int> idx(n);
  for (int i = 0; i < n; ++i) idx[i] = i;
  std::stable_sort(idx.begin(), idx.end(),
                   [&](int a, int b) { return rem[a] > rem[b]; });
  for (int k = 0; k < n && left > 0; ++k) {
    if (w[idx[k]] <= 0) continue;
    q[idx[k]] += 1;
    --left;
  }
  return q;
}

// Band height: minimise band + ceil(s / band) for s tiles in flight per XCD;
// ties go to a band dividing tiles_m, then to the taller band.
static int choose_band(int tiles_m, int s) {
  if (s < 1) s = 1;
  int best = 1, best_cost = 1 << 30;
  bool best_div = false;
  for (int h = 1; h <= std::min(tiles_m, s); ++h) {
    const int cost = h + (s + h - 1) / h;
    const bool div = (tiles_m % h) == 0;
    if (cost < best_cost || (cost == best_cost && (div && !best_div)) ||
        (cost == best_cost && div == best_div)) {
      best = h;
      best_cost = cost;
      best_div = div;
    }
  }
  return best;
}

int build_schedule(int tiles_m, int tiles_n, int n_xcds, const int* slots,
                   int mapping, int band, Schedule& s) {
  if (tiles_m < 1 || tiles_n < 1) return fail(ASYM_EINVAL, "schedule: empty tile grid");
  if ((int64_t)tiles_m * tiles_n > (1 << 30)) return fail(ASYM_EINVAL, "schedule: tile grid too large");
  if (n_xcds < 1 || n_xcds > ASYM_MAX_XCDS) return fail(ASYM_EINVAL, "schedule: bad XCD count");
  if (!slots) return fail(ASYM_EINVAL, "schedule: null slots");
  if (band < 0) return fail(ASYM_EINVAL, "schedule: negative band");
  int P = 0, smax = 0;
  for (int x = 0; x < n_xcds; ++x) {
    if (slots[x] < 0) return fail(ASYM_EINVAL, "schedule: negative slot count");
    P += slots[x];
    smax = std::max(smax, slots[x]);
  }
  if (P < 1) return fail(ASYM_EINVAL, "schedule: no workgroup slots");
  if (mapping != ASYM_MAP_AWARE && mapping != ASYM_MAP_OBLIVIOUS_GROUPED &&
      mapping != ASYM_MAP_OBLIVIOUS_ROWMAJOR)
    return fail(ASYM_EINVAL, "schedule: bad mapping");

  const int T = tiles_m * tiles_n;
  s.tiles_m = tiles_m;
  s.tiles_n = tiles_n;
  s.n_xcds = n_xcds;
  s.order.assign(T, 0);
  s.off.assign(n_xcds + 1, 0);
  s.quota.assign(n_xcds, 0);

  if (mapping == ASYM_MAP_OBLIVIOUS_ROWMAJOR) {
    for (int i = 0; i < T; ++i) s.order[i] = i;
  } else {
    const int h = band > 0 ? std::min(band, tiles_m) : choose_band(tiles_m, smax);
    int i = 0;
    for (int r0 = 0; r0 < tiles_m; r0 += h) {
      const int r1 = std::min(tiles_m, r0 + h);
      for (int c = 0; c < tiles_n; ++c)
        for (int r = r0; r < r1; ++r) s.order[i++] = r * tiles_n + c;
    }
  }

  // the block-dealing form of the aware lists (auto band only)
  bool blocks = mapping == ASYM_MAP_AWARE && band == 0 && slots[0] >= 1;
  for (int x = 1; x < n_xcds && blocks; ++x) blocks = slots[x] == slots[0];
  const int bh = blocks ? choose_band(tiles_m, smax) : 1;
  const int bw = blocks ? slots[0] / bh : 1;
  if (blocks)
    blocks = slots[0] % bh == 0 && tiles_m % bh == 0 && tiles_n % bw == 0 &&
             (int64_t)bh * tiles_n < (int64_t)n_xcds * slots[0] && (T / slots[0]) % n_xcds == 0;
  if (blocks) {
    std::vector<std::vector<int>> lists(n_xcds);
    int k = 0;
    for (int r0 = 0; r0 < tiles_m; r0 += bh)
      for (int c0 = 0; c0 < tiles_n; c0 += bw, ++k)
        for (int c = c0; c < c0 + bw; ++c)
          for (int r = r0; r < r0 + bh; ++r) lists[k % n_xcds].push_back(r * tiles_n + c);
    int o = 0;
    for (int x = 0; x < n_xcds; ++x) {
      std::copy(lists[x].begin(), lists[x].end(), s.order.begin() + o);
      s.quota[x] = (int)lists[x].size();
      o += s.quota[x];
      s.off[x + 1] = o;
    }
  } else if (mapping == ASYM_MAP_AWARE) {
    // per band: apportion the band's tiles, cut the band's banded order into
    // one contiguous run per XCD; then concatenate each XCD's runs band by band
    const int h = band > 0 ? std::min(band, tiles_m) : choose_band(tiles_m, smax);
    std::vector<int> w(slots, slots + n_xcds);
    std::vector<std::vector<int>> lists(n_xcds);
    int i = 0;
    for (int r0 = 0; r0 < tiles_m; r0 += h) {
      const int len = (std::min(tiles_m, r0 + h) - r0) * tiles_n;
      const std::vector<int> q = largest_remainder_quotas(len, w);
      int pos = i;
      for (int x = 0; x < n_xcds; ++x) {
        lists[x].insert(lists[x].end(), s.order.begin() + pos, s.order.begin() + pos + q[x]);
        pos += q[x];
      }
      i += len;
    }
    int o = 0;
    for (int x = 0; x < n_xcds; ++x) {
      std::copy(lists[x].begin(), lists[x].end(), s.order.begin() + o);
      s.quota[x] = (int)lists[x].size();
      o += s.quota[x];
      s.off[x + 1] = o;
    }
  } else {
    // one shared list; quota[x] counts tiles that workgroup i mod P, placed on
    // XCD (i mod P) mod n_xcds by round-robin dispatch, would run on XCD x
    for (int x = 0; x <= n_xcds; ++x) s.off[x] = (x == n_xcds) ? T : 0;
    for (int i = 0; i < T; ++i) s.quota[(i % P) % n_xcds] += 1;
  }
  return ASYM_OK;
}

// Grouped GEMM (the same recipe applied to grouped GEMM, Section 7.1: the
// expert layer of mixture-of-experts models).  Group g has tiles_m[g] tile rows
// of tiles_n columns; tile ids number the groups' tiles in group order,
// row-major inside a group (id = base_g + r * tiles_n + c).  Every group is one
// band: walked column by column, top to bottom, so the tiles that share a
// column panel of the group's weights follow each other.
//   AWARE:             every group is shared out among the XCDs as a band of
//                      the plain schedule is: contiguous runs of its walk, of
//                      largest-remainder lengths by the XCDs' workgroups; an
//                      XCD's list is its runs, group after group.  An XCD's
//                      concurrent tiles then hold few column panels of few
//                      groups, each panel fetched into its L2 once.
//   OBLIVIOUS_GROUPED: the same walk, tile i to workgroup i mod P.
//   OBLIVIOUS_ROWMAJOR: tile ids in order, tile i to workgroup i mod P.
int build_grouped_schedule(int G, const int* tiles_m, int tiles_n, int n_xcds, const int* slots,
                           int mapping, Schedule& s) {
  if (G < 1) return fail(ASYM_EINVAL, "grouped schedule: no groups");
  if (!tiles_m || !slots) return fail(ASYM_EINVAL, "grouped schedule: null argument");
  if (tiles_n < 1) return fail(ASYM_EINVAL, "grouped schedule: no tile columns");
  if (n_xcds < 1 || n_xcds > ASYM_MAX_XCDS) return fail(ASYM_EINVAL, "grouped schedule: bad XCD count");
  if (mapping != ASYM_MAP_AWARE && mapping != ASYM_MAP_OBLIVIOUS_GROUPED &&
      mapping != ASYM_MAP_OBLIVIOUS_ROWMAJOR)
    return fail(ASYM_EINVAL, "grouped schedule: bad mapping");
  int P = 0;
  for (int x = 0; x < n_xcds; ++x) {
    if (slots[x] < 0) return fail(ASYM_EINVAL, "grouped schedule: negative slot count");
    P += slots[x];
  }
  if (P < 1) return fail(ASYM_EINVAL, "grouped schedule: no workgroup slots");
  int64_t rows = 0;
  for (int g = 0; g < G; ++g) {
    if (tiles_m[g] < 0) return fail(ASYM_EINVAL, "grouped schedule: negative tile rows");
    rows += tiles_m[g];
  }
  if (rows * tiles_n > (1 << 30)) return fail(ASYM_EINVAL, "grouped schedule: too many tiles");
  const int T = (int)(rows * tiles_n);
  s.tiles_m = (int)rows;
  s.tiles_n = tiles_n;
  s.n_xcds = n_xcds;
  s.order.assign(T, 0);
  s.off.assign(n_xcds + 1, 0);
  s.quota.assign(n_xcds, 0);
  if (T == 0) return ASYM_OK;

  // the walk, one band per group
  std::vector<int> walk(T), band_start(G + 1, 0);
  {
    int i = 0, base = 0;
    for (int g = 0; g < G; ++g) {
      band_start[g] = i;
      for (int c = 0; c < tiles_n; ++c)
        for (int r = 0; r < tiles_m[g]; ++r) walk[i++] = base + r * tiles_n + c;
      base += tiles_m[g] * tiles_n;
    }
    band_start[G] = i;
  }
  if (mapping == ASYM_MAP_AWARE) {
    std::vector<int> w(slots, slots + n_xcds);
    std::vector<std::vector<int>> lists(n_xcds);
    for (int g = 0; g < G; ++g) {
      const int len = band_start[g + 1] - band_start[g];
      if (len == 0) continue;
      const std::vector<int> q = largest_remainder_quotas(len, w);
      int pos = band_start[g];
      for (int x = 0; x < n_xcds; ++x) {
        lists[x].insert(lists[x].end(), walk.begin() + pos, walk.begin() + pos + q[x]);
        pos += q[x];
      }
    }
    int o = 0;
    for (int x = 0; x < n_xcds; ++x) {
      std::copy(lists[x].begin(), lists[x].end(), s.order.begin() + o);
      s.quota[x] = (int)lists[x].size();
      o += s.quota[x];
      s.off[x + 1] = o;
    }
  } else {
    if (mapping == ASYM_MAP_OBLIVIOUS_GROUPED)
      s.order = walk;
    else
      for (int i = 0; i < T; ++i) s.order[i] = i;
    for (int x = 0; x <= n_xcds; ++x) s.off[x] = (x == n_xcds) ? T : 0;
    for (int i = 0; i < T; ++i) s.quota[(i % P) % n_xcds] += 1;
  }
  return ASYM_OK;
}

}  // namespace asym

extern "C" int asym_grouped_schedule_build(int G, const int* tiles_m, int tiles_n, int n_xcds,
                                           const int* slots, int mapping, int* order, int* off,
                                           int* quota) {
  asym::Schedule s;
  int rc = asym::build_grouped_schedule(G, tiles_m, tiles_n, n_xcds, slots, mapping, s);
  if (rc != ASYM_OK) return rc;
  if (order) std::copy(s.order.begin(), s.order.end(), order);
  if (off) std::copy(s.off.begin(), s.off.end(), off);
  if (quota) std::copy(s.quota.begin(), s.quota.end(), quota);
  return ASYM_OK;
}

extern "C" int asym_schedule_build(int tiles_m, int tiles_n, int n_xcds,
                                   const int* slots, int mapping, int band,
                                   int* order, int* off, int* quota) {
  asym::Schedule s;
  int rc = asym::build_schedule(tiles_m, tiles_n, n_xcds, slots, mapping, band, s);
  if (rc != ASYM_OK) return rc;
  if (order) std::copy(s.order.begin(), s.order.end(), order);
  if (off) std::copy(s.off.begin(), s.off.end(), off);
  if (quota) std::copy(s.quota.begin(), s.quota.end(), quota);
  return ASYM_OK;
}
