// Partition-hash discovery (Section 6.1, NUMA partition identification).
//
// The paper finds the bits of the XOR hash that maps physical addresses to
// memory partitions by flipping one address bit at a time and watching, by
// latency, whether the address moves to the other partition.  Here the
// partition is the home affinity group of the latency analysis; the probe lays
// out blocks of a base line and its one- and two-bit variants in one fresh
// allocation, times them from every XCD in the HBM regime (the latency probe's
// measurement), and the analysis turns the homes into per-bit flip fractions,
// verdicts, the granularity, and a linearity check on the two-bit variants.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <vector>

#include "internal.h"

namespace asym {
namespace {

constexpr uint64_t kPage = 2ull << 20;
// translation warm-up line: five bits inside the 2 MiB page, so that it
// differs from every line of the block in at least three bits
constexpr uint64_t kTouch = 0x1F0000ull;

uint64_t mix64(uint64_t& s) {
  uint64_t z = (s += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

int validate(const asym_interleave_params& p) {
  if (p.n_bases < 1 || p.n_bases > 4096) return fail(ASYM_EINVAL, "interleave probe: n_bases must be in [1, 4096]");
  if (p.lo_bit < 7 || p.hi_bit > 36 || p.lo_bit >= p.hi_bit)
    return fail(ASYM_EINVAL, "interleave probe: need 7 <= lo_bit < hi_bit <= 36");
  if (p.n_pairs < 0 || p.n_pairs > 64 || (p.n_pairs > 0 && p.hi_bit - p.lo_bit < 2))
    return fail(ASYM_EINVAL, "interleave probe: n_pairs must be in [0, 64], 0 with one bit");
  if (p.passes < 1 || p.passes > 64) return fail(ASYM_EINVAL, "interleave probe: passes must be in [1, 64]");
  if (!(p.decide > 0.0 && p.decide < 0.5)) return fail(ASYM_EINVAL, "interleave probe: decide must be in (0, 0.5)");
  if (!(p.tie_cycles >= 0.0) || !(p.group_threshold > -1.0 && p.group_threshold < 1.0))
    return fail(ASYM_EINVAL, "interleave probe: threshold must be in (-1, 1), tie margin >= 0");
  return ASYM_OK;
}

}  // namespace

int analyze_interleave(const uint32_t* L, int n_x, int n_a, const uint64_t* offs, int block,
                       double threshold, double tie, double decide, int8_t* home_out,
                       asym_interleave_result& r) {
  if (!L || !offs || n_x < 1 || n_x > ASYM_MAX_XCDS || n_a < 1 || block < 1 || n_a % block)
    return fail(ASYM_EINVAL, "interleave analysis: bad sizes or a partial block");
  if (!(decide > 0.0 && decide < 0.5)) return fail(ASYM_EINVAL, "interleave analysis: decide must be in (0, 0.5)");
  asym_latency_summary s;
  std::vector<int8_t> home(n_a);
  int rc = analyze_latency(L, n_x, n_a, threshold, tie, s, home.data());
  if (rc != ASYM_OK) return rc;

  std::memset(&r, 0, sizeof r);
  r.n_xcds = n_x;
  r.n_groups = s.n_groups;
  for (int x = 0; x < ASYM_MAX_XCDS; ++x) r.group_of_xcd[x] = x < n_x ? s.group_of_xcd[x] : -1;
  r.n_addresses = n_a;
  r.block = block;
  r.unclassified_share = s.unclassified_share;

  int usable[64] = {0}, flips[64] = {0};
  bool tested[64] = {false};
  struct Pair { int b0, j, i, k; };
  std::vector<Pair> pairs;
  for (int b0 = 0; b0 < n_a; b0 += block) {
    for (int j = b0 + 1; j < b0 + block; ++j) {
      const uint64_t d = offs[j] ^ offs[b0];
      const int c = __builtin_popcountll(d);
      if (c == 1) {
        const int i = __builtin_ctzll(d);
        tested[i] = true;
        if (home[b0] >= 0 && home[j] >= 0) {
          usable[i] += 1;
          flips[i] += home[b0] != home[j];
        }
      } else if (c == 2) {
        const int i = __builtin_ctzll(d);
        const int k = 63 - __builtin_clzll(d);
        pairs.push_back({b0, j, i, k});
      }
    }
  }
  for (int i = 0; i < 64; ++i) {
    r.usable[i] = usable[i];
    r.flip_fraction[i] = usable[i] ? (double)flips[i] / usable[i] : -1.0;
    if (!tested[i])
      r.verdict[i] = ASYM_BIT_NOT_TESTED;
    else if (!usable[i])
      r.verdict[i] = ASYM_BIT_UNDETERMINED;
    else if (r.flip_fraction[i] >= 1.0 - decide)
      r.verdict[i] = 1;
    else if (r.flip_fraction[i] <= decide)
      r.verdict[i] = 0;
    else
      r.verdict[i] = ASYM_BIT_UNDETERMINED;
  }
  for (const Pair& p : pairs) {
    const int vi = r.verdict[p.i], vk = r.verdict[p.k];
    if (vi < 0 || vk < 0 || home[p.b0] < 0 || home[p.j] < 0) continue;
    r.pair_checks += 1;
    r.pair_agree += (home[p.b0] != home[p.j]) == ((vi ^ vk) == 1);
  }
  r.linear_consistency = r.pair_checks ? (double)r.pair_agree / r.pair_checks : -1.0;
  r.hash_mask = 0;
  r.lowest_bit = -1;
  int highest_tested = -1, lowest_undet = -1;
  for (int i = 0; i < 64; ++i) {
    if (r.verdict[i] == 1) {
      r.hash_mask |= 1ull << i;
      if (r.lowest_bit < 0) r.lowest_bit = i;
    }
    if (tested[i]) highest_tested = i;
    if (r.verdict[i] == ASYM_BIT_UNDETERMINED && lowest_undet < 0) lowest_undet = i;
  }
  r.determined_below = lowest_undet >= 0 ? lowest_undet : highest_tested + 1;
  r.granularity = (r.lowest_bit >= 0 && r.lowest_bit < r.determined_below) ? (int64_t)1 << r.lowest_bit : -1;

  // local and remote tiers over (XCD, classified line) pairs (integer sums)
  unsigned long long ls = 0, rs = 0, ln = 0, rn = 0;
  for (int x = 0; x < n_x; ++x)
    for (int i = 0; i < n_a; ++i) {
      if (home[i] < 0) continue;
      const uint32_t v = L[(size_t)x * n_a + i];
      if (home[i] == s.group_of_xcd[x]) {
        ls += v;
        ln += 1;
      } else {
        rs += v;
        rn += 1;
      }
    }
  r.local_cycles = ln ? (double)ls / ln : -1.0;
  r.remote_cycles = rn ? (double)rs / rn : -1.0;
  r.base_align = 0;
  if (home_out) std::memcpy(home_out, home.data(), n_a);
  return ASYM_OK;
}

int interleave_probe(int device, const asym_interleave_params& p, uint64_t* offs_out,
                     uint32_t* lat_out, int8_t* home_out, asym_interleave_result& out) {
  int rc = validate(p);
  if (rc != ASYM_OK) return rc;
  const int nb = p.hi_bit - p.lo_bit;
  const int block = 1 + nb + p.n_pairs;
  const uint64_t span = 1ull << p.hi_bit;
  LatencyMeasure m;
  m.alloc = std::max<uint64_t>(span, kPage);
  m.passes = p.passes;
  m.l2_samples = 0;
  m.mall = false;
  m.touch_delta = kTouch;
  size_t free_b = 0, total_b = 0;
  ASYM_HIP(hipSetDevice(device));
  ASYM_HIP(hipMemGetInfo(&free_b, &total_b));
  if (m.alloc + kPage + (2ull << 30) > free_b)
    return fail(ASYM_ENOMEM, "interleave probe: 2^hi_bit bytes plus the flush buffer exceed free memory");

  uint64_t st = p.seed;
  m.offs.reserve((size_t)p.n_bases * block);
  for (int b = 0; b < p.n_bases; ++b) {
    const uint64_t base = (mix64(st) % (span >> 7)) << 7;
    m.offs.push_back(base);
    for (int k = p.lo_bit; k < p.hi_bit; ++k) m.offs.push_back(base ^ (1ull << k));
    for (int q = 0; q < p.n_pairs; ++q) {
      const int i = p.lo_bit + (int)(mix64(st) % (uint64_t)nb);
      int k = p.lo_bit + (int)(mix64(st) % (uint64_t)(nb - 1));
      if (k >= i) k += 1;
      m.offs.push_back(base ^ (1ull << i) ^ (1ull << k));
    }
  }
  if ((rc = latency_measure(device, m)) != ASYM_OK) return rc;
  const int n_a = (int)m.offs.size();
  const uint32_t* hbm = &m.best[(size_t)2 * m.n_x * n_a];
  rc = analyze_interleave(hbm, m.n_x, n_a, m.offs.data(), block, p.group_threshold, p.tie_cycles,
                          p.decide, home_out, out);
  if (rc != ASYM_OK) return rc;
  out.base_align = m.base_align;
  if (offs_out) std::memcpy(offs_out, m.offs.data(), sizeof(uint64_t) * n_a);
  if (lat_out) std::memcpy(lat_out, hbm, sizeof(uint32_t) * (size_t)m.n_x * n_a);
  return ASYM_OK;
}

}  // namespace asym

extern "C" void asym_interleave_params_default(asym_interleave_params* p) {
  if (!p) return;
  p->n_bases = 128;
  p->lo_bit = 7;
  p->hi_bit = 32;
  p->n_pairs = 4;
  p->passes = 8;
  p->seed = 1;
  p->group_threshold = 0.5;
  p->tie_cycles = 20.0;
  p->decide = 0.1;
}

extern "C" int asym_interleave_probe(int device, const asym_interleave_params* p, uint64_t* offs,
                                     uint32_t* lat, int8_t* home, asym_interleave_result* out) {
  using namespace asym;
  if (!out) return fail(ASYM_EINVAL, "interleave probe: null output");
  asym_interleave_params q;
  if (p)
    q = *p;
  else
    asym_interleave_params_default(&q);
  return interleave_probe(device, q, offs, lat, home, *out);
}

extern "C" int asym_interleave_analyze(const uint32_t* hbm_lat, int n_xcds, int n_addr,
                                       const uint64_t* offs, int block, double group_threshold,
                                       double tie_cycles, double decide, int8_t* home,
                                       asym_interleave_result* out) {
  if (!out) return asym::fail(ASYM_EINVAL, "interleave analysis: null output");
  return asym::analyze_interleave(hbm_lat, n_xcds, n_addr, offs, block, group_threshold, tie_cycles,
                                  decide, home, *out);
}
