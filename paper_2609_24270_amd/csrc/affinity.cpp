// XCD-to-memory affinity from per-address latencies (host only).
//
// Appendix G probes the same sampled addresses from every XCD, groups XCDs
// whose address-dependent latency patterns correlate, and gives each address
// the home group with the lowest mean latency; Section 6.1 reads local and
// remote tiers off the same data.  Here the correlation is Pearson's over the
// sampled addresses, groups are the connected components of "correlation
// above a threshold", and an address whose two best group means are closer
// than a tie margin stays unclassified (the paper states none of these three
// choices).
#include <cmath>
#include <cstring>
#include <vector>

#include "internal.h"

namespace asym {

int analyze_latency(const uint32_t* L, int n_x, int n_s, double threshold, double tie,
                    asym_latency_summary& out, int8_t* home) {
  if (!L || n_x < 1 || n_x > ASYM_MAX_XCDS || n_s < 1)
    return fail(ASYM_EINVAL, "latency analysis: bad sizes");
  if (!std::isfinite(threshold) || !std::isfinite(tie) || tie < 0)
    return fail(ASYM_EINVAL, "latency analysis: bad threshold or tie margin");
  asym_latency_summary s;
  std::memset(&s, 0, sizeof s);
  s.n_xcds = n_x;
  s.n_samples = n_s;
  s.passes = -1;
  s.l2_samples = -1;
  s.timer_overhead = -1;
  s.clock_mhz = -1;
  for (int x = 0; x < ASYM_MAX_XCDS; ++x) {
    s.l2_hit[x] = s.mall_hit[x] = s.hbm[x] = -1;
    s.group_of_xcd[x] = -1;
    s.home_share[x] = 0;
    for (int y = 0; y < ASYM_MAX_XCDS; ++y) {
      s.corr[x][y] = 0;
      s.hbm_by_home[x][y] = -1;
    }
  }

  // per-XCD means (sums of integers are exact in double below 2^53)
  std::vector<double> mean(n_x);
  for (int x = 0; x < n_x; ++x) {
    double sum = 0;
    for (int i = 0; i < n_s; ++i) sum += L[(size_t)x * n_s + i];
    mean[x] = sum / n_s;
    s.hbm[x] = mean[x];
  }
  // Pearson correlation of the per-address latency rows
  std::vector<double> ss(n_x, 0.0);
  for (int x = 0; x < n_x; ++x)
    for (int i = 0; i < n_s; ++i) {
      const double d = L[(size_t)x * n_s + i] - mean[x];
      ss[x] += d * d;
    }
  for (int x = 0; x < n_x; ++x) {
    s.corr[x][x] = 1.0;
    for (int y = x + 1; y < n_x; ++y) {
      double c = 0;
      if (ss[x] > 0 && ss[y] > 0) {
        double sxy = 0;
        for (int i = 0; i < n_s; ++i)
          sxy += (L[(size_t)x * n_s + i] - mean[x]) * (L[(size_t)y * n_s + i] - mean[y]);
        c = sxy / std::sqrt(ss[x] * ss[y]);
      }
      s.corr[x][y] = s.corr[y][x] = c;
    }
  }
  // connected components of corr > threshold, numbered by lowest member
  int n_g = 0;
  for (int x = 0; x < n_x; ++x) {
    if (s.group_of_xcd[x] >= 0) continue;
    const int g = n_g++;
    std::vector<int> stack{x};
    s.group_of_xcd[x] = g;
    while (!stack.empty()) {
      const int u = stack.back();
      stack.pop_back();
      for (int v = 0; v < n_x; ++v)
        if (s.group_of_xcd[v] < 0 && s.corr[u][v] > threshold) {
          s.group_of_xcd[v] = g;
          stack.push_back(v);
        }
    }
  }
  s.n_groups = n_g;
  std::vector<int> gsize(n_g, 0);
  for (int x = 0; x < n_x; ++x) gsize[s.group_of_xcd[x]] += 1;

  // home group of every address
  std::vector<long long> home_count(n_g, 0);
  std::vector<std::vector<double>> by_home_sum(n_x, std::vector<double>(n_g, 0.0));
  long long unclassified = 0;
  std::vector<double> gsum(n_g);
  for (int i = 0; i < n_s; ++i) {
    std::fill(gsum.begin(), gsum.end(), 0.0);
    for (int x = 0; x < n_x; ++x) gsum[s.group_of_xcd[x]] += L[(size_t)x * n_s + i];
    int best = 0;
    double b1 = gsum[0] / gsize[0];
    for (int g = 1; g < n_g; ++g) {
      const double m = gsum[g] / gsize[g];
      if (m < b1) {
        b1 = m;
        best = g;
      }
    }
    bool tied = false;
    for (int g = 0; g < n_g; ++g)
      if (g != best && gsum[g] / gsize[g] - b1 < tie) tied = true;
    if (home) home[i] = (int8_t)(tied ? -1 : best);
    if (tied) {
      ++unclassified;
      continue;
    }
    home_count[best] += 1;
    for (int x = 0; x < n_x; ++x) by_home_sum[x][best] += L[(size_t)x * n_s + i];
  }
  for (int g = 0; g < n_g; ++g) {
    s.home_share[g] = (double)home_count[g] / n_s;
    for (int x = 0; x < n_x; ++x)
      s.hbm_by_home[x][g] = home_count[g] > 0 ? by_home_sum[x][g] / home_count[g] : -1.0;
  }
  s.unclassified_share = (double)unclassified / n_s;
  out = s;
  return ASYM_OK;
}

}  // namespace asym

extern "C" int asym_latency_analyze(const uint32_t* hbm_lat, int n_xcds, int n_samples,
                                    double group_threshold, double tie_cycles,
                                    asym_latency_summary* out) {
  if (!out) return asym::fail(ASYM_EINVAL, "latency analysis: null output");
  return asym::analyze_latency(hbm_lat, n_xcds, n_samples, group_threshold, tie_cycles, *out);
}

extern "C" void asym_latency_params_default(asym_latency_params* p) {
  if (!p) return;
  p->alloc_bytes = 0;
  p->n_samples = 16384;
  p->passes = 8;
  p->l2_samples = 4096;
  p->seed = 0;
  p->group_threshold = 0.5;
  p->tie_cycles = 20.0;
}
