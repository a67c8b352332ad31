// Page placement of the paged decode-attention cache (Appendix E: memory
// remapping by home).  Host only.
//
// A task of the aware mapping is owned by the XCD whose share of the task
// list holds it (the shares are consecutive in XCD order, each sized to the
// XCD's CUs); that XCD's workgroups claim it first.  Every 32-token page of a
// head is read by the task of its first token, so placing a page in memory
// homed on that XCD's die keeps its reads local.
#include <string>
#include <vector>

#include "internal.h"

using asym::fail;

extern "C" int asym_attn_pages_place(const asym_attn_plan_info* plan, int B, int H_kv, int S_k,
                                     const int8_t* pool_home, size_t pool_pages, const int* group_of_xcd,
                                     int policy, int32_t* pages) {
  if (!plan || !pages) return fail(ASYM_EINVAL, "page placement: null argument");
  if (B < 1 || H_kv < 1 || S_k < 1) return fail(ASYM_EINVAL, "page placement: B, H_kv, S_k must be >= 1");
  const int L = plan->split_tokens;
  if (L < 16 || L % 16) return fail(ASYM_EINVAL, "page placement: the plan's split is not a multiple of 16");
  const long long n_splits = (S_k + (long long)L - 1) / L;
  if (plan->n_splits != n_splits || plan->tasks != (long long)B * H_kv * n_splits)
    return fail(ASYM_EINVAL, "page placement: the plan is not one of this B, H_kv, S_k");
  const int T = asym::attn_page_tokens();
  const long long pph = (S_k + (long long)T - 1) / T;
  const long long total = (long long)B * H_kv * pph;
  if ((size_t)total > pool_pages) return fail(ASYM_EINVAL, "page placement: the pool has fewer pages than the cache");
  if (total > (1ll << 31) - 1) return fail(ASYM_EINVAL, "page placement: too many pages");
  if (policy == ASYM_PAGES_IN_ORDER) {
    for (long long i = 0; i < total; ++i) pages[i] = (int32_t)i;
    return ASYM_OK;
  }
  if (policy != ASYM_PAGES_LOCAL && policy != ASYM_PAGES_REMOTE)
    return fail(ASYM_EINVAL, "page placement: unknown policy");
  if (!pool_home || !group_of_xcd) return fail(ASYM_EINVAL, "page placement: homes and groups are needed");
  const int n_x = plan->n_xcds;
  if (n_x < 1 || n_x > ASYM_MAX_XCDS) return fail(ASYM_EINVAL, "page placement: bad XCD count in the plan");
  std::vector<long long> off(n_x + 1, 0);
  for (int x = 0; x < n_x; ++x) {
    if (plan->tasks_per_xcd[x] < 0) return fail(ASYM_EINVAL, "page placement: negative share");
    if (group_of_xcd[x] != 0 && group_of_xcd[x] != 1)
      return fail(ASYM_EINVAL, "page placement: groups must be 0 or 1");
    off[x + 1] = off[x] + plan->tasks_per_xcd[x];
  }
  if (off[n_x] != plan->tasks) return fail(ASYM_EINVAL, "page placement: shares do not add up to the tasks");
  // free pool pages of each group, in address order
  std::vector<size_t> cursor(2, 0);
  std::vector<std::vector<int32_t>> free_of(2);
  for (size_t i = 0; i < pool_pages; ++i)
    if (pool_home[i] == 0 || pool_home[i] == 1) free_of[pool_home[i]].push_back((int32_t)i);
  int x = 0;
  for (long long bh = 0; bh < (long long)B * H_kv; ++bh) {
    for (long long pg = 0; pg < pph; ++pg) {
      const long long task = bh * n_splits + (pg * T) / L;
      while (x > 0 && task < off[x]) --x;  // tasks rise with (bh, pg); the owner only moves forward
      while (task >= off[x + 1]) ++x;
      const int g = group_of_xcd[x] ^ (policy == ASYM_PAGES_REMOTE ? 1 : 0);
      if (cursor[g] >= free_of[g].size())
        return fail(ASYM_EINVAL, "page placement: the pool has too few pages homed on group " + std::to_string(g));
      pages[bh * pph + pg] = free_of[g][cursor[g]++];
    }
  }
  return ASYM_OK;
}
