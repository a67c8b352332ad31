// Topology probes for gfx950.
//
// Identity probe (the AMD analogue of Section 5.1's cluster probing): every
// workgroup reads the XCC_ID and HW_ID hardware registers, which name the XCD,
// shader engine, shader array and CU it runs on, and writes them out with its
// block index and a timestamp.  Each workgroup reserves a large slice of LDS so
// that at most two share a CU, and spins for a few microseconds so that the
// launch spreads over every CU; the spin is bounded by an iteration cap.
//
// Mask map: CU masks are given as bits, and which physical CU a bit controls
// is not documented for multi-XCD parts, so it is measured.  For each bit b a
// stream is created whose mask has every bit except b, the identity probe is
// run on it, and the one CU that never reports is the CU of bit b.  Every XCD
// keeps all its other CUs, so no launch can be left without a CU to run on.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <map>
#include <set>
#include <thread>
#include <tuple>

#include "internal.h"

namespace asym {
namespace {

constexpr int kProbeLds = 64 * 1024;  // bytes of LDS reserved per workgroup

__global__ void __launch_bounds__(64) probe_identity_kernel(int32_t* rec, long spin_cycles) {
  extern __shared__ int lds_reserve[];
  uint32_t x, h;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(x));
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_HW_ID)" : "=s"(h));
  const unsigned long long t0 = __builtin_amdgcn_s_memtime();
  unsigned long long t = t0;
  for (int it = 0; it < (1 << 20) && (long)(t - t0) < spin_cycles; ++it) t = __builtin_amdgcn_s_memtime();
  if (threadIdx.x == 0) {
    lds_reserve[0] = (int)x;  // keeps the reservation observable
    int32_t* r = rec + 4 * (size_t)blockIdx.x;
    r[0] = (int32_t)x;
    r[1] = (int32_t)h;
    r[2] = (int32_t)blockIdx.x;
    r[3] = (int32_t)(uint32_t)t0;
  }
}

}  // namespace

int probe_identity_run(int device, hipStream_t s, int n_blocks, std::vector<int32_t>& rec, int pre_blocks) {
  (void)device;
  if (n_blocks < 1 || pre_blocks < 0) return fail(ASYM_EINVAL, "probe: no blocks");
  int32_t* d = nullptr;
  const size_t bytes = sizeof(int32_t) * 4 * (size_t)(n_blocks + pre_blocks);
  ASYM_HIP(hipMalloc(&d, bytes));
  hipError_t e = hipMemsetAsync(d, 0xFF, bytes, s);
  if (e == hipSuccess && pre_blocks > 0) {
    // a launch of pre_blocks workgroups right before the probed one, on the same stream
    hipLaunchKernelGGL(probe_identity_kernel, dim3(pre_blocks), dim3(64), kProbeLds, s, d + 4 * (size_t)n_blocks,
                       20000L);
    e = hipGetLastError();
  }
  if (e == hipSuccess) {
    hipLaunchKernelGGL(probe_identity_kernel, dim3(n_blocks), dim3(64), kProbeLds, s, d, 20000L);
    e = hipGetLastError();
  }
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  rec.assign(4 * (size_t)n_blocks, -1);
  if (e == hipSuccess) e = hipMemcpy(rec.data(), d, sizeof(int32_t) * 4 * (size_t)n_blocks, hipMemcpyDeviceToHost);
  (void)hipFree(d);
  if (e != hipSuccess) return hip_fail(e, "identity probe");
  for (int i = 0; i < n_blocks; ++i)
    if (rec[4 * i + 2] != i) return fail(ASYM_EHIP, "identity probe: a workgroup left no record");
  return ASYM_OK;
}

// Map every mask bit to the CU it controls (see file comment).
static int probe_maskmap(int device, const Topology& t, const std::vector<int32_t>& base_rec,
                         std::vector<int32_t>& bit_record) {
  using Key = std::tuple<int, int, int, int>;
  std::map<Key, int> rec_of;  // tuple -> index of a record in base_rec
  const int nb = (int)base_rec.size() / 4;
  for (int i = 0; i < nb; ++i) {
    const uint32_t x = (uint32_t)base_rec[4 * i], h = (uint32_t)base_rec[4 * i + 1];
    rec_of.emplace(Key(xccid(x), hwid_se(h), hwid_sh(h), hwid_cu(h)), i);
  }
  bit_record.assign(t.n_cus, -1);
  const int n_blocks = 16 * t.n_cus;
  for (int b = 0; b < t.n_cus; ++b) {
    uint32_t mask[ASYM_MASK_WORDS] = {0};
    for (int c = 0; c < t.n_cus; ++c)
      if (c != b) mask[c >> 5] |= 1u << (c & 31);
    hipStream_t s = nullptr;
    ASYM_HIP(hipExtStreamCreateWithCUMask(&s, ASYM_MASK_WORDS, mask));
    std::vector<int32_t> rec;
    int rc = probe_identity_run(device, s, n_blocks, rec);
    (void)hipStreamDestroy(s);
    if (rc != ASYM_OK) return rc;
    std::set<Key> seen;
    for (int i = 0; i < n_blocks; ++i) {
      const uint32_t x = (uint32_t)rec[4 * i], h = (uint32_t)rec[4 * i + 1];
      seen.insert(Key(xccid(x), hwid_se(h), hwid_sh(h), hwid_cu(h)));
    }
    int missing = -1, n_missing = 0;
    for (const CuRecord& c : t.cus) {
      const Key k(c.xcc, c.se, c.sh, c.cu);
      if (!seen.count(k)) {
        ++n_missing;
        missing = rec_of[k];
      }
    }
    if (n_missing != 1)
      return fail(ASYM_EINVARIANT, "mask map: mask without bit " + std::to_string(b) + " left " +
                                       std::to_string(n_missing) + " CUs silent (expected 1)");
    bit_record[b] = missing;
  }
  return ASYM_OK;
}

}  // namespace asym

struct asym_topology;
namespace asym {
asym_topology* wrap_topology(Topology&& t);
const Topology* unwrap(const asym_topology* p);
}

extern "C" int asym_probe_topology(int device, unsigned flags, const char* cache_path, asym_topology** out) {
  using namespace asym;
  if (!out) return fail(ASYM_EINVAL, "null out");
  *out = nullptr;
  if (flags & ~(unsigned)(ASYM_PROBE_IDENTITY | ASYM_PROBE_MASKMAP | ASYM_PROBE_LATENCY))
    return fail(ASYM_EINVAL, "probe: unknown flags");
  // every probe includes the identity probe (the mask map and the latency
  // probe are built on its CU records)
  flags |= ASYM_PROBE_IDENTITY;
  asym_device_info info;
  std::string key;
  int rc = device_key(device, &key, &info);
  if (rc != ASYM_OK) return rc;
  if (cache_path) {
    Topology cached;
    if (topology_load(cache_path, key, flags, &cached) == ASYM_OK) {
      cached.device = device;
      *out = wrap_topology(std::move(cached));
      return ASYM_OK;
    }
  }
  ASYM_HIP(hipSetDevice(device));
  if (info.n_cus > ASYM_MAX_CUS || info.n_xccs > ASYM_MAX_XCDS)
    return fail(ASYM_EUNSUPPORTED, "probe: device larger than the mask format");
  // oversubscribe: 32 workgroups per CU, two resident per CU at a time
  const int n_blocks = 32 * info.n_cus;
  hipStream_t s = nullptr;
  ASYM_HIP(hipStreamCreateWithFlags(&s, hipStreamNonBlocking));
  std::vector<int32_t> rec;
  rc = probe_identity_run(device, s, n_blocks, rec);
  (void)hipStreamDestroy(s);
  if (rc != ASYM_OK) return rc;
  Topology t;
  rc = build_topology(rec.data(), n_blocks, info.n_cus, info.n_xccs, nullptr, t);
  if (rc != ASYM_OK) return rc;
  t.device = device;
  if (flags & ASYM_PROBE_MASKMAP) {
    std::vector<int32_t> bit_record;
    rc = probe_maskmap(device, t, rec, bit_record);
    if (rc != ASYM_OK) return rc;
    Topology t2;
    rc = build_topology(rec.data(), n_blocks, info.n_cus, info.n_xccs, bit_record.data(), t2);
    if (rc != ASYM_OK) return rc;
    t2.device = device;
    t = std::move(t2);
  }
  if (flags & ASYM_PROBE_LATENCY) {
    rc = probe_latency_run(device, t);
    if (rc != ASYM_OK) return rc;
  }
  t.flags = flags;
  t.key = key;
  t.compute_partition = info.compute_partition;
  t.memory_partition = info.memory_partition;
  if (cache_path) (void)topology_save(t, cache_path);  // a failed write leaves the probe result valid
  *out = wrap_topology(std::move(t));
  return ASYM_OK;
}

// Where a launch on a CU set lands: the identity kernel is run on a stream
// restricted to `mask` (NULL = every CU), optionally right after a launch of
// pre_blocks workgroups, and each workgroup's XCC is compared with its block
// index mod the XCD count.  The measure is per residue class: the share of
// workgroups that sit on the XCD holding most of their class (block index mod
// n), and the rotation k for which XCC = (b + k) mod n fits most workgroups.
// The aware schedules need each class on one XCD; which XCD a class lands on
// (the rotation) matters only where XCDs differ in CU count.  All of this is a
// performance assumption: no kernel's correctness depends on it.
static int dispatch_run(const asym_topology* topo, const uint32_t* mask, int pre_blocks, double* class_fraction,
                        int* rotation, int* blocks_per_xcd) {
  using namespace asym;
  const Topology* t = unwrap(topo);
  if (!t || !class_fraction || !rotation) return fail(ASYM_EINVAL, "dispatch check: null argument");
  int device = 0;
  ASYM_HIP(hipGetDevice(&device));
  if (t->device >= 0 && t->device != device)
    return fail(ASYM_EINVAL, "dispatch check: topology was probed on another device");
  void* sv = nullptr;
  int rc = asym_stream_create(topo, mask, &sv);
  if (rc != ASYM_OK) return rc;
  hipStream_t s = static_cast<hipStream_t>(sv);
  const int n_blocks = 4 * t->n_cus;
  std::vector<int32_t> rec;
  rc = probe_identity_run(device, s, n_blocks, rec, pre_blocks);
  asym_stream_destroy(sv);
  if (rc != ASYM_OK) return rc;
  std::vector<int> per(ASYM_MAX_XCDS, 0), xs(n_blocks), blk(n_blocks);
  for (int b = 0; b < n_blocks; ++b) {
    blk[b] = b;
    xs[b] = xccid((uint32_t)rec[4 * b]);
    if (xs[b] < ASYM_MAX_XCDS) per[xs[b]] += 1;
  }
  dispatch_stats(blk.data(), xs.data(), n_blocks, t->n_xccs, class_fraction, rotation);
  if (blocks_per_xcd)
    for (int x = 0; x < ASYM_MAX_XCDS; ++x) blocks_per_xcd[x] = per[x];
  return ASYM_OK;
}

extern "C" int asym_dispatch_check(const asym_topology* topo, const uint32_t* mask,
                                   double* rr_fraction, int* blocks_per_xcd) {
  if (!rr_fraction) return asym::fail(ASYM_EINVAL, "dispatch check: null argument");
  int rot = 0;
  return dispatch_run(topo, mask, 0, rr_fraction, &rot, blocks_per_xcd);
}

extern "C" int asym_dispatch_probe(const asym_topology* topo, const uint32_t* mask, int pre_blocks,
                                   double* class_fraction, int* rotation, int* blocks_per_xcd) {
  if (!class_fraction || !rotation || pre_blocks < 0 || pre_blocks > (1 << 20))
    return asym::fail(ASYM_EINVAL, "dispatch probe: bad argument");
  return dispatch_run(topo, mask, pre_blocks, class_fraction, rotation, blocks_per_xcd);
}
