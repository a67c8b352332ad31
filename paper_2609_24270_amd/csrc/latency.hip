// Per-XCD memory latency probe (Section 6.1 access latency distribution,
// Appendix C kernel details, Appendix G per-XCD probing on an AMD part).
//
// One lane of one workgroup on the chosen XCD walks a list of sampled
// 128-byte lines and times each load on its own: the load is issued between
// two reads of the shader clock (s_memtime), with every earlier memory access
// drained first, so one line's latency is one window.  The workgroup learns
// its XCD from the XCC_ID register; the launch has several workgroups per XCD
// and the first one on the wanted XCD to take a ticket does the walk, the
// rest exit at once.  Before each timed load the lane loads another line of
// the same 2 MiB page (translation warm-up, outside the window); the host
// picks that line's distance so that it is never a line timed later in the
// same walk.
//
// Regimes are set up around the walk by the host: an untimed walk by the same
// XCD first (L2), or a cache flush followed by an untimed walk on another XCD
// (memory-side cache), or a flush alone (HBM).  The flush is a fill of a
// buffer four times the memory-side cache by the runtime's fill kernel, which
// runs on every XCD.  Every loop here is bounded by the sample count.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cstring>
#include <vector>

#include "internal.h"

namespace asym {
namespace {

constexpr int kModeTimed = 0;
constexpr int kModeWarm = 1;
constexpr uint64_t kPage = 2ull << 20;       // translation page assumed by the warm-up touch
constexpr uint64_t kTouchDelta = kPage / 2;  // the touched line: same page, other half
constexpr size_t kFlushBytes = 1ull << 30;   // 4 x the 256 MiB memory-side cache

struct LatArgs {
  const char* base;
  const uint64_t* offs;   // [n] byte offsets of the sampled lines
  uint32_t* lat;          // [n] timed windows (timed mode)
  uint64_t* info;         // [8]: sink, memtime0, memtime1, realtime0, realtime1,
                          //      min empty window, done, xcc
  int* ticket;            // zero before the launch
  uint64_t touch;         // translation warm-up: the line at offset ^ touch
  int n;
  int target;             // XCC that runs the walk
  int mode;
};

__global__ void __launch_bounds__(64) latency_kernel(LatArgs a) {
  uint32_t xcc;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
  if ((int)(xcc & 0xFu) != a.target || threadIdx.x != 0) return;
  if (atomicAdd(a.ticket, 1) != 0) return;

  uint64_t ov = ~0ull;
  for (int r = 0; r < 32; ++r) {
    uint64_t t0, t1;
    asm volatile(
        "s_waitcnt vmcnt(0) lgkmcnt(0)\n\t"
        "s_memtime %0\n\t"
        "s_waitcnt lgkmcnt(0)\n\t"
        "s_memtime %1\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&s"(t0), "=&s"(t1)::"memory");
    ov = t1 - t0 < ov ? t1 - t0 : ov;
  }
  const uint64_t mt0 = __builtin_amdgcn_s_memtime();
  const uint64_t rt0 = __builtin_amdgcn_s_memrealtime();
  uint32_t sink = 0;
  for (int i = 0; i < a.n; ++i) {
    const uint64_t off = a.offs[i];
    const uint32_t* p = reinterpret_cast<const uint32_t*>(a.base + off);
    if (a.mode == kModeTimed) {
      const uint32_t* q = reinterpret_cast<const uint32_t*>(a.base + (off ^ a.touch));
      uint32_t w, v;
      uint64_t t0, t1;
      asm volatile(
          "global_load_dword %0, %1, off\n\t"
          "s_waitcnt vmcnt(0)"
          : "=v"(w)
          : "v"(q)
          : "memory");
      asm volatile(
          "s_waitcnt vmcnt(0) lgkmcnt(0)\n\t"
          "s_memtime %[t0]\n\t"
          "s_waitcnt lgkmcnt(0)\n\t"
          "global_load_dword %[v], %[p], off\n\t"
          "s_waitcnt vmcnt(0)\n\t"
          "s_memtime %[t1]\n\t"
          "s_waitcnt lgkmcnt(0)"
          : [t0] "=&s"(t0), [t1] "=&s"(t1), [v] "=&v"(v)
          : [p] "v"(p)
          : "memory");
      a.lat[i] = (uint32_t)(t1 - t0);
      sink += v ^ w;
    } else {
      uint32_t v;
      asm volatile(
          "global_load_dword %0, %1, off\n\t"
          "s_waitcnt vmcnt(0)"
          : "=v"(v)
          : "v"(p)
          : "memory");
      sink += v;
    }
  }
  const uint64_t mt1 = __builtin_amdgcn_s_memtime();
  const uint64_t rt1 = __builtin_amdgcn_s_memrealtime();
  a.info[0] = sink;
  a.info[1] = mt0;
  a.info[2] = mt1;
  a.info[3] = rt0;
  a.info[4] = rt1;
  a.info[5] = ov;
  a.info[7] = xcc;
  __threadfence();
  a.info[6] = 1;
}

uint64_t splitmix64(uint64_t& s) {
  uint64_t z = (s += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

struct DevBufs {  // frees on every exit path
  void* p[6] = {nullptr, nullptr, nullptr, nullptr, nullptr, nullptr};
  hipStream_t s = nullptr;
  ~DevBufs() {
    if (s) (void)hipStreamSynchronize(s);
    for (void* q : p)
      if (q) (void)hipFree(q);
    if (s) (void)hipStreamDestroy(s);
  }
};

int validate(const asym_latency_params& p) {
  if (p.n_samples < 1 || p.n_samples > (1 << 22))
    return fail(ASYM_EINVAL, "latency probe: n_samples must be in [1, 4194304]");
  if (p.passes < 1 || p.passes > 64) return fail(ASYM_EINVAL, "latency probe: passes must be in [1, 64]");
  if (p.l2_samples < 0 || p.l2_samples > p.n_samples || p.l2_samples > 8192)
    return fail(ASYM_EINVAL, "latency probe: l2_samples must be in [0, min(n_samples, 8192)]");
  if (p.alloc_bytes != 0 && p.alloc_bytes < (64ull << 20))
    return fail(ASYM_EINVAL, "latency probe: alloc_bytes must be 0 or at least 64 MiB");
  if (!(p.tie_cycles >= 0.0) || !(p.group_threshold > -1.0 && p.group_threshold < 1.0))
    return fail(ASYM_EINVAL, "latency probe: threshold must be in (-1, 1), tie margin >= 0");
  return ASYM_OK;
}

}  // namespace

int latency_measure(int device, LatencyMeasure& m) {
  ASYM_HIP(hipSetDevice(device));
  int n_x = 0, wall_khz = 0;
  ASYM_HIP(hipDeviceGetAttribute(&n_x, hipDeviceAttributeNumberOfXccs, device));
  ASYM_HIP(hipDeviceGetAttribute(&wall_khz, hipDeviceAttributeWallClockRate, device));
  if (n_x < 1 || n_x > ASYM_MAX_XCDS) return fail(ASYM_EUNSUPPORTED, "latency probe: XCD count");
  const int n_s = (int)m.offs.size();
  if (n_s < 1 || m.alloc % kPage || m.alloc == 0 || m.passes < 1 || m.l2_samples < 0 ||
      m.l2_samples > n_s || (reinterpret_cast<uintptr_t>(m.ext_base) % kPage))
    return fail(ASYM_EINVAL, "latency probe: bad measurement set-up");
  for (uint64_t o : m.offs)
    if (o % 128 || o >= m.alloc || (o ^ m.touch_delta) >= m.alloc || ((o ^ m.touch_delta) % 128))
      return fail(ASYM_EINVAL, "latency probe: offset or its translation touch outside the allocation");

  DevBufs b;
  ASYM_HIP(hipStreamCreateWithFlags(&b.s, hipStreamNonBlocking));
  uintptr_t base;
  if (m.ext_base) {
    base = reinterpret_cast<uintptr_t>(m.ext_base);
  } else {
    // one page more than asked, so the walked range can start on a 2 MiB boundary
    ASYM_HIP(hipMalloc(&b.p[0], m.alloc + kPage));
    ASYM_HIP(hipMemset(b.p[0], 0, m.alloc + kPage));
    const uintptr_t raw = reinterpret_cast<uintptr_t>(b.p[0]);
    base = (raw + kPage - 1) & ~(uintptr_t)(kPage - 1);
  }
  ASYM_HIP(hipMalloc(&b.p[1], kFlushBytes));
  ASYM_HIP(hipMalloc(&b.p[2], sizeof(uint64_t) * n_s));
  ASYM_HIP(hipMalloc(&b.p[3], sizeof(uint32_t) * n_s));
  ASYM_HIP(hipMalloc(&b.p[4], sizeof(uint64_t) * 8));
  ASYM_HIP(hipMalloc(&b.p[5], sizeof(int) * 4));
  ASYM_HIP(hipMemcpy(b.p[2], m.offs.data(), sizeof(uint64_t) * n_s, hipMemcpyHostToDevice));
  m.base_align = base & (~base + 1);

  LatArgs a;
  a.base = reinterpret_cast<const char*>(base);
  a.offs = static_cast<const uint64_t*>(b.p[2]);
  a.lat = static_cast<uint32_t*>(b.p[3]);
  a.info = static_cast<uint64_t*>(b.p[4]);
  a.ticket = static_cast<int*>(b.p[5]);
  a.touch = m.touch_delta;

  m.n_x = n_x;
  m.best.assign((size_t)3 * n_x * n_s, UINT32_MAX);
  std::vector<uint32_t> host(n_s);
  uint64_t ov_min = ~0ull, d_mt = 0, d_rt = 0;
  int flush_value = 1;

  auto walk = [&](int target, int mode, int n, uint32_t* keep) -> int {
    if (n < 1) return ASYM_OK;
    a.target = target;
    a.mode = mode;
    a.n = n;
    ASYM_HIP(hipMemsetAsync(a.ticket, 0, sizeof(int) * 4, b.s));
    ASYM_HIP(hipMemsetAsync(a.info, 0, sizeof(uint64_t) * 8, b.s));
    hipLaunchKernelGGL(latency_kernel, dim3(8 * n_x), dim3(64), 0, b.s, a);
    ASYM_HIP(hipGetLastError());
    ASYM_HIP(hipStreamSynchronize(b.s));
    uint64_t info[8];
    ASYM_HIP(hipMemcpy(info, a.info, sizeof info, hipMemcpyDeviceToHost));
    if (info[6] != 1 || (int)(info[7] & 0xF) != target)
      return fail(ASYM_ETIMEOUT, "latency probe: no workgroup ran on XCD " + std::to_string(target));
    if (mode == kModeTimed) {
      ov_min = std::min(ov_min, info[5]);
      d_mt += info[2] - info[1];
      d_rt += info[4] - info[3];
      ASYM_HIP(hipMemcpy(host.data(), a.lat, sizeof(uint32_t) * n, hipMemcpyDeviceToHost));
      for (int i = 0; i < n; ++i) keep[i] = std::min(keep[i], host[i]);
    }
    return ASYM_OK;
  };
  auto flush = [&]() -> int {
    ASYM_HIP(hipMemsetAsync(b.p[1], flush_value++ & 0xFF, kFlushBytes, b.s));
    return ASYM_OK;
  };

  int rc = ASYM_OK;
  for (int pass = 0; pass < m.passes; ++pass) {
    for (int x = 0; x < n_x; ++x) {
      uint32_t* l2 = &m.best[((size_t)0 * n_x + x) * n_s];
      uint32_t* mall = &m.best[((size_t)1 * n_x + x) * n_s];
      uint32_t* hbm = &m.best[((size_t)2 * n_x + x) * n_s];
      // L2: the same XCD loads the lines, then times them
      if (m.l2_samples > 0 && ((rc = flush()) || (rc = walk(x, kModeWarm, m.l2_samples, nullptr)) ||
                               (rc = walk(x, kModeTimed, m.l2_samples, l2))))
        return rc;
      // memory-side cache: flush, another XCD loads the lines, x times them
      if (m.mall && ((rc = flush()) || (rc = walk((x + 1) % n_x, kModeWarm, n_s, nullptr)) ||
                     (rc = walk(x, kModeTimed, n_s, mall))))
        return rc;
      // HBM: flush, x times the lines
      if ((rc = flush()) || (rc = walk(x, kModeTimed, n_s, hbm))) return rc;
    }
  }
  m.timer_overhead = (double)ov_min;
  m.clock_mhz = d_rt > 0 ? (double)d_mt / (double)d_rt * (wall_khz / 1000.0) : -1.0;
  return ASYM_OK;
}

int latency_probe(int device, const asym_latency_params& p, uint32_t* lat_out,
                  asym_latency_summary& out) {
  int rc = validate(p);
  if (rc != ASYM_OK) return rc;
  ASYM_HIP(hipSetDevice(device));
  size_t free_b = 0, total_b = 0;
  ASYM_HIP(hipMemGetInfo(&free_b, &total_b));
  size_t alloc = p.alloc_bytes ? p.alloc_bytes : (32ull << 30);
  const size_t room = free_b > kFlushBytes + (1ull << 30) ? free_b - kFlushBytes - (1ull << 30) : 0;
  if (alloc > room) {
    if (p.alloc_bytes) return fail(ASYM_ENOMEM, "latency probe: allocation larger than free memory");
    alloc = room / 2;
  }
  alloc -= alloc % kPage;
  if (alloc < (64ull << 20)) return fail(ASYM_ENOMEM, "latency probe: not enough free device memory");

  LatencyMeasure m;
  m.alloc = alloc;
  m.passes = p.passes;
  m.l2_samples = p.l2_samples;
  m.mall = true;
  m.touch_delta = kTouchDelta;
  const int n_s = p.n_samples;
  m.offs.resize(n_s);
  uint64_t st = p.seed;
  const uint64_t lines = alloc / 128;
  for (int i = 0; i < n_s; ++i) m.offs[i] = (splitmix64(st) % lines) * 128;
  if ((rc = latency_measure(device, m)) != ASYM_OK) return rc;
  const int n_x = m.n_x;
  std::vector<uint32_t>& best = m.best;

  rc = analyze_latency(&best[(size_t)2 * n_x * n_s], n_x, n_s, p.group_threshold, p.tie_cycles, out);
  if (rc != ASYM_OK) return rc;
  for (int x = 0; x < n_x; ++x) {
    double s2 = 0, sm = 0;
    for (int i = 0; i < p.l2_samples; ++i) s2 += best[((size_t)0 * n_x + x) * n_s + i];
    for (int i = 0; i < n_s; ++i) sm += best[((size_t)1 * n_x + x) * n_s + i];
    out.l2_hit[x] = p.l2_samples > 0 ? s2 / p.l2_samples : -1.0;
    out.mall_hit[x] = sm / n_s;
  }
  out.passes = p.passes;
  out.l2_samples = p.l2_samples;
  out.timer_overhead = m.timer_overhead;
  out.clock_mhz = m.clock_mhz;
  if (lat_out) {
    for (int x = 0; x < n_x; ++x)
      for (int i = p.l2_samples; i < n_s; ++i) best[((size_t)0 * n_x + x) * n_s + i] = 0;
    std::memcpy(lat_out, best.data(), sizeof(uint32_t) * best.size());
  }
  return ASYM_OK;
}

int probe_latency_run(int device, Topology& t) {
  asym_latency_params p;
  asym_latency_params_default(&p);
  asym_latency_summary s;
  const int rc = latency_probe(device, p, nullptr, s);
  if (rc != ASYM_OK) return rc;
  if (s.n_xcds != t.n_xccs)
    return fail(ASYM_EINVARIANT, "latency probe: XCD count differs from the identity map");
  t.lat = s;
  t.has_latency = true;
  return ASYM_OK;
}

}  // namespace asym

extern "C" int asym_latency_probe(int device, const asym_latency_params* p, uint32_t* lat,
                                  asym_latency_summary* out) {
  using namespace asym;
  if (!out) return fail(ASYM_EINVAL, "latency probe: null output");
  asym_latency_params q;
  if (p)
    q = *p;
  else
    asym_latency_params_default(&q);
  return latency_probe(device, q, lat, *out);
}
