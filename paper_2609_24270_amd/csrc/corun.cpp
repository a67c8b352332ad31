// Co-running kernels on partitioned CU sets (Section 7.2: prefill and decode
// multiplexed on two SM partitions; Section 7.3: co-located tenants on equal
// SM counts whose physical placement differs).  Each task gets its own stream:
// a hardware CU-masked queue when the task names a CU mask, an unmasked queue
// with the kernels' own XCD filter when it names whole XCDs.  Tasks are
// enqueued back to back, after one untimed launch of each GEMM (its one-time
// setup), and timed with events on their own streams.  The bandwidth-bound
// tenants are a streaming copy and a whole-buffer reader, each a fixed number
// of passes (no tenant runs "until the others end": a tenant that waits for a
// persistent GEMM to finish, while that GEMM's workgroups dealt to the
// tenant's XCDs wait for the tenant's CUs, never ends).
#include <hip/hip_runtime.h>

#include <cstring>
#include <vector>

#include "internal.h"

struct asym_topology;

namespace asym {
int gemm_bf16(const asym_topology* topo, int M, int N, int K, const void* A, int lda,
              const void* B, int ldb, int b_layout, void* C, int ldc, int mapping,
              uint32_t xcd_mask, hipStream_t stream);
}

using asym::fail;

namespace {

struct Guard {  // releases streams, events and sinks on every exit path
  std::vector<hipStream_t> streams;
  std::vector<hipEvent_t> events;
  std::vector<void*> sinks;
  ~Guard() {
    for (hipStream_t s : streams) (void)hipStreamSynchronize(s);
    for (hipEvent_t e : events) (void)hipEventDestroy(e);
    for (hipStream_t s : streams) asym_stream_destroy(s);
    for (void* p : sinks) (void)hipFree(p);
  }
};

bool mask_empty(const uint32_t* m) {
  for (int i = 0; i < ASYM_MASK_WORDS; ++i)
    if (m[i]) return false;
  return true;
}

}  // namespace

extern "C" int asym_corun(const asym_topology* topo, const asym_task* tasks, int n_tasks,
                          asym_task_result* out) {
  if (!tasks || !out || n_tasks < 1 || n_tasks > 16) return fail(ASYM_EINVAL, "corun: bad task list");
  std::memset(out, 0, sizeof(asym_task_result) * n_tasks);
  Guard g;
  for (int i = 0; i < n_tasks; ++i) {
    const asym_task& t = tasks[i];
    if (t.warm_iters < 0) return fail(ASYM_EINVAL, "corun: warm_iters must be >= 0");
    if (t.kind == 0) {
      if (t.iters < 1 || !t.A || !t.B || !t.C) return fail(ASYM_EINVAL, "corun: bad GEMM task");
    } else if (t.kind == 1) {
      if (!t.src || !t.dst || t.n_bytes < 16 || t.n_bytes % 16)
        return fail(ASYM_EINVAL, "corun: a copy task needs a source and destination of a multiple of 16 bytes");
      const char* sp = static_cast<const char*>(t.src);
      const char* dp = static_cast<const char*>(t.dst);
      if (sp < dp + t.n_bytes && dp < sp + t.n_bytes)
        return fail(ASYM_EINVAL, "corun: a copy task's source and destination overlap");
      if (((uintptr_t)t.src & 15u) || ((uintptr_t)t.dst & 15u))
        return fail(ASYM_EINVAL, "corun: a copy task's buffers must be 16-byte aligned");
      if (t.iters < 1)
        return fail(ASYM_EINVAL,
                    "corun: a copy task runs a fixed number of passes (iters >= 1); an open-ended copy beside a "
                    "persistent GEMM can deadlock (the GEMM's workgroups dealt to the copy's XCDs wait for its CUs)");
    } else if (t.kind == 2) {
      if (!t.src || t.n_bytes < 16 || t.n_bytes % 16 || t.iters < 1)
        return fail(ASYM_EINVAL, "corun: a read task needs a source of a multiple of 16 bytes and iters >= 1");
    } else {
      return fail(ASYM_EINVAL, "corun: unknown task kind");
    }
    void* s = nullptr;
    int rc = asym_stream_create(topo, mask_empty(t.mask) ? nullptr : t.mask, &s);
    if (rc != ASYM_OK) return rc;
    g.streams.push_back(static_cast<hipStream_t>(s));
  }
  int n_x = 0, dev = 0;
  ASYM_HIP(hipGetDevice(&dev));
  ASYM_HIP(hipDeviceGetAttribute(&n_x, hipDeviceAttributeNumberOfXccs, dev));
  // copy and read tasks: the working CUs per XCD (the task's mask, or every
  // CU, less the XCDs its filter leaves out) and the grid
  std::vector<std::vector<int>> read_cus(n_tasks);
  std::vector<int> read_grid(n_tasks, 0);
  std::vector<void*> sink(n_tasks, nullptr);
  for (int i = 0; i < n_tasks; ++i) {
    const asym_task& t = tasks[i];
    if (t.kind != 1 && t.kind != 2) continue;
    if (n_x < 1 || n_x > 16 || (t.xcd_mask >> n_x) != 0u)
      return fail(ASYM_EINVAL, "corun: a copy or read task's XCD filter names an XCD the device does not have");
    if (t.grid < 0 || t.grid > (1 << 20))
      return fail(ASYM_EINVAL, "corun: a copy or read task's grid must be in [0, 2^20]");
    std::vector<int>& cus = read_cus[i];
    cus.assign(ASYM_MAX_XCDS, 0);
    if (!mask_empty(t.mask)) {
      int rc = asym_cuset_counts(topo, t.mask, cus.data());
      if (rc != ASYM_OK) return rc;
    } else if (topo) {
      int rc = asym_topology_info(topo, nullptr, nullptr, cus.data(), nullptr);
      if (rc != ASYM_OK) return rc;
    } else {
      int n_cus = 0;
      ASYM_HIP(hipDeviceGetAttribute(&n_cus, hipDeviceAttributeMultiprocessorCount, dev));
      for (int x = 0; x < n_x; ++x) cus[x] = n_cus / n_x;
    }
    for (int x = 0; x < n_x; ++x)
      if (t.xcd_mask && !((t.xcd_mask >> x) & 1u)) cus[x] = 0;
    int any = 0;
    for (int x = 0; x < n_x; ++x) any += cus[x];
    if (!any) return fail(ASYM_EINVAL, "corun: a copy or read task's XCD filter leaves it no CU");
    if (t.kind == 1) {
      read_grid[i] = t.grid > 0 ? t.grid : asym::copy_grid(cus.data(), n_x);
      continue;
    }
    read_grid[i] = t.grid > 0 ? t.grid : asym::stream_read_grid(cus.data(), n_x);
    ASYM_HIP(hipMalloc(&sink[i], (size_t)read_grid[i] * 256 * 16));
    g.sinks.push_back(sink[i]);
  }
  bool warm = false;
  for (int i = 0; i < n_tasks; ++i) warm |= tasks[i].warm_iters > 0;
  std::vector<hipEvent_t> ev0(n_tasks), ev1(n_tasks), evw(n_tasks);
  for (int i = 0; i < n_tasks; ++i) {
    ASYM_HIP(hipEventCreate(&ev0[i]));
    g.events.push_back(ev0[i]);
    ASYM_HIP(hipEventCreate(&ev1[i]));
    g.events.push_back(ev1[i]);
    ASYM_HIP(hipEventCreateWithFlags(&evw[i], hipEventDisableTiming));
    g.events.push_back(evw[i]);
  }
  // `n` launches (GEMM) or passes (copy, read) of task i on its stream
  auto enqueue = [&](int i, int n) -> int {
    const asym_task& t = tasks[i];
    hipStream_t s = g.streams[i];
    if (n < 1) return ASYM_OK;
    if (t.kind == 2)
      return asym::launch_stream_read(t.src, t.n_bytes, n, sink[i], read_grid[i], read_cus[i].data(), n_x, s);
    if (t.kind == 1)
      return asym::launch_copy(t.dst, t.src, t.n_bytes, n, nullptr, read_cus[i].data(), n_x, read_grid[i], s);
    for (int it = 0; it < n; ++it) {
      int rc = asym::gemm_bf16(topo, t.M, t.N, t.K, t.A, t.K, t.B, t.K, ASYM_B_NK, t.C, t.N, t.mapping,
                               t.xcd_mask, s);
      if (rc != ASYM_OK) return rc;
    }
    return ASYM_OK;
  };
  // one untimed launch of every GEMM task on its own stream before the
  // release: its first launch on a new stream or CU set does one-time setup
  // (workspace, schedule upload) that waits on its stream, which must not
  // happen while the other tasks already run
  for (int i = 0; i < n_tasks; ++i) {
    const asym_task& t = tasks[i];
    if (t.kind != 0) continue;
    int rc = asym::gemm_bf16(topo, t.M, t.N, t.K, t.A, t.K, t.B, t.K, ASYM_B_NK, t.C, t.N, t.mapping,
                             t.xcd_mask, g.streams[i]);
    if (rc != ASYM_OK) return rc;
  }
  ASYM_HIP(hipDeviceSynchronize());

  // warm-up: every task's untimed part, then each stream waits for all of
  // them (no cycle: each stream records its event before its own waits)
  if (warm) {
    for (int pass = 0; pass < 2; ++pass)
      for (int i = 0; i < n_tasks; ++i) {
        if ((pass == 0) != (tasks[i].kind != 0)) continue;
        int rc = enqueue(i, tasks[i].warm_iters);
        if (rc != ASYM_OK) return rc;
        ASYM_HIP(hipEventRecord(evw[i], g.streams[i]));
      }
    for (int i = 0; i < n_tasks; ++i)
      for (int j = 0; j < n_tasks; ++j)
        if (j != i) ASYM_HIP(hipStreamWaitEvent(g.streams[i], evw[j], 0));
  }
  // copies and reads first, so they are streaming when the GEMMs start
  for (int pass = 0; pass < 2; ++pass) {
    for (int i = 0; i < n_tasks; ++i) {
      const asym_task& t = tasks[i];
      if ((pass == 0) != (t.kind != 0)) continue;
      ASYM_HIP(hipEventRecord(ev0[i], g.streams[i]));
      int rc = enqueue(i, t.iters);
      if (rc != ASYM_OK) return rc;
      ASYM_HIP(hipEventRecord(ev1[i], g.streams[i]));
    }
  }
  for (int i = 0; i < n_tasks; ++i) ASYM_HIP(hipEventSynchronize(ev1[i]));
  for (int i = 0; i < n_tasks; ++i) {
    float ms = 0.f;
    ASYM_HIP(hipEventElapsedTime(&ms, ev0[i], ev1[i]));
    asym_task_result& r = out[i];
    const asym_task& t = tasks[i];
    r.ms_total = ms;
    if (t.kind == 0) {
      r.iters_done = t.iters;
      r.ms_per_iter = ms / t.iters;
      r.tflops = 2.0 * t.M * t.N * (double)t.K * t.iters / (ms * 1e-3) / 1e12;
    } else if (t.kind == 1) {
      r.iters_done = t.iters;
      r.ms_per_iter = ms / t.iters;
      r.gbps = 2.0 * (double)t.n_bytes * t.iters / (ms * 1e-3) / 1e9;
    } else if (t.kind == 2) {
      r.iters_done = t.iters;
      r.ms_per_iter = ms / t.iters;
      r.gbps = (double)t.n_bytes * t.iters / (ms * 1e-3) / 1e9;
      std::vector<uint32_t> h((size_t)read_grid[i] * 256 * 4);
      ASYM_HIP(hipMemcpy(h.data(), sink[i], sizeof(uint32_t) * h.size(), hipMemcpyDeviceToHost));
      for (size_t w = 0; w < h.size(); ++w) r.checksum[w & 3] ^= h[w];
    }
  }
  return ASYM_OK;
}
