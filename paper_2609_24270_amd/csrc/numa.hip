// Home map of an allocation and local / remote read bandwidth (Section 6.1:
// pages classified by partition inside a contiguous region, then a read
// kernel restricted to local or to remote pages; the appendix on NUMA-aware
// address remapping places data by the same classification).
//
// On MI355X a partition is an affinity group of XCDs (an I/O die and its
// memory).  The map times one line per 2 MiB page from every XCD and extends
// the page's home to its chunks with the partition hash's in-page bits.  The
// read kernel is a plain strided reader: workgroup b runs on XCD b mod n (the
// hardware's round-robin dispatch) and walks that XCD's chunk list with a
// fixed stride, so it has no atomics, no barriers and a bounded loop.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <vector>

#include "internal.h"

namespace asym {
namespace {

constexpr uint64_t kPage = 2ull << 20;
constexpr int kReadThreads = 256;
constexpr int kReadWorkersPerXcd = 256;  // 8 workgroups per CU at 32 CUs per XCD

typedef unsigned v4u __attribute__((ext_vector_type(4)));

// Each lane reads the 16-byte words at lane * 16 + j * 4096 of every chunk of
// its workgroup's share; the XOR of what it read goes to sink[b * 256 + lane].
// A workgroup reads the list of the XCD it runs on (XCC_ID) and strides over
// it as the (b / n_x)-th of that XCD's workers: the workgroups of one residue
// class of block indices, which the hardware deals to one XCD (if two classes
// shared an XCD one list would be read twice and another not at all; every
// index stays inside the lists either way).
__global__ void __launch_bounds__(kReadThreads)
chunk_read_kernel(const char* __restrict__ base, int chunk_log2, const uint32_t* __restrict__ chunks,
                  const int* __restrict__ off, int n_x, v4u* __restrict__ sink) {
  const int b = blockIdx.x;
  uint32_t xr;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xr));
  const int x = (int)(xr & 0xFu);
  const int r = b / n_x;
  const int workers = gridDim.x / n_x;
  v4u acc = {0u, 0u, 0u, 0u};
  if (x < n_x) {
    const int i0 = off[x], i1 = off[x + 1];
    const int words = 1 << (chunk_log2 - 12);  // 16-byte words per lane per chunk
    for (int i = i0 + r; i < i1; i += workers) {
      const v4u* p = reinterpret_cast<const v4u*>(base + ((size_t)chunks[i] << chunk_log2)) + threadIdx.x;
#pragma unroll 4
      for (int j = 0; j < words; ++j) acc ^= p[(size_t)j * kReadThreads];
    }
  }
  sink[(size_t)b * kReadThreads + threadIdx.x] = acc;
}

// Whole-buffer reader for a bandwidth-bound co-runner: `passes` passes over
// n16 16-byte words, bounded by the pass count, no atomics or barriers.  The
// buffer is cut into one contiguous slice per reading XCD, sized in proportion
// to the CUs the reader has there (sh.cus), in XCD order.  A workgroup reads
// its XCC_ID: on an XCD with no share (outside the XCD filter, or no CUs) it
// leaves at once after its sink store; otherwise the workgroups of its residue
// class of block indices mod n_x (which the dispatcher deals to one XCD)
// stride over that XCD's slice in blocks of 8 x 256 words, each lane keeping 8
// independent 16-byte loads in flight.  If two classes shared an XCD, one
// slice would be read twice and another not at all; every index stays inside
// the buffer either way.
struct ReadShares {
  int cus[16];  // reading CUs per XCD, 0 where the reader has no share
};

constexpr int kReadUnroll = 8;

__global__ void __launch_bounds__(kReadThreads)
stream_read_kernel(const v4u* __restrict__ src, size_t n16, int passes, v4u* __restrict__ sink,
                   ReadShares sh, int n_x) {
  v4u acc = {0u, 0u, 0u, 0u};
  uint32_t x;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(x));
  x &= 0xFu;
  unsigned before = 0, total = 0;
  for (int y = 0; y < 16; ++y) {
    before += y < (int)x ? (unsigned)sh.cus[y] : 0u;
    total += (unsigned)sh.cus[y];
  }
  if (sh.cus[x] > 0 && total > 0) {
    // n16 < 2^36 and the CU sums <= 1024: the products fit in 64 bits
    const size_t lo = (size_t)((uint64_t)n16 * before / total);
    const size_t hi = (size_t)((uint64_t)n16 * (before + (unsigned)sh.cus[x]) / total);
    const unsigned cls = blockIdx.x % (unsigned)n_x;
    const unsigned members = (gridDim.x - cls + (unsigned)n_x - 1u) / (unsigned)n_x;
    constexpr size_t kBlock = (size_t)kReadUnroll * kReadThreads;
    const size_t first = lo + (size_t)(blockIdx.x / (unsigned)n_x) * kBlock + threadIdx.x;
    const size_t stride = (size_t)members * kBlock;
    for (int pass = 0; pass < passes; ++pass)
      for (size_t i = first; i < hi; i += stride) {
        v4u v[kReadUnroll];
        if (i + (size_t)(kReadUnroll - 1) * kReadThreads < hi) {
#pragma unroll
          for (int j = 0; j < kReadUnroll; ++j) v[j] = src[i + (size_t)j * kReadThreads];
        } else {  // the slice's last block
#pragma unroll
          for (int j = 0; j < kReadUnroll; ++j) {
            const size_t k = i + (size_t)j * kReadThreads;
            v[j] = k < hi ? src[k] : v4u{0u, 0u, 0u, 0u};
          }
        }
#pragma unroll
        for (int j = 0; j < kReadUnroll; ++j) acc ^= v[j];
      }
  }
  sink[(size_t)blockIdx.x * kReadThreads + threadIdx.x] = acc;
}

uint64_t mix64(uint64_t& s) {
  uint64_t z = (s += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}


struct Bufs {  // frees on every exit path
  void* p[3] = {nullptr, nullptr, nullptr};
  hipEvent_t e[2] = {nullptr, nullptr};
  ~Bufs() {
    for (void* q : p)
      if (q) (void)hipFree(q);
    for (hipEvent_t v : e)
      if (v) (void)hipEventDestroy(v);
  }
};

}  // namespace

int home_map(int device, const void* ptr, size_t bytes, uint64_t hash_mask, int chunk_log2,
             const int* grp_in, int passes, int n_verify, uint64_t seed, double tie,
             int8_t* chunk_home, asym_home_map_info& info) {
  if (!ptr || !chunk_home) return fail(ASYM_EINVAL, "home map: null pointer");
  if (reinterpret_cast<uintptr_t>(ptr) % kPage || bytes == 0 || bytes % kPage)
    return fail(ASYM_EINVAL, "home map: ptr and bytes must be nonzero multiples of 2 MiB");
  if (chunk_log2 < 12 || chunk_log2 > 21) return fail(ASYM_EINVAL, "home map: chunk_log2 must be in [12, 21]");
  if ((hash_mask & (kPage - 1)) & ((1ull << chunk_log2) - 1))
    return fail(ASYM_EINVAL, "home map: the hash has bits below the chunk size, a chunk would have two homes");
  if (passes < 1 || passes > 64 || n_verify < 0 || n_verify > (1 << 20) || !(tie >= 0.0))
    return fail(ASYM_EINVAL, "home map: passes in [1, 64], n_verify in [0, 2^20], tie >= 0");
  const size_t n_pages = bytes / kPage;
  if (n_pages > (1u << 22)) return fail(ASYM_EINVAL, "home map: range too large");
  if (!grp_in && n_pages < 16) return fail(ASYM_EINVAL, "home map: at least 16 pages to find the groups");

  LatencyMeasure m;
  m.alloc = bytes;
  m.ext_base = ptr;
  m.passes = passes;
  m.l2_samples = 0;
  m.mall = false;
  m.touch_delta = 1ull << 20;
  for (size_t p = 0; p < n_pages; ++p) m.offs.push_back(p * kPage);
  uint64_t st = seed;
  for (int v = 0; v < n_verify; ++v) m.offs.push_back((mix64(st) % (bytes / 128)) * 128);
  int rc = latency_measure(device, m);
  if (rc != ASYM_OK) return rc;
  const int n_x = m.n_x, n_s = (int)m.offs.size();
  const uint32_t* L = &m.best[(size_t)2 * n_x * n_s];
  std::vector<int> grp(n_x);
  if (grp_in) {
    std::copy(grp_in, grp_in + n_x, grp.begin());
  } else {
    asym_latency_summary s;
    if ((rc = analyze_latency(L, n_x, n_s, 0.5, tie, s)) != ASYM_OK) return rc;
    if (s.n_groups != 2)
      return fail(ASYM_EUNSUPPORTED, "home map: the timed lines show " + std::to_string(s.n_groups) +
                                         " XCD groups, not two");
    for (int x = 0; x < n_x; ++x) grp[x] = s.group_of_xcd[x];
  }
  return home_map_analyze(L, n_x, (int)n_pages, m.offs.data() + n_pages, n_verify, grp.data(), hash_mask,
                          chunk_log2, tie, chunk_home, info);
}

int chunk_read_bw(const void* base, size_t bytes, int chunk_log2, const uint32_t* chunks, const int* off,
                  int n_x, int iters, hipStream_t s, uint32_t* checksum, double* ms, int workers_per_xcd) {
  if (!base || !chunks || !off || !ms) return fail(ASYM_EINVAL, "chunk read: null pointer");
  if (reinterpret_cast<uintptr_t>(base) % 16) return fail(ASYM_EINVAL, "chunk read: base must be 16-byte aligned");
  if (chunk_log2 < 12 || chunk_log2 > 21) return fail(ASYM_EINVAL, "chunk read: chunk_log2 must be in [12, 21]");
  if (iters < 1 || iters > 10000) return fail(ASYM_EINVAL, "chunk read: iters must be in [1, 10000]");
  if (workers_per_xcd < 1 || workers_per_xcd > 4096)
    return fail(ASYM_EINVAL, "chunk read: workers per XCD must be in [1, 4096]");
  int dev = 0, dev_x = 0;
  ASYM_HIP(hipGetDevice(&dev));
  ASYM_HIP(hipDeviceGetAttribute(&dev_x, hipDeviceAttributeNumberOfXccs, dev));
  if (n_x != dev_x) return fail(ASYM_EINVAL, "chunk read: n_xcds must be the device's XCD count");
  const uint64_t n_chunks = bytes >> chunk_log2;
  if (off[0] != 0) return fail(ASYM_EINVAL, "chunk read: off[0] must be 0");
  for (int x = 0; x < n_x; ++x)
    if (off[x + 1] < off[x]) return fail(ASYM_EINVAL, "chunk read: off must not decrease");
  const int n = off[n_x];
  for (int i = 0; i < n; ++i)
    if (chunks[i] >= n_chunks) return fail(ASYM_EINVAL, "chunk read: chunk index beyond the range");

  const int grid = n_x * workers_per_xcd;
  Bufs b;
  ASYM_HIP(hipMalloc(&b.p[0], sizeof(uint32_t) * std::max(n, 1)));
  ASYM_HIP(hipMalloc(&b.p[1], sizeof(int) * (n_x + 1)));
  ASYM_HIP(hipMalloc(&b.p[2], sizeof(v4u) * (size_t)grid * kReadThreads));
  if (n) ASYM_HIP(hipMemcpy(b.p[0], chunks, sizeof(uint32_t) * n, hipMemcpyHostToDevice));
  ASYM_HIP(hipMemcpy(b.p[1], off, sizeof(int) * (n_x + 1), hipMemcpyHostToDevice));
  ASYM_HIP(hipEventCreate(&b.e[0]));
  ASYM_HIP(hipEventCreate(&b.e[1]));
  const char* cb = static_cast<const char*>(base);
  auto launch = [&]() -> int {
    hipLaunchKernelGGL(chunk_read_kernel, dim3(grid), dim3(kReadThreads), 0, s, cb, chunk_log2,
                       static_cast<const uint32_t*>(b.p[0]), static_cast<const int*>(b.p[1]), n_x,
                       static_cast<v4u*>(b.p[2]));
    ASYM_HIP(hipGetLastError());
    return ASYM_OK;
  };
  int rc = launch();  // untimed first pass
  if (rc != ASYM_OK) return rc;
  ASYM_HIP(hipEventRecord(b.e[0], s));
  for (int it = 0; it < iters; ++it)
    if ((rc = launch()) != ASYM_OK) return rc;
  ASYM_HIP(hipEventRecord(b.e[1], s));
  ASYM_HIP(hipEventSynchronize(b.e[1]));
  float t = 0.f;
  ASYM_HIP(hipEventElapsedTime(&t, b.e[0], b.e[1]));
  *ms = (double)t / iters;
  if (checksum) {
    std::vector<v4u> h((size_t)grid * kReadThreads);
    ASYM_HIP(hipMemcpy(h.data(), b.p[2], sizeof(v4u) * h.size(), hipMemcpyDeviceToHost));
    v4u acc = {0u, 0u, 0u, 0u};
    for (const v4u& v : h) acc ^= v;
    for (int w = 0; w < 4; ++w) checksum[w] = acc[w];
  }
  return ASYM_OK;
}

// The reader's grid for reading CUs cus[x] per XCD: the same count w on every
// XCD (workgroups are dealt round-robin), 8 workgroups of 4 waves per CU of
// the XCD with the most reading CUs (its slice is the largest).  XCDs with
// fewer CUs hold their workgroups in the queue until CUs free up; XCDs with no
// share see theirs leave at once.
int stream_read_grid(const int* cus, int n_x) {
  int hi = 0;
  for (int x = 0; x < n_x; ++x) hi = std::max(hi, cus[x]);
  return n_x * std::max(1, 8 * hi);
}

int launch_stream_read(const void* src, size_t n_bytes, int passes, void* sink, int grid, const int* cus,
                       int n_x, hipStream_t s) {
  if (!src || !sink || !cus || n_bytes < 16 || n_bytes % 16 || (n_bytes >> 40) || passes < 1 || grid < 1 ||
      n_x < 1 || n_x > 16)
    return fail(ASYM_EINVAL, "stream read: bad arguments");
  ReadShares sh{};
  int any = 0;
  for (int x = 0; x < n_x; ++x) {
    if (cus[x] < 0 || cus[x] > 64) return fail(ASYM_EINVAL, "stream read: bad CU count");
    sh.cus[x] = cus[x];
    any += cus[x];
  }
  if (!any) return fail(ASYM_EINVAL, "stream read: no reading CU");
  hipLaunchKernelGGL(stream_read_kernel, dim3(grid), dim3(kReadThreads), 0, s, static_cast<const v4u*>(src),
                     n_bytes / 16, passes, static_cast<v4u*>(sink), sh, n_x);
  ASYM_HIP(hipGetLastError());
  return ASYM_OK;
}

}  // namespace asym

extern "C" int asym_home_map(int device, const void* ptr, size_t bytes, uint64_t hash_mask, int chunk_log2,
                             const int* group_of_xcd, int passes, int n_verify, uint64_t seed,
                             double tie_cycles, int8_t* chunk_home, asym_home_map_info* info) {
  if (!info) return asym::fail(ASYM_EINVAL, "home map: null info");
  return asym::home_map(device, ptr, bytes, hash_mask, chunk_log2, group_of_xcd, passes, n_verify, seed,
                        tie_cycles, chunk_home, *info);
}

extern "C" int asym_chunk_read_bw(const void* base, size_t bytes, int chunk_log2, const uint32_t* chunks,
                                  const int* off, int n_xcds, int iters, void* stream,
                                  uint32_t* checksum_out, double* ms_per_iter) {
  return asym::chunk_read_bw(base, bytes, chunk_log2, chunks, off, n_xcds, iters,
                             static_cast<hipStream_t>(stream), checksum_out, ms_per_iter,
                             asym::kReadWorkersPerXcd);
}

extern "C" int asym_chunk_read(const void* base, size_t bytes, int chunk_log2, const uint32_t* chunks,
                               const int* off, int n_xcds, int workers_per_xcd, int iters, void* stream,
                               uint32_t* checksum_out, double* ms_per_iter) {
  return asym::chunk_read_bw(base, bytes, chunk_log2, chunks, off, n_xcds, iters,
                             static_cast<hipStream_t>(stream), checksum_out, ms_per_iter, workers_per_xcd);
}
