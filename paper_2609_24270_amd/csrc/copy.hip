// Streaming copy, the bandwidth-bound co-runner of the co-location study
// (Section 7.3 places a second tenant on the complementary units; here that
// tenant is an HBM-bound copy, so the GEMM's CU set competes for memory
// bandwidth and power as real co-located work does).
//
// dst[i] = src[i] with 16-byte accesses from every lane.  The work is fixed
// before launch and nothing is shared between workgroups: the buffer is cut
// into one slice per XCD, in proportion to the copy's CUs on that XCD, and a
// slice is copied by the workgroups the hardware deals to that XCD (one
// residue class of block indices), each striding by the class's size.  There
// are no atomics, no LDS and no barriers; every loop has a trip count fixed by
// the arguments (at most `passes` passes over at most the slice), so every
// wave ends and the grid drains whatever the other tenants do.  An optional
// stop flag, read by each wave before every pass after the first, can end the
// copy earlier; it never extends it.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "internal.h"

namespace asym {
namespace {

constexpr int kCopyThreads = 256;
constexpr int kCopyUnroll = 4;  // 16-byte words in flight per lane
typedef unsigned v4u __attribute__((ext_vector_type(4)));

struct CopyShares {
  int cus[ASYM_MAX_XCDS];  // the copy's CUs per XCD (0: no slice there)
};

__global__ void __launch_bounds__(kCopyThreads)
copy_kernel(v4u* __restrict__ dst, const v4u* __restrict__ src, size_t n16, int passes,
            const int* stop_flag, CopyShares sh, int n_x) {
  uint32_t x;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(x));
  x &= 0xFu;
  if ((int)x >= n_x) return;
  unsigned before = 0, total = 0;
  for (int y = 0; y < n_x; ++y) {
    before += y < (int)x ? (unsigned)sh.cus[y] : 0u;
    total += (unsigned)sh.cus[y];
  }
  if (sh.cus[x] <= 0 || total == 0) return;
  // n16 < 2^40 and the CU sums <= 1024: the products fit in 64 bits
  const size_t lo = (size_t)((uint64_t)n16 * before / total);
  const size_t hi = (size_t)((uint64_t)n16 * (before + (unsigned)sh.cus[x]) / total);
  const unsigned cls = blockIdx.x % (unsigned)n_x;
  const unsigned members = (gridDim.x - cls + (unsigned)n_x - 1u) / (unsigned)n_x;
  constexpr size_t kBlock = (size_t)kCopyUnroll * kCopyThreads;
  const size_t first = lo + (size_t)(blockIdx.x / (unsigned)n_x) * kBlock + threadIdx.x;
  const size_t stride = (size_t)members * kBlock;
  for (int pass = 0; pass < passes; ++pass) {
    if (pass > 0 && stop_flag &&
        __hip_atomic_load(stop_flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM) != 0)
      break;
    for (size_t i = first; i < hi; i += stride) {
      v4u v[kCopyUnroll];
      if (i + (size_t)(kCopyUnroll - 1) * kCopyThreads < hi) {
#pragma unroll
        for (int j = 0; j < kCopyUnroll; ++j) v[j] = __builtin_nontemporal_load(src + i + (size_t)j * kCopyThreads);
#pragma unroll
        for (int j = 0; j < kCopyUnroll; ++j) __builtin_nontemporal_store(v[j], dst + i + (size_t)j * kCopyThreads);
      } else {  // the slice's last block
#pragma unroll
        for (int j = 0; j < kCopyUnroll; ++j) {
          const size_t k = i + (size_t)j * kCopyThreads;
          if (k < hi) __builtin_nontemporal_store(__builtin_nontemporal_load(src + k), dst + k);
        }
      }
    }
  }
}

// Up to kPutWords 4-byte words carried in the kernel's arguments, written to
// device memory: host data reaches the device without a staging buffer or a
// copy engine (the runtime copies kernel arguments itself).
constexpr int kPutWords = 960;
struct PutWords {
  int w[kPutWords];
};

__global__ void put_words_kernel(int* __restrict__ dst, int n, PutWords src) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) dst[i] = src.w[i];
}

__global__ void zero_words_kernel(uint32_t* p, size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

}  // namespace

int copy_grid(const int* cus, int n_x) {
  int hi = 0;
  for (int x = 0; x < n_x; ++x) hi = std::max(hi, cus[x]);
  return n_x * std::max(1, 8 * hi);
}

int launch_copy(void* dst, const void* src, size_t n_bytes, int passes, const int* stop_flag,
                const int* cus, int n_x, int grid, hipStream_t s) {
  if (!dst || !src || !cus || n_bytes < 16 || n_bytes % 16 || (n_bytes >> 40) || passes < 1 || grid < 1 ||
      n_x < 1 || n_x > ASYM_MAX_XCDS)
    return fail(ASYM_EINVAL, "copy: bad arguments");
  CopyShares sh{};
  int any = 0;
  for (int x = 0; x < n_x; ++x) {
    if (cus[x] < 0 || cus[x] > 64) return fail(ASYM_EINVAL, "copy: bad CU count");
    sh.cus[x] = cus[x];
    any += cus[x];
  }
  if (!any) return fail(ASYM_EINVAL, "copy: no copying CU");
  hipLaunchKernelGGL(copy_kernel, dim3(grid), dim3(kCopyThreads), 0, s, static_cast<v4u*>(dst),
                     static_cast<const v4u*>(src), n_bytes / 16, passes, stop_flag, sh, n_x);
  ASYM_HIP(hipGetLastError());
  return ASYM_OK;
}

// dst[0 .. n) = host[0 .. n), ordered on stream s, through kernel arguments
// (ceil(n / 960) launches).
int launch_put_words(int* dst, const int* host, size_t n, hipStream_t s) {
  if (!n) return ASYM_OK;
  if (!dst || !host) return fail(ASYM_EINVAL, "put words: null pointer");
  for (size_t i = 0; i < n; i += kPutWords) {
    const int m = (int)std::min<size_t>(kPutWords, n - i);
    PutWords w{};
    for (int j = 0; j < m; ++j) w.w[j] = host[i + j];
    hipLaunchKernelGGL(put_words_kernel, dim3(1), dim3(256), 0, s, dst + i, m, w);
    ASYM_HIP(hipGetLastError());
  }
  return ASYM_OK;
}

// Stream-ordered zero fill of n 4-byte words (a kernel, not a memset node, so
// that it also behaves under graph capture).
int launch_zero_words(void* p, size_t n, hipStream_t s) {
  if (!p || !n) return ASYM_OK;
  const int grid = (int)std::min<size_t>((n + 255) / 256, 1024);
  hipLaunchKernelGGL(zero_words_kernel, dim3(grid), dim3(256), 0, s, static_cast<uint32_t*>(p), n);
  ASYM_HIP(hipGetLastError());
  return ASYM_OK;
}

}  // namespace asym
