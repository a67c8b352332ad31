// Streaming copy, the bandwidth-bound co-runner of the co-location study
// (Section 7.3 places a second tenant on the complementary units; here that
// tenant is an HBM-bound copy so the GEMM's CU set competes for memory
// bandwidth and clocks as real co-located work does).
//
// dst[i] = src[i] with 16-byte accesses from every lane.  Work is cut into
// 64 KiB chunks; workgroups claim chunks from a counter (pass p, chunk c is
// claim p * chunks + c), so any subset of workgroups covers the whole buffer.
// The kernel ends after `passes` passes, or at the next claim once *stop_flag
// is nonzero; every wave reaches one of the two, so the grid always drains.
// Workgroups on XCDs outside xcd_mask exit at once, which confines the copy to
// whole XCDs without a hardware CU mask.  The last workgroup to leave resets
// the counters, so back-to-back launches on one stream need no memset.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "internal.h"

namespace asym {
namespace {

constexpr int kCopyThreads = 256;
typedef unsigned v4u __attribute__((ext_vector_type(4)));

constexpr size_t kChunk16 = 4096;  // 16-byte units per chunk (64 KiB)
constexpr int kPerThread = (int)(kChunk16 / kCopyThreads);  // 16

// The claim loop keeps all lane-divergent work at the top of its body (thread
// 0's claim, before the first barrier); everything after the barriers has the
// same trip count in every lane.  Divergent code at the end of a loop body that
// also holds barriers can be restructured by the compiler into an inner loop
// around the barriers that the claiming lane never re-enters, so the byte count
// is kept in a register and added once on exit.
__global__ void __launch_bounds__(kCopyThreads)
copy_kernel(v4u* __restrict__ dst, const v4u* __restrict__ src, size_t n16, int passes,
            const int* stop_flag, uint32_t xcd_mask, unsigned long long* ctr) {
  uint32_t x;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(x));
  x &= 0xFu;
  __shared__ unsigned long long s_claim;
  const unsigned long long chunks = (n16 + kChunk16 - 1) / kChunk16;
  const unsigned long long total = chunks * (unsigned long long)passes;
  unsigned long long moved = 0;
  if (xcd_mask == 0u || ((xcd_mask >> x) & 1u)) {
    for (;;) {
      if (threadIdx.x == 0) {
        unsigned long long c = total;
        if (!(stop_flag && __hip_atomic_load(stop_flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM)))
          c = atomicAdd(&ctr[0], 1ull);
        s_claim = c;
      }
      __syncthreads();
      const unsigned long long c = s_claim;
      __syncthreads();
      if (c >= total) break;
      const size_t b0 = (size_t)(c % chunks) * kChunk16;
      const size_t b1 = b0 + kChunk16 < n16 ? b0 + kChunk16 : n16;
#pragma unroll
      for (int k = 0; k < kPerThread; k += 4) {
        v4u v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const size_t i = b0 + (size_t)(k + u) * kCopyThreads + threadIdx.x;
          v[u] = i < b1 ? __builtin_nontemporal_load(src + i) : v4u{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const size_t i = b0 + (size_t)(k + u) * kCopyThreads + threadIdx.x;
          if (i < b1) __builtin_nontemporal_store(v[u], dst + i);
        }
      }
      moved += (unsigned long long)(b1 - b0) * 16ull;
    }
  }
  if (threadIdx.x == 0) {
    if (moved) atomicAdd(&ctr[2], moved);
    __threadfence();
    const unsigned long long done = atomicAdd(&ctr[1], 1ull);
    if (done == gridDim.x - 1ull) {
      atomicExch(&ctr[0], 0ull);
      atomicExch(&ctr[1], 0ull);
      __threadfence();
    }
  }
}

__global__ void zero_words_kernel(uint32_t* p, size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

__global__ void set_flag_kernel(int* flag, int v) {
  if (threadIdx.x == 0) __hip_atomic_store(flag, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

}  // namespace

// ctr: 3 device words {next claim, exits, bytes moved}; the first two must be
// zero before the first launch and are zero again after every launch; the
// third accumulates until the caller clears it.
int launch_copy(void* dst, const void* src, size_t n_bytes, int passes, const int* stop_flag,
                uint32_t xcd_mask, int grid, unsigned long long* ctr, hipStream_t s) {
  hipLaunchKernelGGL(copy_kernel, dim3(grid), dim3(kCopyThreads), 0, s, static_cast<v4u*>(dst),
                     static_cast<const v4u*>(src), n_bytes / 16, passes, stop_flag, xcd_mask, ctr);
  ASYM_HIP(hipGetLastError());
  return ASYM_OK;
}

// The claim-loop copy kernel did not finish in two device runs whose cause is
// not understood; it stays unreachable until the cause is shown.
bool copy_kernel_enabled() { return false; }

// Stream-ordered zero fill of n 4-byte words (a kernel, not a memset node, so
// that it also behaves under graph capture).
int launch_zero_words(void* p, size_t n, hipStream_t s) {
  if (!p || !n) return ASYM_OK;
  const int grid = (int)std::min<size_t>((n + 255) / 256, 1024);
  hipLaunchKernelGGL(zero_words_kernel, dim3(grid), dim3(256), 0, s, static_cast<uint32_t*>(p), n);
  ASYM_HIP(hipGetLastError());
  return ASYM_OK;
}

int launch_set_flag(int* flag, int v, hipStream_t s) {
  hipLaunchKernelGGL(set_flag_kernel, dim3(1), dim3(64), 0, s, flag, v);
  ASYM_HIP(hipGetLastError());
  return ASYM_OK;
}

}  // namespace asym
