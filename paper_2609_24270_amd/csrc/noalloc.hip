// The GEMM entry point that allocates nothing, for callers that cannot call
// the allocator (code under stream capture, tight serving loops, harnesses
// that forbid it).  It runs the same kernels as asym_gemm_bf16; the device
// buffers that call keeps in its per-stream workspace (the tile schedule, the
// claim counters of the aware kernel's claiming form, the fp32 partial tiles
// of a split K) live instead in `scratch`, one fixed array per GPU that the
// library holds until the process ends.
//
// `scratch` is a device symbol: in host code its name is not a device address.
// Its address on each GPU is looked up once, with that GPU current, on the
// first call there (hipGetSymbolAddress), and only that address is handed to
// kernels.  Every call on a GPU shares its array, which keeps what the last
// call left: the schedule it holds is tracked on the host and rewritten when
// a call needs another one, and the counters are cleared before each
// claiming launch.  Calls that overlap in time on one GPU race.
#include <hip/hip_runtime.h>

#include <mutex>

#include "internal.h"

// The per-GPU array (device memory; each GPU holds its own copy).
static __device__ __align__(256) unsigned char scratch[asym::kScratchBytes];

namespace asym {
namespace {

std::mutex g_scratch_mu;
constexpr int kMaxDevices = 64;
unsigned char* g_scratch_ptr[kMaxDevices] = {};

// The current device's copy of `scratch` (looked up once per device).
int scratch_for_current_device(unsigned char** out) {
  int dev = 0;
  ASYM_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(ASYM_EUNSUPPORTED, "gemm (no allocation): device ordinal too large");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    ASYM_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(ASYM_EHIP, "gemm (no allocation): no device address for the scratch array");
    g_scratch_ptr[dev] = static_cast<unsigned char*>(p);
  }
  *out = g_scratch_ptr[dev];
  return ASYM_OK;
}

}  // namespace
}  // namespace asym

extern "C" int asym_gemm_bf16_noalloc(const asym_topology* topo, int M, int N, int K, const void* A, int lda,
                                      const void* B, int ldb, int b_layout, void* C, int ldc, int mapping,
                                      uint32_t xcd_mask, void* stream) {
  using namespace asym;
  int rc = gemm_noalloc_check(topo, M, N, b_layout);  // before any device call
  if (rc != ASYM_OK) return rc;
  unsigned char* base = nullptr;
  rc = scratch_for_current_device(&base);
  if (rc != ASYM_OK) return rc;
  return gemm_bf16_scratch(topo, M, N, K, A, lda, B, ldb, b_layout, C, ldc, mapping, xcd_mask,
                           static_cast<hipStream_t>(stream), base, kScratchBytes);
}

extern "C" int asym_gemm_noalloc_limits(size_t* scratch_bytes, int* max_tiles, size_t* max_partial_bytes) {
  if (scratch_bytes) *scratch_bytes = asym::kScratchBytes;
  if (max_tiles) *max_tiles = asym::kScratchMaxTiles;
  if (max_partial_bytes) *max_partial_bytes = asym::kScratchPartBytes;
  return ASYM_OK;
}
