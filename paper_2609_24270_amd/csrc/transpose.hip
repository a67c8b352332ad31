// Transpose of a bf16 matrix, for the B operand stored [K][N] (N contiguous):
// the GEMM kernels read B as [N][K] (K contiguous, a linear layer's weight
// layout), so a [K][N] operand is first rewritten as its transpose.  The copy
// is exact (it moves 16-bit words), so the product is bitwise the one of the
// same logical B stored [N][K].
//
// 64 x 64 tiles through LDS: a workgroup of 256 threads reads a tile with
// 16-byte loads along N (rows of the source), and writes it with 16-byte
// stores along K (rows of the destination).  The LDS tile is padded by one
// 16-bit word per row so that the column reads of the write phase fall in
// different banks.  Ragged edges are bounds-checked per element.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace asym {
namespace {

constexpr int kT = 64;        // tile edge
constexpr int kThreads = 256;

__global__ void __launch_bounds__(kThreads)
transpose_bf16_kernel(const uint16_t* __restrict__ src, int rows, int cols, int lds,
                      uint16_t* __restrict__ dst, int ldd) {
  __shared__ uint16_t tile[kT][kT + 1];
  const int r0 = blockIdx.y * kT, c0 = blockIdx.x * kT;
  const int t = threadIdx.x;
  // read: 64 rows x 8 chunks of 8 words; thread t takes chunk t % 8 of rows t / 8 + 32 i
  const int ch = t & 7;
  for (int i = 0; i < 2; ++i) {
    const int r = (t >> 3) + 32 * i;
    const int gr = r0 + r, gc = c0 + ch * 8;
    uint16_t w[8];
    if (gr < rows && gc + 7 < cols && ((((uintptr_t)(src + (size_t)gr * lds + gc)) & 15u) == 0)) {
      const uint4 v = *reinterpret_cast<const uint4*>(src + (size_t)gr * lds + gc);
      const uint32_t u[4] = {v.x, v.y, v.z, v.w};
      for (int e = 0; e < 4; ++e) {
        w[2 * e] = (uint16_t)(u[e] & 0xFFFFu);
        w[2 * e + 1] = (uint16_t)(u[e] >> 16);
      }
    } else {
      for (int e = 0; e < 8; ++e) w[e] = (gr < rows && gc + e < cols) ? src[(size_t)gr * lds + gc + e] : 0;
    }
    for (int e = 0; e < 8; ++e) tile[r][ch * 8 + e] = w[e];
  }
  __syncthreads();
  // write: destination row c (source column), 8 words of source rows ch*8 ..
  for (int i = 0; i < 2; ++i) {
    const int c = (t >> 3) + 32 * i;
    const int gd = c0 + c, gk = r0 + ch * 8;
    if (gd >= cols) continue;
    uint16_t w[8];
    for (int e = 0; e < 8; ++e) w[e] = tile[ch * 8 + e][c];
    uint16_t* out = dst + (size_t)gd * ldd + gk;
    if (gk + 7 < rows && ((((uintptr_t)out) & 15u) == 0)) {
      uint4 v;
      v.x = (uint32_t)w[0] | ((uint32_t)w[1] << 16);
      v.y = (uint32_t)w[2] | ((uint32_t)w[3] << 16);
      v.z = (uint32_t)w[4] | ((uint32_t)w[5] << 16);
      v.w = (uint32_t)w[6] | ((uint32_t)w[7] << 16);
      *reinterpret_cast<uint4*>(out) = v;
    } else {
      for (int e = 0; e < 8; ++e)
        if (gk + e < rows) out[e] = w[e];
    }
  }
}

}  // namespace

// dst[c][r] = src[r][c] for r < rows, c < cols; src has row pitch lds >= cols,
// dst row pitch ldd >= rows (elements); columns rows .. ldd-1 of dst untouched.
int launch_transpose_bf16(const void* src, int rows, int cols, int lds, void* dst, int ldd, hipStream_t s) {
  if (!src || !dst || rows < 1 || cols < 1 || lds < cols || ldd < rows)
    return fail(ASYM_EINVAL, "transpose: bad arguments");
  const dim3 grid((unsigned)((cols + kT - 1) / kT), (unsigned)((rows + kT - 1) / kT));
  if (grid.y > 65535u) return fail(ASYM_EUNSUPPORTED, "transpose: too many rows");
  hipLaunchKernelGGL(transpose_bf16_kernel, grid, dim3(kThreads), 0, s, static_cast<const uint16_t*>(src), rows,
                     cols, lds, static_cast<uint16_t*>(dst), ldd);
  ASYM_HIP(hipGetLastError());
  return ASYM_OK;
}

}  // namespace asym
