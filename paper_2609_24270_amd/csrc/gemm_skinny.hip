// Small-M GEMM: C = A . B^T for at most 64 rows per row tile (decode-sized
// products and the expert layer's small groups), bf16 in, fp32 accumulation,
// bf16 out, the same product and rounding as the persistent kernel.
//
// With a few rows the work is bound by streaming B from HBM once (2 N K bytes
// against 2 M N K flops), so the kernel is built for memory-level parallelism
// rather than for operand reuse: a workgroup owns a 32-column slice of C for
// its row tile and all of K; its four waves split K into four ranges and
// each wave streams its range of the 32 B rows straight into MFMA operand
// registers (no LDS staging: a lane's 8 bf16 of a 16x32 fragment are 16
// contiguous bytes of one row), U k-steps of 32 ahead of the MFMAs.  The four
// partial tiles meet in LDS at the end and are summed in wave order, so the
// result does not depend on timing.  Every B byte is fetched once; there is no
// tile reuse for a placement to exploit, so the grid is a plain launch over
// the tiles and the hardware spreads it.
//
// A row tile is one plain problem (rows 0..M-1) or one group of a grouped
// problem, given by a descriptor {first row, rows, first B row, unused}.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace asym {
namespace {

constexpr int SK_THREADS = 256;
constexpr int SK_WAVES = 4;
constexpr int SK_NBW = 2;            // 16-column blocks per tile: 32 columns
constexpr int SK_COLS = 16 * SK_NBW;
constexpr int SK_U = 4;              // k-steps of 32 loaded ahead
constexpr uint32_t kSkOOB = 0x80000000u;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef unsigned v4u __attribute__((ext_vector_type(4)));
typedef unsigned v2u __attribute__((ext_vector_type(2)));

struct SkinnyParams {
  const uint16_t* A;
  const uint16_t* B;
  uint16_t* C;
  int M, N, K, lda, ldb, ldc;
  int tiles_n;        // 32-column tiles per row tile
  const int4* desc;   // per row tile {first row, rows, first B row, 0}; null = one tile of M rows
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t sk_rsrc(const void* base, uint32_t bytes) {
  const unsigned long long a = (unsigned long long)base;
  const unsigned long long u = ((unsigned long long)__builtin_amdgcn_readfirstlane((uint32_t)(a >> 32)) << 32) |
                               (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)a);
  return __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<void*>(u), (short)0,
                                           (int)__builtin_amdgcn_readfirstlane(bytes), 0x00020000);
}

__device__ __forceinline__ bf16x8 sk_load(__amdgpu_buffer_rsrc_t rs, uint32_t vo, int so) {
  const v4u x = __builtin_amdgcn_raw_buffer_load_b128(rs, vo, so, 0);
  return __builtin_bit_cast(bf16x8, x);
}

__device__ __forceinline__ uint32_t sk_pack(float a, float b) {
  bf16x2 v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

// MB: 16-row blocks of the row tile (1, 2 or 4).
template <int MB>
__global__ void __launch_bounds__(SK_THREADS) gemm_bf16_small_m(SkinnyParams p) {
  __shared__ f32x4 red[SK_WAVES][SK_NBW * MB][64];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int tile = blockIdx.x;
  const int rt = tile / p.tiles_n, ct = tile - rt * p.tiles_n;
  int row0 = 0, rows = p.M, brow0 = 0;
  if (p.desc) {
    const int4 d = p.desc[rt];
    row0 = __builtin_amdgcn_readfirstlane(d.x);
    rows = __builtin_amdgcn_readfirstlane(d.y);
    brow0 = __builtin_amdgcn_readfirstlane(d.z);
  }
  const int n0 = ct * SK_COLS;
  const int cols = min(SK_COLS, p.N - n0);

  // operands: rows past the tile read as zero (outside the resource); k-steps
  // at or past K are sent out of range per lane (K is a multiple of 8, so a
  // lane's 8 elements are all inside or all outside)
  const __amdgpu_buffer_rsrc_t ra = sk_rsrc(p.A + (size_t)row0 * p.lda, (uint32_t)rows * p.lda * 2u);
  const __amdgpu_buffer_rsrc_t rb = sk_rsrc(p.B + (size_t)(brow0 + n0) * p.ldb, (uint32_t)cols * p.ldb * 2u);
  const int lr = lane & 15, lk = (lane >> 4) * 8;
  const uint32_t voa = (uint32_t)(lr * p.lda + lk) * 2u;
  const uint32_t vob = (uint32_t)(lr * p.ldb + lk) * 2u;

  const int steps = (p.K + 31) >> 5;
  const int per = (steps + SK_WAVES - 1) / SK_WAVES;
  const int s0 = min(steps, wave * per), s1 = min(steps, s0 + per);

  f32x4 acc[SK_NBW][MB];
#pragma unroll
  for (int j = 0; j < SK_NBW; ++j)
#pragma unroll
    for (int i = 0; i < MB; ++i) acc[j][i] = f32x4{0.f, 0.f, 0.f, 0.f};

  // two register sets in turn: the loads of one group of U k-steps are in
  // flight while the MFMAs consume the other
  bf16x8 b0[SK_U][SK_NBW], a0[SK_U][MB], b1[SK_U][SK_NBW], a1[SK_U][MB];
  auto load_group = [&](int s, bf16x8 (&b)[SK_U][SK_NBW], bf16x8 (&a)[SK_U][MB]) {
#pragma unroll
    for (int u = 0; u < SK_U; ++u) {
      const int k = (s + u) * 32;
      const bool in = s + u < s1 && k + lk < p.K;
      const uint32_t vb = in ? vob : kSkOOB, va = in ? voa : kSkOOB;
#pragma unroll
      for (int j = 0; j < SK_NBW; ++j) b[u][j] = sk_load(rb, vb, (16 * j * p.ldb + k) * 2);
#pragma unroll
      for (int i = 0; i < MB; ++i) a[u][i] = sk_load(ra, va, (16 * i * p.lda + k) * 2);
    }
  };
  auto compute = [&](int s, const bf16x8 (&b)[SK_U][SK_NBW], const bf16x8 (&a)[SK_U][MB]) {
#pragma unroll
    for (int u = 0; u < SK_U; ++u) {
      if (s + u >= s1) break;
#pragma unroll
      for (int j = 0; j < SK_NBW; ++j)
#pragma unroll
        for (int i = 0; i < MB; ++i)
          acc[j][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(b[u][j], a[u][i], acc[j][i], 0, 0, 0);
    }
  };
  if (s0 < s1) load_group(s0, b0, a0);
  for (int s = s0; s < s1; s += 2 * SK_U) {
    if (s + SK_U < s1) load_group(s + SK_U, b1, a1);
    compute(s, b0, a0);
    if (s + 2 * SK_U < s1) load_group(s + 2 * SK_U, b0, a0);
    if (s + SK_U < s1) compute(s + SK_U, b1, a1);
  }

  // the four K ranges meet in LDS; block q = j * MB + i is summed by wave
  // q % 4 in wave order 0, 1, 2, 3
#pragma unroll
  for (int j = 0; j < SK_NBW; ++j)
#pragma unroll
    for (int i = 0; i < MB; ++i) red[wave][j * MB + i][lane] = acc[j][i];
  __syncthreads();

  // in a 16x16 block the lane with row r = lane % 16 holds columns 4c..4c+3,
  // c = lane / 16; rows past the tile fall outside the resource
  const __amdgpu_buffer_rsrc_t rc = sk_rsrc(p.C + (size_t)row0 * p.ldc, (uint32_t)rows * p.ldc * 2u);
  const bool vec_c = ((p.ldc & 3) == 0) && ((reinterpret_cast<uintptr_t>(p.C) & 7) == 0);
#pragma unroll
  for (int q = 0; q < SK_NBW * MB; ++q) {
    if (q % SK_WAVES != wave) continue;
    const int j = q / MB, i = q - (q / MB) * MB;
    f32x4 v = red[0][q][lane];
#pragma unroll
    for (int w = 1; w < SK_WAVES; ++w) v += red[w][q][lane];
    const int m = i * 16 + lr;
    const int nl = j * 16 + (lane >> 4) * 4;  // column inside the tile
    const uint32_t base = (uint32_t)(m * p.ldc + n0 + nl) * 2u;
    if (vec_c && nl + 3 < cols) {
      v2u w2;
      w2.x = sk_pack(v[0], v[1]);
      w2.y = sk_pack(v[2], v[3]);
      __builtin_amdgcn_raw_buffer_store_b64(w2, rc, base, 0, 0);
    } else {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const __bf16 h = (__bf16)v[r];
        __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(unsigned short, h), rc,
                                              nl + r < cols ? base + 2u * r : kSkOOB, 0, 0);
      }
    }
  }
}

}  // namespace

int small_m_blocks(int max_rows) {
  if (max_rows <= 16) return 1;
  if (max_rows <= 32) return 2;
  if (max_rows <= 64) return 4;
  return 0;
}

int launch_gemm_small_m(const SmallMLaunch& g, hipStream_t s) {
  SkinnyParams p;
  p.A = static_cast<const uint16_t*>(g.A);
  p.B = static_cast<const uint16_t*>(g.B);
  p.C = static_cast<uint16_t*>(g.C);
  p.M = g.M;
  p.N = g.N;
  p.K = g.K;
  p.lda = g.lda;
  p.ldb = g.ldb;
  p.ldc = g.ldc;
  p.tiles_n = (g.N + SK_COLS - 1) / SK_COLS;
  p.desc = static_cast<const int4*>(g.d_desc);
  const long long grid = (long long)g.row_tiles * p.tiles_n;
  if (grid < 1 || grid > (1ll << 31) - 1) return fail(ASYM_EINVAL, "small-M GEMM: grid out of range");
  switch (g.mb) {
    case 1:
      hipLaunchKernelGGL(gemm_bf16_small_m<1>, dim3((unsigned)grid), dim3(SK_THREADS), 0, s, p);
      break;
    case 2:
      hipLaunchKernelGGL(gemm_bf16_small_m<2>, dim3((unsigned)grid), dim3(SK_THREADS), 0, s, p);
      break;
    case 4:
      hipLaunchKernelGGL(gemm_bf16_small_m<4>, dim3((unsigned)grid), dim3(SK_THREADS), 0, s, p);
      break;
    default:
      return fail(ASYM_EINVAL, "small-M GEMM: row blocks must be 1, 2 or 4");
  }
  ASYM_HIP(hipGetLastError());
  return ASYM_OK;
}

int small_m_tile_cols() { return SK_COLS; }

}  // namespace asym
