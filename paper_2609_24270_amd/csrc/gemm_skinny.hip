// Small-M GEMM: C = A . B^T for at most 64 rows per row tile (decode-sized
// products and the expert layer's small groups), bf16 in, fp32 accumulation,
// bf16 out, the same product and rounding as the persistent kernel.
//
// With a few rows the work is bound by streaming B from HBM once (2 N K bytes
// against 2 M N K flops), so the kernel is built for memory-level parallelism
// rather than for operand reuse.  A workgroup owns a 64-column slice of C for
// its row tile; each of its four waves owns 16 of those columns and all of K,
// and streams its 16 B rows straight into MFMA operand registers (a lane's 8
// bf16 of a 16x32 fragment are 16 contiguous bytes of one row), two groups of
// U k-steps in flight.  A, the same for every wave, goes through LDS once per
// stage of U k-steps (double-buffered, one barrier per stage), so the vector
// memory path carries B and little else: with A loaded by every wave, one A
// fragment load per B fragment load, the kernel streamed B at about 4 TB/s;
// shared through LDS, close to the chip's read rate.  Each output element is
// one wave's MFMA chain over k in order, as in the persistent kernel.  Every B
// byte is fetched once and no tile is reused, so there is no placement to
// choose: the grid is a plain launch over the tiles.
//
// A plain problem is cut into row tiles of 16 MB rows (one tile up to 64
// rows); a grouped problem's workgroups each read a descriptor {first row,
// rows, first B row, first column}.  Where a B panel is read by several row
// tiles, the aware order runs them one after another on one XCD, so the panel
// crosses into that XCD's L2 once; the oblivious orders put them on
// neighbouring workgroups (column-major, dealt to different XCDs) or a row of
// tiles apart (row-major).
#include <hip/hip_runtime.h>

#include "internal.h"

namespace asym {
namespace {

constexpr int SK_WAVES = 4;
constexpr int SK_THREADS = 64 * SK_WAVES;
constexpr int SK_COLS = 16 * SK_WAVES;  // 64 columns per tile, 16 per wave
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
  int tiles_n;        // 64-column tiles
  int row_tiles;      // plain GEMM: row tiles of 16 MB rows
  int order;          // plain GEMM: 0 aware, 1 column-major, 2 row-major
  int n_x;            // XCDs (workgroup i runs on XCD i mod n_x)
  const int4* desc;   // grouped: per workgroup {first row, rows, first B row, first column}; rows 0 = none
  int tile_cols;      // columns per column tile (a multiple of 8, at most 64)
  int ksplit;         // plain GEMM, one row tile: K ranges per column tile (1 = none)
  float* part;        // ksplit > 1: fp32 partial tiles [column tile][range][16 MB][64]
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t sk_rsrc(const void* base, uint32_t bytes) {
  const unsigned long long a = (unsigned long long)base;
  const unsigned long long u = ((unsigned long long)__builtin_amdgcn_readfirstlane((uint32_t)(a >> 32)) << 32) |
                               (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)a);
  return __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<void*>(u), (short)0,
                                           (int)__builtin_amdgcn_readfirstlane(bytes), 0x00020000);
}

__device__ __forceinline__ uint32_t sk_pack(float a, float b) {
  bf16x2 v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

// MB: 16-row blocks of the row tile (1, 2 or 4); U: k-steps of 32 per stage.
template <int MB, int U>
__global__ void __launch_bounds__(SK_THREADS) gemm_bf16_small_m(SkinnyParams p) {
  // A stage in LDS, in MFMA operand order: fragment (u, i) is 64 lanes x 16 bytes
  __shared__ bf16x8 sa[2][U * MB * 64];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  int row0, rows, brow0, ncol0, kr = 0, ctile = 0;
  if (p.desc) {
    const int4 d = p.desc[blockIdx.x];
    row0 = __builtin_amdgcn_readfirstlane(d.x);
    rows = __builtin_amdgcn_readfirstlane(d.y);
    brow0 = __builtin_amdgcn_readfirstlane(d.z);
    ncol0 = __builtin_amdgcn_readfirstlane(d.w);
    if (rows <= 0) return;
  } else {
    // plain GEMM: which (row tile r, column tile c) this workgroup computes
    const int i = blockIdx.x;
    int r, c;
    if (p.ksplit > 1) {
      // one row tile; workgroups i = c * ksplit + range
      c = i / p.ksplit;
      kr = i - c * p.ksplit;
      r = 0;
    } else if (p.order == 0) {
      // aware: the row tiles of column tile c run one after another on XCD
      // c mod n_x, so the B panel they all read crosses into that XCD's L2 once
      const int lane_x = i % p.n_x, q = i / p.n_x;
      const int cb = q / p.row_tiles;
      r = q - cb * p.row_tiles;
      c = cb * p.n_x + lane_x;
    } else if (p.order == 1) {
      c = i / p.row_tiles;  // column-major: a column's row tiles on neighbouring workgroups
      r = i - c * p.row_tiles;
    } else {
      r = i / p.tiles_n;    // row-major
      c = i - r * p.tiles_n;
    }
    if (c >= p.tiles_n || r >= p.row_tiles) return;
    row0 = r * 16 * MB;
    rows = min(16 * MB, p.M - row0);
    brow0 = 0;
    ncol0 = c * p.tile_cols;
    ctile = c;
  }
  // this wave's 16 columns (fewer at the tile's or the product's edge); a wave
  // past either has an empty B range and stores nothing
  const int n0 = ncol0 + wave * 16;
  const int cols = max(0, min(16, min(p.N, ncol0 + p.tile_cols) - n0));

  // rows past the tile read as zero (outside the resource); a 16-byte chunk at
  // k >= K is sent out of range (K is a multiple of 8: a chunk is all inside
  // or all outside)
  const __amdgpu_buffer_rsrc_t ra = sk_rsrc(p.A + (size_t)row0 * p.lda, (uint32_t)rows * p.lda * 2u);
  const __amdgpu_buffer_rsrc_t rb =
      sk_rsrc(p.B + (size_t)(brow0 + min(n0, p.N)) * p.ldb, (uint32_t)cols * p.ldb * 2u);
  const int lr = lane & 15, lk = (lane >> 4) * 8;
  const uint32_t vob = (uint32_t)(lr * p.ldb + lk) * 2u;
  // this workgroup's k-steps of 32: all of K, or its range of a split K
  const int steps = (p.K + 31) >> 5;
  const int per = (steps + p.ksplit - 1) / p.ksplit;
  const int ks0 = min(steps, kr * per), ks1 = min(steps, ks0 + per);
  const int stages = (ks1 - ks0 + U - 1) / U;

  // A staging: chunk c of a stage is (row, k-step u, quarter kq) in row-major
  // order; thread t carries chunks t, t + 256, ...
  constexpr int CHUNKS = MB * 16 * U * 4;
  constexpr int A_PER = (CHUNKS + SK_THREADS - 1) / SK_THREADS;
  auto a_load = [&](int st, v4u (&r)[A_PER]) {
#pragma unroll
    for (int e = 0; e < A_PER; ++e) {
      const int c = threadIdx.x + e * SK_THREADS;
      const int row = c / (U * 4), cc = c % (U * 4);
      const int ks = ks0 + st * U + (cc >> 2);
      const int k = ks * 32 + (cc & 3) * 8;
      const bool in = c < CHUNKS && ks < ks1 && k < p.K;
      r[e] = __builtin_amdgcn_raw_buffer_load_b128(ra, in ? (uint32_t)(row * p.lda + k) * 2u : kSkOOB, 0, 0);
    }
  };
  auto a_store = [&](int buf, const v4u (&r)[A_PER]) {
#pragma unroll
    for (int e = 0; e < A_PER; ++e) {
      const int c = threadIdx.x + e * SK_THREADS;
      if (c >= CHUNKS) continue;
      const int row = c / (U * 4), cc = c % (U * 4);
      const int u = cc >> 2, kq = cc & 3;
      sa[buf][(u * MB + (row >> 4)) * 64 + (row & 15) + 16 * kq] = __builtin_bit_cast(bf16x8, r[e]);
    }
  };
  auto b_load = [&](int st, bf16x8 (&b)[U]) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int ks = ks0 + st * U + u;
      const int k = ks * 32;
      const v4u x = __builtin_amdgcn_raw_buffer_load_b128(rb, ks < ks1 && k + lk < p.K ? vob : kSkOOB, k * 2, 0);
      b[u] = __builtin_bit_cast(bf16x8, x);
    }
  };
  f32x4 acc[MB];
#pragma unroll
  for (int i = 0; i < MB; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto compute = [&](int buf, const bf16x8 (&b)[U]) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      bf16x8 a[MB];
#pragma unroll
      for (int i = 0; i < MB; ++i) a[i] = sa[buf][(u * MB + i) * 64 + lane];
#pragma unroll
      for (int i = 0; i < MB; ++i) acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(b[u], a[i], acc[i], 0, 0, 0);
    }
  };

  // stage s uses LDS buffer s % 2 and B registers b0 (even) / b1 (odd); the
  // loads of stage s + 1 are in flight while stage s is computed
  // a wave with no columns (past the tile's or the product's edge) stages A
  // and meets the barriers but loads no B and computes nothing
  const bool busy = cols > 0;
  bf16x8 b0[U], b1[U];
  v4u ar[A_PER];
  a_load(0, ar);
  a_store(0, ar);
  if (stages > 1) a_load(1, ar);
  if (busy) b_load(0, b0);
  __syncthreads();
  for (int st = 0; st < stages; st += 2) {
    if (busy && st + 1 < stages) b_load(st + 1, b1);
    if (busy) compute(0, b0);
    if (st + 1 < stages) {
      a_store(1, ar);
      if (st + 2 < stages) a_load(st + 2, ar);
    }
    __syncthreads();
    if (st + 1 >= stages) break;
    if (busy && st + 2 < stages) b_load(st + 2, b0);
    if (busy) compute(1, b1);
    if (st + 2 < stages) {
      a_store(0, ar);
      if (st + 3 < stages) a_load(st + 3, ar);
    }
    __syncthreads();
  }

  // in a 16x16 block the lane with row r = lane % 16 holds columns 4c..4c+3,
  // c = lane / 16; rows past the tile fall outside the resource
  const int nl = (lane >> 4) * 4;  // column inside the wave's 16
  if (p.ksplit > 1) {
    // split K: every range writes its fp32 tile; a second launch adds them
    float* mine = p.part + ((size_t)ctile * p.ksplit + kr) * (16 * MB * 64);
#pragma unroll
    for (int i = 0; i < MB; ++i)
      *reinterpret_cast<f32x4*>(mine + (i * 16 + lr) * 64 + wave * 16 + nl) = acc[i];
    return;
  }
  const __amdgpu_buffer_rsrc_t rc = sk_rsrc(p.C + (size_t)row0 * p.ldc, (uint32_t)rows * p.ldc * 2u);
  const bool vec_c = ((p.ldc & 3) == 0) && ((reinterpret_cast<uintptr_t>(p.C) & 7) == 0);
#pragma unroll
  for (int i = 0; i < MB; ++i) {
    const f32x4 v = acc[i];
    const int m = i * 16 + lr;
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

// The sum of a split K: for each (column tile, row, 4 columns), the ranges'
// partial tiles added in range order, rounded to bf16 and stored.  One thread
// per 4 outputs.
__global__ void __launch_bounds__(256) small_m_reduce(const float* __restrict__ part, int tiles_n, int ksplit,
                                                      int tile_rows, int M, int N, uint16_t* __restrict__ C,
                                                      int ldc) {
  const long long id = (long long)blockIdx.x * 256 + threadIdx.x;
  const long long per_tile = (long long)tile_rows * 16;   // 16 groups of 4 columns per row
  if (id >= per_tile * tiles_n) return;
  const int c = (int)(id / per_tile);
  const int rem = (int)(id - (long long)c * per_tile);
  const int m = rem / 16, q = rem % 16;
  if (m >= M) return;
  const float* src = part + (size_t)c * ksplit * tile_rows * 64 + m * 64 + 4 * q;
  f32x4 v = {0.f, 0.f, 0.f, 0.f};
  for (int s = 0; s < ksplit; ++s) v += *reinterpret_cast<const f32x4*>(src + (size_t)s * tile_rows * 64);
  const int n = c * SK_COLS + 4 * q;
  uint16_t* dst = C + (size_t)m * ldc + n;
#pragma unroll
  for (int r = 0; r < 4; ++r)
    if (n + r < N) dst[r] = __builtin_bit_cast(unsigned short, (__bf16)v[r]);
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
  if (g.tile_cols < 8 || g.tile_cols > SK_COLS || g.tile_cols % 8 || (g.ksplit > 1 && g.tile_cols != SK_COLS))
    return fail(ASYM_EINVAL, "small-M GEMM: column tiles of 8 to 64 columns (64 when split)");
  p.tile_cols = g.tile_cols;
  p.tiles_n = (g.N + g.tile_cols - 1) / g.tile_cols;
  p.row_tiles = g.row_tiles;
  p.order = g.order;
  p.n_x = g.n_x;
  p.desc = static_cast<const int4*>(g.d_desc);
  p.ksplit = g.ksplit;
  p.part = g.part;
  if (p.ksplit > 1 && (p.desc || p.row_tiles != 1 || !p.part))
    return fail(ASYM_EINVAL, "small-M GEMM: a split K needs one row tile and a workspace");
  const long long grid = g.grid;
  if (grid < 1 || grid > (1ll << 31) - 1) return fail(ASYM_EINVAL, "small-M GEMM: grid out of range");
  switch (g.mb) {
    // stages of 8 k-steps (A stage 16 / 32 KiB of LDS); 4 with 64 rows (32 KiB)
    case 1:
      hipLaunchKernelGGL((gemm_bf16_small_m<1, 8>), dim3((unsigned)grid), dim3(SK_THREADS), 0, s, p);
      break;
    case 2:
      hipLaunchKernelGGL((gemm_bf16_small_m<2, 8>), dim3((unsigned)grid), dim3(SK_THREADS), 0, s, p);
      break;
    case 4:
      hipLaunchKernelGGL((gemm_bf16_small_m<4, 4>), dim3((unsigned)grid), dim3(SK_THREADS), 0, s, p);
      break;
    default:
      return fail(ASYM_EINVAL, "small-M GEMM: row blocks must be 1, 2 or 4");
  }
  ASYM_HIP(hipGetLastError());
  if (p.ksplit > 1) {
    const long long threads = (long long)p.tiles_n * 16 * g.mb * 16;
    hipLaunchKernelGGL(small_m_reduce, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s, g.part, p.tiles_n,
                       p.ksplit, 16 * g.mb, g.M, g.N, static_cast<uint16_t*>(g.C), g.ldc);
    ASYM_HIP(hipGetLastError());
  }
  return ASYM_OK;
}

int small_m_tile_cols() { return SK_COLS; }

}  // namespace asym
