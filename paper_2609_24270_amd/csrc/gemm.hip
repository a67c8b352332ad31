// Persistent bf16 GEMM for gfx950 with XCD-aware tile placement.
//
// Section 7.1 ("Integration with popular kernels") makes a kernel
// asymmetry-aware by running one persistent block per compute unit, letting
// each block look up the unit it landed on, and giving it the tasks whose data
// is local to that unit's partition, with work in proportion to each
// partition's units.  Here a task is a 256x256 output tile, the partition is
// the XCD (private 4 MB L2), and the lookup is one read of the XCC_ID hardware
// register.  In AWARE mode a workgroup takes a rank ticket on its XCD, exits if
// the XCD already has as many persistent workgroups as it has scheduled CUs,
// and then claims tiles from its XCD's region of the schedule with a per-XCD
// atomic counter (then from other XCDs' regions once its own is empty, so the
// result never depends on where the hardware placed workgroups).  The
// OBLIVIOUS modes walk one shared order statically (tile i on workgroup i mod
// P), which is how a persistent GEMM without topology knowledge runs.
//
// C = A . B with A [M][lda], B stored [N][ldb] (K contiguous), C [M][ldc], all
// bf16; fp32 accumulation in the matrix cores (v_mfma_f32_16x16x32_bf16);
// bf16 round-to-nearest-even output (v_cvt_pk_bf16_f32).
//
// Tile 256x256x64, 256 threads = 4 waves in a 2x2 grid, 128x128 per wave
// (8x8 MFMA blocks, 256 fp32 accumulators per lane).  LDS: two stages of A and
// B, rows padded to 72 bf16 (144 B) so that the 16-byte reads of 16 different
// rows fall in distinct banks; 144 KiB in all, one workgroup per CU.
// Global->LDS staging goes through registers with 16-byte loads: the next
// k-step's loads are issued before the current step's MFMAs and written to the
// other LDS stage after them, with one barrier per k-step.
//
// The MFMA's first operand is taken from B and its second from A, so each
// lane's four accumulators are four consecutive columns of one C row: the
// epilogue stores 8 contiguous bytes per lane.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace asym {
namespace {

constexpr int BM = 256, BN = 256, BK = 64, NT = 256;
constexpr int LDP = BK + 8;  // padded LDS row pitch, in bf16 elements
constexpr int WM = 128, WN = 128;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

struct Params {
  const uint16_t* A;
  const uint16_t* B;
  uint16_t* C;
  int M, N, K, lda, ldb, ldc;
  int tiles_m, tiles_n, n_tiles;
  int mapping;
  int n_xccs;
  const int* order;
  const int* off;    // [ASYM_MAX_XCDS + 1]
  const int* slots;  // [ASYM_MAX_XCDS]
  int* ctr;          // [0,16) rank tickets, [16,32) tile counters, [32] exits
};

__device__ __forceinline__ uint32_t read_xcc_id() {
  uint32_t v;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(v));
  return v & 0xFu;
}

// Buffer resource over `bytes` bytes at `base`: loads beyond the range return
// zero and stores beyond it are dropped, so tile edges need no branches.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}
constexpr uint32_t kOOB = 0x80000000u;  // an offset past any range used here

typedef unsigned v4u __attribute__((ext_vector_type(4)));
typedef unsigned v2u __attribute__((ext_vector_type(2)));

// Load one 256x64 k-slice of a K-contiguous operand into registers: thread t
// covers rows t/8 + 32*i, 16-byte chunk t%8.  `rs` spans the tile's rows
// (rows past the matrix edge are outside it and read as zero); chunks at
// k >= K are sent out of range as well.  The per-thread part of the offset is
// one VGPR (`vo`, row t/8 and chunk t%8 at k = 0); the row-block and k parts
// are uniform and go in the scalar offset.
template <bool VEC>
__device__ __forceinline__ void load_tile(uint4 (&r)[8], __amdgpu_buffer_rsrc_t rs, int ld,
                                          uint32_t vo, int K, int k0) {
  const int kc = (threadIdx.x & 7) * 8;
  if constexpr (VEC) {
    const uint32_t v = k0 + kc < K ? vo : kOOB;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int so = (32 * i * ld + k0) * 2;
      const v4u x = __builtin_amdgcn_raw_buffer_load_b128(rs, v, so, 0);
      r[i] = make_uint4(x.x, x.y, x.z, x.w);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int so = (32 * i * ld + k0) * 2;
      uint32_t w[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int k = k0 + kc + 2 * e;
        const uint32_t lo = __builtin_amdgcn_raw_buffer_load_b16(rs, k < K ? vo + 4u * e : kOOB, so, 0);
        const uint32_t hi = __builtin_amdgcn_raw_buffer_load_b16(rs, k + 1 < K ? vo + 4u * e + 2u : kOOB, so, 0);
        w[e] = lo | (hi << 16);
      }
      r[i] = make_uint4(w[0], w[1], w[2], w[3]);
    }
  }
}

__device__ __forceinline__ void store_tile(uint16_t* __restrict__ s, const uint4 (&r)[8]) {
  const int t = threadIdx.x;
  const int kc = (t & 7) * 8;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int row = (t >> 3) + 32 * i;
    *reinterpret_cast<uint4*>(s + row * LDP + kc) = r[i];
  }
}

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  bf16x2 v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

template <bool VEC>
__device__ __forceinline__ void compute_tile(const Params& p, int tile, uint16_t* sA, uint16_t* sB) {
  const int tm = tile / p.tiles_n, tn = tile - tm * p.tiles_n;
  const int m0 = tm * BM, n0 = tn * BN;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int KT = (p.K + BK - 1) / BK;

  f32x4 acc[8][8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int rows_a = min(BM, p.M - m0), rows_b = min(BN, p.N - n0);
  const __amdgpu_buffer_rsrc_t rsa = make_rsrc(p.A + (size_t)m0 * p.lda, (uint32_t)rows_a * p.lda * 2u);
  const __amdgpu_buffer_rsrc_t rsb = make_rsrc(p.B + (size_t)n0 * p.ldb, (uint32_t)rows_b * p.ldb * 2u);
  const uint32_t voa = (uint32_t)((threadIdx.x >> 3) * p.lda + (threadIdx.x & 7) * 8) * 2u;
  const uint32_t vob = (uint32_t)((threadIdx.x >> 3) * p.ldb + (threadIdx.x & 7) * 8) * 2u;
  uint4 ra[8], rb[8];
  load_tile<VEC>(ra, rsa, p.lda, voa, p.K, 0);
  load_tile<VEC>(rb, rsb, p.ldb, vob, p.K, 0);
  store_tile(sA, ra);
  store_tile(sB, rb);
  __syncthreads();

  const int lrow = lane & 15, lk = (lane >> 4) * 8;
  for (int kt = 0; kt < KT; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < KT;
    if (more) {
      load_tile<VEC>(ra, rsa, p.lda, voa, p.K, (kt + 1) * BK);
      load_tile<VEC>(rb, rsb, p.ldb, vob, p.K, (kt + 1) * BK);
    }
    const uint16_t* a_s = sA + cur * (BM * LDP) + (wm * WM + lrow) * LDP + lk;
    const uint16_t* b_s = sB + cur * (BN * LDP) + (wn * WN + lrow) * LDP + lk;
#pragma unroll
    for (int ks = 0; ks < BK / 32; ++ks) {
      bf16x8 xa[8], xb[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        xa[i] = *reinterpret_cast<const bf16x8*>(a_s + i * 16 * LDP + ks * 32);
        xb[i] = *reinterpret_cast<const bf16x8*>(b_s + i * 16 * LDP + ks * 32);
      }
#pragma unroll
      for (int nb = 0; nb < 8; ++nb)
#pragma unroll
        for (int mb = 0; mb < 8; ++mb)
          acc[nb][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xb[nb], xa[mb], acc[nb][mb], 0, 0, 0);
    }
    if (more) {
      store_tile(sA + (cur ^ 1) * (BM * LDP), ra);
      store_tile(sB + (cur ^ 1) * (BN * LDP), rb);
    }
    __syncthreads();
  }

  // epilogue: lane holds C[m][n..n+3] for each (nb, mb) block; rows past M
  // fall outside the resource and their stores are dropped
  const int rows_c = min(BM, p.M - m0);
  const __amdgpu_buffer_rsrc_t rsc = make_rsrc(p.C + (size_t)m0 * p.ldc, (uint32_t)rows_c * p.ldc * 2u);
#pragma unroll
  for (int nb = 0; nb < 8; ++nb) {
    const int n = n0 + wn * WN + nb * 16 + (lane >> 4) * 4;
#pragma unroll
    for (int mb = 0; mb < 8; ++mb) {
      const int ml = wm * WM + mb * 16 + lrow;
      const f32x4 v = acc[nb][mb];
      const uint32_t base = (uint32_t)(ml * p.ldc + n) * 2u;
      if (VEC && n + 3 < p.N) {
        v2u w;
        w.x = pack_bf16x2(v[0], v[1]);
        w.y = pack_bf16x2(v[2], v[3]);
        __builtin_amdgcn_raw_buffer_store_b64(w, rsc, base, 0, 0);
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const __bf16 h = (__bf16)v[r];
          __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(unsigned short, h), rsc,
                                                n + r < p.N ? base + 2u * r : kOOB, 0, 0);
        }
      }
    }
  }
}

template <bool VEC>
__global__ void __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(1, 1)))
gemm_bf16_persistent(Params p) {
  __shared__ __attribute__((aligned(16))) uint16_t sA[2 * BM * LDP];
  __shared__ __attribute__((aligned(16))) uint16_t sB[2 * BN * LDP];
  __shared__ int s_info[2];

  if (p.mapping == ASYM_MAP_AWARE) {
    const int xcc = (int)read_xcc_id();
    if (threadIdx.x == 0) {
      int r = -1;
      if (xcc < p.n_xccs) r = atomicAdd(&p.ctr[xcc], 1);
      s_info[0] = (xcc < p.n_xccs && r < p.slots[xcc]) ? 1 : 0;
    }
    __syncthreads();
    if (s_info[0]) {
      for (;;) {
        if (threadIdx.x == 0) {
          int tile = -1;
          for (int d = 0; d < p.n_xccs && tile < 0; ++d) {
            const int y = (xcc + d) % p.n_xccs;
            const int q = p.off[y + 1] - p.off[y];
            if (q <= 0) continue;
            // a cheap read first, so exhausted regions are not hammered
            if (__hip_atomic_load(&p.ctr[16 + y], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= q) continue;
            const int t = atomicAdd(&p.ctr[16 + y], 1);
            if (t < q) tile = p.order[p.off[y] + t];
          }
          s_info[1] = tile;
        }
        __syncthreads();
        const int tile = s_info[1];
        if (tile < 0) break;
        compute_tile<VEC>(p, tile, sA, sB);
      }
    }
    // the last workgroup to leave resets the counters for the next launch
    if (threadIdx.x == 0) {
      __threadfence();
      const int done = atomicAdd(&p.ctr[32], 1);
      if (done == (int)gridDim.x - 1) {
        for (int i = 0; i < 33; ++i) atomicExch(&p.ctr[i], 0);
        __threadfence();
      }
    }
  } else {
    for (int i = blockIdx.x; i < p.n_tiles; i += gridDim.x) compute_tile<VEC>(p, p.order[i], sA, sB);
  }
}

}  // namespace

int launch_gemm(const GemmLaunch& g, hipStream_t s) {
  Params p;
  p.A = static_cast<const uint16_t*>(g.A);
  p.B = static_cast<const uint16_t*>(g.B);
  p.C = static_cast<uint16_t*>(g.C);
  p.M = g.M; p.N = g.N; p.K = g.K;
  p.lda = g.lda; p.ldb = g.ldb; p.ldc = g.ldc;
  p.tiles_m = g.tiles_m; p.tiles_n = g.tiles_n; p.n_tiles = g.tiles_m * g.tiles_n;
  p.mapping = g.mapping;
  p.n_xccs = g.n_xccs;
  p.order = g.d_order; p.off = g.d_off; p.slots = g.d_slots; p.ctr = g.d_ctr;
  if (g.vec)
    hipLaunchKernelGGL(gemm_bf16_persistent<true>, dim3(g.grid), dim3(NT), 0, s, p);
  else
    hipLaunchKernelGGL(gemm_bf16_persistent<false>, dim3(g.grid), dim3(NT), 0, s, p);
  ASYM_HIP(hipGetLastError());
  return ASYM_OK;
}

int gemm_tile_m() { return BM; }
int gemm_tile_n() { return BN; }

}  // namespace asym
