// Persistent bf16 GEMM for gfx950 with XCD-aware tile placement.
//
// Section 7.1 ("Integration with popular kernels") makes a kernel
// asymmetry-aware by running one persistent block per compute unit, finding
// the unit each block runs on, and giving it the tasks whose data is local to
// that unit's partition, with work in proportion to each partition's units.
// Here a task is a 256x256 output tile and the partition is the XCD (private
// 4 MB L2).  On gfx950 workgroups are dealt to the XCDs round-robin by launch
// index, so every residue class of block indices mod n lands on one XCD (the
// identity probe measures this); which XCD a class lands on depends on where
// the dealing starts, which has differed between streams.  Where the CU set
// has the same count on every XCD, AWARE mode needs only the classes: workgroup
// b is the (b / n)-th worker of region b mod n of the schedule and runs it with
// a stride of the region's worker count.  A region's workers then share one
// L2 whatever the rotation, no counters or atomics are involved, and every
// tile is computed whatever the actual placement.  Where the XCD's identity
// matters (unequal CU counts, a whole-XCD restriction) workgroups read XCC_ID
// and claim tiles instead (dynamic form below).  The OBLIVIOUS modes walk one
// shared order (tile i on workgroup i mod P), which is how a persistent GEMM
// without topology knowledge runs.
//
// C = A . B with A [M][lda], B stored [N][ldb] (K contiguous), C [M][ldc], all
// bf16; fp32 accumulation in the matrix cores (v_mfma_f32_16x16x32_bf16);
// bf16 round-to-nearest-even output (v_cvt_pk_bf16_f32).
//
// Tile 256x256, 256 threads = 4 waves in a 2x2 grid, 128x128 per wave (8x8
// MFMA blocks, 256 fp32 accumulators per lane in AGPRs).
//
// Vector path (16-byte aligned operands, K a multiple of 8): k advances in
// stages of 64 through LDS rings, three slots for A and two for B (32 KiB per
// slot at the 256-wide tile, 160 KiB in all).  Operands go from HBM straight
// into LDS with buffer_load_dwordx4 ... lds (no staging registers, no LDS
// write instructions), eight lanes per whole 128-byte line; A's loads for
// stage t+2 are issued during the first half of stage t and B's during the
// second half, so MFMA work covers their latency.  Inside a row the eight
// 16-byte chunks are stored XOR-swizzled by (row >> 1) & 7, which keeps the 16
// rows read by one ds_read_b128 free of bank conflicts.  MFMA fragments are
// double-buffered: the next half-stage's fragments are read while the current
// half-stage's 64 MFMAs run.  One barrier per stage publishes the next stage;
// waits on the loads are explicit, so the barrier does not drain the
// prefetch.  Tiles 224 and 192 wide (7 and 6 B fragments per wave) exist for
// shapes whose tile count fits the workers better at those widths.
//
// Generic path (any alignment or K): 256x256x64 tiles, register-staged
// element loads into two padded LDS stages.
#include <hip/hip_runtime.h>

#include <type_traits>

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
  int* ctr;          // dynamic aware: [0,16) rank tickets, [16,32) tile counters, [32] exits
  int dynamic;       // aware mapping with claims instead of the static assignment
  const int4* desc;  // grouped GEMM: per tile {first row, rows, group's first B row, first column}
  asym_wg_record* trace;  // traced launches: one record per workgroup (null otherwise)
};

// Where a tile lies.  Plain GEMM: tile = row-major index in the tile grid.
// Grouped GEMM (Section 7.1 applies the recipe to grouped GEMM, the expert
// layer of mixture-of-experts models): tile = index into `desc`; its rows are
// rows [m0, m0 + rows) of the packed A and C (the group's rows, at most BM),
// and its B rows are the group's weight rows b0 + [n0, n0 + width).
struct TileGeom {
  int m0, rows, b0, n0;
};

__device__ __forceinline__ TileGeom tile_geom(const Params& p, int tile, int width, int height = BM) {
  TileGeom g;
  if (p.desc) {
    const int4 d = p.desc[tile];
    g.m0 = __builtin_amdgcn_readfirstlane(d.x);
    g.rows = __builtin_amdgcn_readfirstlane(d.y);
    g.b0 = __builtin_amdgcn_readfirstlane(d.z);
    g.n0 = __builtin_amdgcn_readfirstlane(d.w);
  } else {
    const int tm = tile / p.tiles_n, tn = tile - tm * p.tiles_n;
    g.m0 = tm * height;
    g.rows = min(height, p.M - g.m0);
    g.b0 = 0;
    g.n0 = tn * width;
  }
  return g;
}

// Buffer resource over `bytes` bytes at `base`: loads beyond the range return
// zero and stores beyond it are dropped, so tile edges need no branches.
// Every argument here is the same in all lanes; reading it from the first lane
// tells the compiler so, and the resource stays in SGPRs (a resource it takes
// for lane-varying is re-checked lane by lane around every access).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  const unsigned long long a = (unsigned long long)base;
  const unsigned long long u = ((unsigned long long)__builtin_amdgcn_readfirstlane((uint32_t)(a >> 32)) << 32) |
                               (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)a);
  return __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<void*>(u), (short)0,
                                           (int)__builtin_amdgcn_readfirstlane(bytes), 0x00020000);
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
template <bool VEC, int NR = 8>
__device__ __forceinline__ void load_tile(uint4 (&r)[NR], __amdgpu_buffer_rsrc_t rs, int ld,
                                          uint32_t vo, int K, int k0) {
  const int kc = (threadIdx.x & 7) * 8;
  if constexpr (VEC) {
    const uint32_t v = k0 + kc < K ? vo : kOOB;
#pragma unroll
    for (int i = 0; i < NR; ++i) {
      const int so = (32 * i * ld + k0) * 2;
      const v4u x = __builtin_amdgcn_raw_buffer_load_b128(rs, v, so, 0);
      r[i] = make_uint4(x.x, x.y, x.z, x.w);
    }
  } else {
#pragma unroll
    for (int i = 0; i < NR; ++i) {
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

template <int NR = 8>
__device__ __forceinline__ void store_tile(uint16_t* __restrict__ s, const uint4 (&r)[NR]) {
  const int t = threadIdx.x;
  const int kc = (t & 7) * 8;
#pragma unroll
  for (int i = 0; i < NR; ++i) {
    const int row = (t >> 3) + 32 * i;
    *reinterpret_cast<uint4*>(s + row * LDP + kc) = r[i];
  }
}

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  bf16x2 v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

// Register-staged path: tiles TE x TE (TE = 256, or 128 for products too
// small to give every CU a 256-wide tile), 4 waves of TE/2 x TE/2, k-stages
// of 64 in two padded LDS buffers.  Each output is the same chain of MFMAs as
// on the vector path (k-stages in order, two 32-wide steps each), so every
// tile size gives the same bits.
template <bool VEC, int TE = 256>
__device__ __forceinline__ void compute_tile(const Params& p, int tile, uint16_t* sA, uint16_t* sB) {
  constexpr int TW = TE / 2;      // per-wave rows and columns
  constexpr int FR = TW / 16;     // fragments per wave and dimension
  constexpr int NR = TE / 32;     // rows per thread in the tile loads
  const TileGeom tg = tile_geom(p, tile, TE, TE);
  const int m0 = tg.m0, n0 = tg.n0;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int KT = (p.K + BK - 1) / BK;

  f32x4 acc[FR][FR];
#pragma unroll
  for (int i = 0; i < FR; ++i)
#pragma unroll
    for (int j = 0; j < FR; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int rows_a = tg.rows, rows_b = min(TE, p.N - n0);
  const __amdgpu_buffer_rsrc_t rsa = make_rsrc(p.A + (size_t)m0 * p.lda, (uint32_t)rows_a * p.lda * 2u);
  const __amdgpu_buffer_rsrc_t rsb =
      make_rsrc(p.B + (size_t)(tg.b0 + n0) * p.ldb, (uint32_t)rows_b * p.ldb * 2u);
  const uint32_t voa = (uint32_t)((threadIdx.x >> 3) * p.lda + (threadIdx.x & 7) * 8) * 2u;
  const uint32_t vob = (uint32_t)((threadIdx.x >> 3) * p.ldb + (threadIdx.x & 7) * 8) * 2u;
  uint4 ra[NR], rb[NR];
  load_tile<VEC, NR>(ra, rsa, p.lda, voa, p.K, 0);
  load_tile<VEC, NR>(rb, rsb, p.ldb, vob, p.K, 0);
  store_tile<NR>(sA, ra);
  store_tile<NR>(sB, rb);
  __syncthreads();

  const int lrow = lane & 15, lk = (lane >> 4) * 8;
  for (int kt = 0; kt < KT; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < KT;
    if (more) {
      load_tile<VEC, NR>(ra, rsa, p.lda, voa, p.K, (kt + 1) * BK);
      load_tile<VEC, NR>(rb, rsb, p.ldb, vob, p.K, (kt + 1) * BK);
    }
    const uint16_t* a_s = sA + cur * (TE * LDP) + (wm * TW + lrow) * LDP + lk;
    const uint16_t* b_s = sB + cur * (TE * LDP) + (wn * TW + lrow) * LDP + lk;
#pragma unroll
    for (int ks = 0; ks < BK / 32; ++ks) {
      bf16x8 xa[FR], xb[FR];
#pragma unroll
      for (int i = 0; i < FR; ++i) {
        xa[i] = *reinterpret_cast<const bf16x8*>(a_s + i * 16 * LDP + ks * 32);
        xb[i] = *reinterpret_cast<const bf16x8*>(b_s + i * 16 * LDP + ks * 32);
      }
#pragma unroll
      for (int nb = 0; nb < FR; ++nb)
#pragma unroll
        for (int mb = 0; mb < FR; ++mb)
          acc[nb][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xb[nb], xa[mb], acc[nb][mb], 0, 0, 0);
    }
    if (more) {
      store_tile<NR>(sA + (cur ^ 1) * (TE * LDP), ra);
      store_tile<NR>(sB + (cur ^ 1) * (TE * LDP), rb);
    }
    __syncthreads();
  }

  // epilogue: lane holds C[m][n..n+3] for each (nb, mb) block; rows past M
  // fall outside the resource and their stores are dropped
  const int rows_c = tg.rows;
  const __amdgpu_buffer_rsrc_t rsc = make_rsrc(p.C + (size_t)m0 * p.ldc, (uint32_t)rows_c * p.ldc * 2u);
#pragma unroll
  for (int nb = 0; nb < FR; ++nb) {
    const int n = n0 + wn * TW + nb * 16 + (lane >> 4) * 4;
#pragma unroll
    for (int mb = 0; mb < FR; ++mb) {
      const int ml = wm * TW + mb * 16 + lrow;
      const f32x4 v = acc[nb][mb];
      const uint32_t base = (uint32_t)(ml * p.ldc + n) * 2u;
      if (VEC && n + 3 < p.N && ((((uintptr_t)p.C) & 7u) == 0) && (p.ldc % 4 == 0)) {
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

// ---- vector path: direct-to-LDS rings ---------------------------------------------
// k advances in stages of 64.  A stage of A (256 rows) and one of B (16 * nbf * 2
// rows, nbf = 16-column B fragments per wave: 8, 7 or 6 for 256-, 224- and
// 192-wide tiles) each hold one 128-byte line of every row.  A has three ring
// slots and B two: A's loads for stage t+2 go out during the first half of
// stage t and B's during the second half, so the load path is busy evenly
// instead of in bursts (a load that cannot issue holds up the MFMAs behind it).
// 3 x 32 KiB + 2 x 32 KiB fill the 160 KiB of LDS at the 256-wide tile.
constexpr int KS = 64;                 // k per stage: one 128-byte line of every row
constexpr int A_SLOTS = 3, B_SLOTS = 2;
constexpr int ROW_BYTES = KS * 2;
constexpr int A_BYTES = BM * ROW_BYTES;                 // one stage of A (32 KiB)
constexpr int A_RING = A_SLOTS * A_BYTES;
template <int NBF> constexpr int b_bytes() { return 32 * NBF * ROW_BYTES; }  // one stage of B
constexpr int RING_BYTES = A_RING + B_SLOTS * b_bytes<8>();  // the widest tile

typedef int i32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ i32x4 rsrc_words(const void* base, uint32_t bytes) {
  const unsigned long long a = (unsigned long long)base;
  return i32x4{(int)(uint32_t)a, (int)(uint32_t)(a >> 32), (int)bytes, 0x00020000};
}

// Direct-to-LDS load of 8 tile rows x 128 bytes (1 KiB): lane L lands at
// M0 + 16 L, i.e. row L/8 of the 8, physical chunk L%8; `vo` already selects
// the logical chunk that belongs there, `so` the row block and k (uniform).
// Eight lanes read one whole 128-byte line of a row: loads of half lines (a
// 32-wide k stage) reach barely 60% of this rate through the vector cache.
// `row` (the row block's byte offset) and `kb` (the stage's k byte offset)
// are added in the scalar unit inside the asm, so no part of the address
// passes through vector registers.  The add writes SCC, which the compiler
// must not keep a value in across the asm (declared clobbered), and M0.
__device__ __forceinline__ void dma_1k(uint32_t lds_dst, i32x4 rs, uint32_t vo, int row, int kb) {
  int so;
  asm volatile("s_add_u32 %0, %1, %2\n\ts_mov_b32 m0, %3\n\tbuffer_load_dwordx4 %4, %5, %0 offen lds"
               : "=&s"(so)
               : "s"(row), "s"(kb), "s"(lds_dst), "v"(vo), "s"(rs)
               : "memory", "scc", "m0");
}

__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// acc += A . B on the matrix cores, with the accumulator pinned to AGPRs and
// the fragments to VGPRs.  Issued as inline asm so the register files and the
// issue order are exactly as written; the compiler does not see these MFMAs,
// so the hazard padding around them is explicit (mfma_fence()).
__device__ __forceinline__ void mfma_acc(f32x4& acc, const bf16x8& a, const bf16x8& b) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
}

// Wait states between VALU accesses of accumulators and the MFMAs that use
// them (covers the longest MFMA-to-VALU dependency of the 16x16x32 shape).
__device__ __forceinline__ void mfma_fence() {
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
}

// 16-byte LDS read of one MFMA fragment into VGPRs.  Issued as inline asm so
// the compiler neither tracks nor waits on it: the stage that consumes the
// fragment starts with lds_barrier(), whose lgkmcnt(0) is the wait, and the
// fragment's registers are not touched before that (checked in the ISA).
template <int OFF>
__device__ __forceinline__ void lds_read_frag(bf16x8& f, uint32_t addr) {
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(f) : "v"(addr), "i"(OFF) : "memory");
}
// A fragments G .. 7 (after the last B group of a tile narrower than 256)
template <int G>
__device__ __forceinline__ void lds_read_frags_from(bf16x8 (&f)[8], uint32_t addr) {
  if constexpr (G < 8) {
    lds_read_frag<G * 2048>(f[G], addr);
    lds_read_frags_from<G + 1>(f, addr);
  }
}

struct RingCtx {
  i32x4 rsa, rsb;
  uint32_t voa[2], vob[2];  // per-lane offsets for even / odd 8-row blocks
  uint32_t dst_a, dst_b;
  int row_a[8], row_b[8];   // byte offsets of the wave's 8-row blocks
  int K;
  int lca[2], lcb[2];       // the lane's logical chunk for even / odd blocks of A, B
};

// The workgroup's next tile.  Static assignment: positions i, i + step,
// i + 2 step, ... (< end) of the tile order: for the oblivious mappings the
// whole order with step = the grid; for the aware mapping the region of the
// workgroup's XCD with step = the XCD's workgroup count.  Dynamic (aware on an
// uneven CU set): claims on a per-XCD counter.  Lane 0 issues the fetch right
// after a tile's k-loop has drained (issue_next); nothing reads it until the
// epilogue's stores are issued (take_next).  Issuing it inside the k-loop
// instead would hold up the ring: the value must stay live across the
// remaining stages, where every VGPR is taken, so it is spilled, and the
// spill waits on memory.
struct NextTile {
  const int* order;
  int* counter;      // dynamic: the own XCD's tile counter; null for static
  int own_off, own_q;
  int i_next, step, end;
  int v;             // lane 0: the claim or the order entry in flight
};

__device__ __forceinline__ void issue_next(NextTile& n) {
  if (threadIdx.x != 0) return;
  if (n.counter)
    n.v = atomicAdd(n.counter, 1);
  else
    n.v = n.order[n.i_next < n.end ? n.i_next : 0];
}

__device__ __forceinline__ int steal_aware(const Params& p, int xcc, int q_lane);

// Wave 0 (all lanes): the next tile, or -1.  Dynamic: the index claimed by
// lane 0 is looked up in the XCD's list; once the own region is exhausted,
// other regions are tried.
__device__ __forceinline__ int take_next(const Params& p, const NextTile& n, int xcc, int q_lane) {
  if (n.counter) {
    const int idx = __builtin_amdgcn_readfirstlane(n.v);
    if (idx < n.own_q) return __builtin_amdgcn_readfirstlane(n.order[n.own_off + idx]);
    return steal_aware(p, xcc, q_lane);
  }
  const int v = __builtin_amdgcn_readfirstlane(n.v);
  return n.i_next < n.end ? v : -1;
}

// The per-lane load offsets of one stage: the lane's chunk of its row, or an
// offset past the range (a zero fill) where that chunk starts at or beyond K.
// Computed once per stage, so the loads themselves need no vector arithmetic.
struct StageOffsets {
  uint32_t a[2], b[2];  // even / odd 8-row blocks
};

__device__ __forceinline__ StageOffsets stage_offsets(const RingCtx& c, int t) {
  const int k0 = t * KS;
  StageOffsets o;
#pragma unroll
  for (int par = 0; par < 2; ++par) {
    o.a[par] = k0 + c.lca[par] * 8 < c.K ? c.voa[par] : kOOB;
    o.b[par] = k0 + c.lcb[par] * 8 < c.K ? c.vob[par] : kOOB;
  }
  return o;
}

// j-th of the 8 + NBF loads of stage t: j < 8 are A's, into A slot t % 3, the
// rest B's, into B slot t % 2; each wave owns 64 rows of A and 8 * NBF rows of
// B, load i covering 8 of them.  `sa_t` is A slot t's byte offset.  The LDS
// address and the row/k offset are uniform (scalar registers); stages past
// the end of K read zeros or go unused.
template <int NBF>
__device__ __forceinline__ void ring_load(const RingCtx& c, const StageOffsets& o, int t, uint32_t sa_t,
                                          int j) {
  const int kb = __builtin_amdgcn_readfirstlane(t * KS * 2);
  if (j < 8)
    dma_1k(c.dst_a + sa_t + j * 1024, c.rsa, o.a[j & 1], c.row_a[j], kb);
  else
    dma_1k(c.dst_b + (uint32_t)(t & 1) * b_bytes<NBF>() + (j - 8) * 1024, c.rsb, o.b[(j - 8) & 1],
           c.row_b[j - 8], kb);
}

// One group of a half-stage (32 of the stage's 64 k): the 8 MFMAs that use B
// fragment G, with the group's other work spread between them: the group's
// share of stage t+2's loads (HALF 0: A's 8, HALF 1: B's NBF; the first right
// after the group's first MFMA, the rest after the first four), then the next
// half-stage's A fragment G into `an`, and after the last four MFMAs its B
// fragment G into `b` (B fragment G has no later use in this half-stage, so it
// is replaced in place; the A fragments feed every group and are double
// buffered).  Spreading the loads and reads keeps the MFMAs fed better than
// bursts do; a load placed before the group's first MFMA (right after the
// previous group's LDS read) measured 1.8% slower at 8192^3.  The last group
// is different: nothing follows it in the half-stage to cover a read issued
// after its MFMAs, and the next half-stage starts by waiting for every read.
// So the last B fragment is double buffered (`bl`: HALF h computes with bl[h]
// and reads the next half-stage's into bl[1 - h]) and the last group issues
// its reads, and the remaining A fragments of a tile narrower than 256, within
// its first two MFMAs.  `sa`/`sb` are the LDS addresses of the next half-stage's
// fragment 0; `sa2` is A slot (t+2)'s byte offset.
template <int NBF, int G, int HALF>
__device__ __forceinline__ void ring_group(const RingCtx& c, const StageOffsets& o, int t, uint32_t sa2,
                                           f32x4 (&acc)[NBF][8], const bf16x8 (&ac)[8],
                                           bf16x8 (&an)[8], bf16x8 (&b)[NBF], bf16x8 (&bl)[2],
                                           uint32_t sa, uint32_t sb) {
  constexpr int lo = HALF == 0 ? G * 8 / NBF : 8 + G, hi = HALF == 0 ? (G + 1) * 8 / NBF : 9 + G;
  if constexpr (G + 1 < NBF) {
    mfma_acc(acc[G][0], b[G], ac[0]);
    if constexpr (lo < hi) ring_load<NBF>(c, o, t + 2, sa2, lo);
#pragma unroll
    for (int mb = 1; mb < 4; ++mb) mfma_acc(acc[G][mb], b[G], ac[mb]);
#pragma unroll
    for (int j = lo + 1; j < hi; ++j) ring_load<NBF>(c, o, t + 2, sa2, j);
    lds_read_frag<G * 2048>(an[G], sa);
#pragma unroll
    for (int mb = 4; mb < 8; ++mb) mfma_acc(acc[G][mb], b[G], ac[mb]);
    lds_read_frag<G * 2048>(b[G], sb);
    ring_group<NBF, G + 1, HALF>(c, o, t, sa2, acc, ac, an, b, bl, sa, sb);
  } else {
    lds_read_frag<G * 2048>(bl[1 - HALF], sb);
    mfma_acc(acc[G][0], bl[HALF], ac[0]);
    if constexpr (lo < hi) ring_load<NBF>(c, o, t + 2, sa2, lo);
    mfma_acc(acc[G][1], bl[HALF], ac[1]);
    lds_read_frags_from<G>(an, sa);
#pragma unroll
    for (int mb = 2; mb < 4; ++mb) mfma_acc(acc[G][mb], bl[HALF], ac[mb]);
#pragma unroll
    for (int j = lo + 1; j < hi; ++j) ring_load<NBF>(c, o, t + 2, sa2, j);
#pragma unroll
    for (int mb = 4; mb < 8; ++mb) mfma_acc(acc[G][mb], bl[HALF], ac[mb]);
  }
}

// Stage t in two halves, branch-free.  First half (k 0..31): its fragments
// were read during the previous half; wait for those reads, compute, load A of
// stage t+2 into A slot (t+2) % 3 (last read in the first half of stage t-1,
// which every wave has left: the barrier of stage t-1), and read the second
// half's fragments from the slots of stage t.  Second half (k 32..63): wait
// for this wave's loads of stage t+1 (all but the 8 A loads just issued; loads
// complete in order), publish stage t+1 to all waves (the barrier also tells
// every wave that B slot t % 2 has been read completely), load B of stage t+2
// into it while computing, and read the first half of stage t+1.  Every
// instruction is inline asm, so the issue order is the program order.
// `sa` holds A slot offsets of stages t, t+1, t+2.
template <int NBF>
__device__ __forceinline__ void ring_stage(const RingCtx& c, int t, const uint32_t (&sa)[3],
                                           f32x4 (&acc)[NBF][8], bf16x8 (&a0)[8], bf16x8 (&a1)[8],
                                           bf16x8 (&b)[NBF], bf16x8 (&bl)[2], const uint32_t (&ra)[2],
                                           const uint32_t (&rb)[2]) {
  const uint32_t sb0 = (uint32_t)(t & 1) * b_bytes<NBF>();
  const uint32_t sb1 = (uint32_t)((t + 1) & 1) * b_bytes<NBF>();
  const StageOffsets o = stage_offsets(c, t + 2);
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  ring_group<NBF, 0, 0>(c, o, t, sa[2], acc, a0, a1, b, bl, ra[1] + sa[0], rb[1] + sb0);
  asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
  lds_barrier();
  ring_group<NBF, 0, 1>(c, o, t, sa[2], acc, a1, a0, b, bl, ra[0] + sa[1], rb[0] + sb1);
}

// An empty asm that redefines one column block's accumulators in AGPRs: the
// values read after it exist only from here on, so their copies to VGPRs
// cannot be scheduled above it (an input-only operand would leave the compiler
// free to copy all 256 accumulators out at the loop exit, and spill).
__device__ __forceinline__ void keep_agprs(f32x4 (&a)[8]) {
  asm volatile("" : "+a"(a[0]), "+a"(a[1]), "+a"(a[2]), "+a"(a[3]), "+a"(a[4]), "+a"(a[5]), "+a"(a[6]), "+a"(a[7]));
}

// The same for one row block of the paired column blocks (0 .. 5 of a tile
// narrower than 256; an odd last block is stored on its own).
template <int NBF>
__device__ __forceinline__ void keep_agprs_row(f32x4 (&a)[NBF][8], int mb) {
  static_assert(NBF == 6 || NBF == 7, "rows are kept for the narrower tiles only");
  asm volatile("" : "+a"(a[0][mb]), "+a"(a[1][mb]), "+a"(a[2][mb]), "+a"(a[3][mb]), "+a"(a[4][mb]), "+a"(a[5][mb]));
}

template <int NBF>
__device__ __forceinline__ void compute_tile_ring(const Params& pin, int tile, unsigned char* lds,
                                                  NextTile& nt) {
  constexpr int WNT = 16 * NBF, BNT = 2 * WNT;  // per-wave and per-tile B width
  // Everything the tile needs passes through an opaque move first, so that no
  // per-lane setup is hoisted out of the tile loop and kept live (and spilled)
  // across the k-loop; recomputing it per tile costs a few instructions.
  Params p = pin;
  int tid = threadIdx.x;
  asm volatile("" : "+v"(tid), "+s"(p.K), "+s"(p.lda), "+s"(p.ldb), "+s"(p.ldc), "+s"(p.M), "+s"(p.N));
  // (and is then read from the first lane, which marks it uniform: address
  // arithmetic on it stays scalar instead of going through vector registers)
  p.K = __builtin_amdgcn_readfirstlane(p.K);
  p.lda = __builtin_amdgcn_readfirstlane(p.lda);
  p.ldb = __builtin_amdgcn_readfirstlane(p.ldb);
  p.ldc = __builtin_amdgcn_readfirstlane(p.ldc);
  p.M = __builtin_amdgcn_readfirstlane(p.M);
  p.N = __builtin_amdgcn_readfirstlane(p.N);
  const TileGeom tg = tile_geom(p, tile, BNT);
  const int m0 = tg.m0, n0 = tg.n0;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int KT = (p.K + KS - 1) / KS;

  f32x4 acc[NBF][8];
#pragma unroll
  for (int i = 0; i < NBF; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  mfma_fence();
  const int rows_a = tg.rows, rows_b = min(BNT, p.N - n0);
  const i32x4 rsa = rsrc_words(p.A + (size_t)m0 * p.lda, (uint32_t)rows_a * p.lda * 2u);
  const i32x4 rsb = rsrc_words(p.B + (size_t)(tg.b0 + n0) * p.ldb, (uint32_t)rows_b * p.ldb * 2u);
  // load side: lane -> (row in its 8-row block, physical chunk L%8); the
  // logical chunk stored there is the physical one XOR (row/2)%8, which for a
  // row 8b + r (b the block's index in the tile) is (r/2) | 4*(b%2): one
  // offset for even blocks, one for odd.  A wave's A blocks start at block
  // 8w (even); its B blocks start at block NBF*w, odd for odd NBF and w.
  const int lrow = lane >> 3;
  const int wv = __builtin_amdgcn_readfirstlane(wave);
  const int bsw = (wv * NBF) & 1;
  int lca[2], lcb[2], voa[2], vob[2];
#pragma unroll
  for (int par = 0; par < 2; ++par) {
    lca[par] = (lane & 7) ^ ((lrow >> 1) | (par << 2));
    lcb[par] = (lane & 7) ^ ((lrow >> 1) | ((par ^ bsw) << 2));
    voa[par] = ((wv * 64 + lrow) * p.lda + lca[par] * 8) * 2;
    vob[par] = ((wv * 8 * NBF + lrow) * p.ldb + lcb[par] * 8) * 2;
  }
  const uint32_t lds0 = (uint32_t)(size_t)lds;
  const uint32_t dst_a = __builtin_amdgcn_readfirstlane(lds0 + wv * 64 * ROW_BYTES);
  const uint32_t dst_b = __builtin_amdgcn_readfirstlane(lds0 + A_RING + wv * 8 * NBF * ROW_BYTES);
  // read side: lane -> row l%16 of a 16-row block, logical chunk l/16 (+4 for
  // the second half-stage), stored at that chunk XOR (row/2)%8: conflict-free
  // 16-byte reads across every 16 lanes
  const int rrow = lane & 15;
  uint32_t ra[2], rb[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int pchunk = ((lane >> 4) | (h << 2)) ^ ((rrow >> 1) & 7);
    ra[h] = lds0 + (uint32_t)((wm * 128 + rrow) * ROW_BYTES + pchunk * 16);
    rb[h] = lds0 + (uint32_t)(A_RING + (wn * WNT + rrow) * ROW_BYTES + pchunk * 16);
  }

  RingCtx c{rsa, rsb, {(uint32_t)voa[0], (uint32_t)voa[1]}, {(uint32_t)vob[0], (uint32_t)vob[1]},
            dst_a, dst_b, {}, {}, p.K, {lca[0], lca[1]}, {lcb[0], lcb[1]}};
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    c.row_a[i] = __builtin_amdgcn_readfirstlane(8 * i * p.lda * 2);
    c.row_b[i] = __builtin_amdgcn_readfirstlane(8 * i * p.ldb * 2);
  }
  // prologue: stages 0 and 1 in flight (a stage past K loads zeros); stage 0
  // published and its first half's fragments read
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const StageOffsets o = stage_offsets(c, t);
#pragma unroll
    for (int j = 0; j < 8 + NBF; ++j) ring_load<NBF>(c, o, t, (uint32_t)t * A_BYTES, j);
  }
  asm volatile("s_waitcnt vmcnt(%0)" :: "n"(8 + NBF) : "memory");
  lds_barrier();
  // (B fragments 0 .. NBF-2 in bf, the last one in bl[0]: see ring_group)
  bf16x8 a0[8], a1[8], bf[NBF], bl[2];
  lds_read_frags_from<0>(a0, ra[0]);
  lds_read_frag<0>(bf[0], rb[0]); lds_read_frag<2048>(bf[1], rb[0]);
  lds_read_frag<4096>(bf[2], rb[0]); lds_read_frag<6144>(bf[3], rb[0]);
  lds_read_frag<8192>(bf[4], rb[0]);
  if constexpr (NBF > 6) lds_read_frag<10240>(bf[5], rb[0]);
  if constexpr (NBF > 7) lds_read_frag<12288>(bf[6 % NBF], rb[0]);
  lds_read_frag<(NBF - 1) * 2048>(bl[0], rb[0]);
  // A slot offsets of stages t, t+1, t+2 (uniform, rotated each stage)
  uint32_t sa[3] = {0u, (uint32_t)A_BYTES, 2u * A_BYTES};
  for (int t = 0; t < KT; ++t) {
    ring_stage<NBF>(c, t, sa, acc, a0, a1, bf, bl, ra, rb);
    const uint32_t s0 = sa[0];
    sa[0] = sa[1];
    sa[1] = sa[2];
    sa[2] = s0;
  }
  // Right after the k-loop, in one asm statement (nothing the compiler places
  // after the loop can come before it): drain the loads still in flight (zero
  // fills past K) before the slots are reused, let this wave's last fragment
  // reads land, and give the last MFMAs their wait states before anything
  // reads the accumulators.
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
  issue_next(nt);
  // every wave is past its last LDS read before the slots are reused
  lds_barrier();

  // epilogue.  In a 16x16 block the lane with row r = lane % 16 holds columns
  // 4c .. 4c+3, c = lane / 16.  Blocks 2q and 2q+1 are paired by one
  // v_permlane16_swap per packed word, after which lane (r, c) holds 8
  // consecutive columns, 8 (c >> 1) .. +7 of block 2q + (c & 1): one 16-byte
  // store per lane covers 16 rows x 32 columns (64 bytes of each row), so two
  // stores, pairs q and q+1, fill a 128-byte line of C.  The order of the
  // stores and their cache policy depend on the tile width (below).  An odd
  // last block (224-wide tiles) keeps the 8-byte layout.  Offsets: the lane's own one is a VGPR, the block's is uniform
  // (scalar offset).  Rows past M fall outside the resource: stores dropped.
  // (the inputs pass through an opaque move so that nothing below is hoisted
  // out of the tile loop and kept live across the k-loop)
  int ldc = p.ldc, nN = p.N, lid = lane;
  const int rows_c = rows_a;
  const __amdgpu_buffer_rsrc_t rsc = make_rsrc(p.C + (size_t)m0 * ldc + n0, (uint32_t)rows_c * ldc * 2u);
  // 16-byte stores need 16-byte aligned rows; otherwise two 8-byte halves
  const bool c16 = (((uintptr_t)p.C & 15u) == 0) && ((ldc & 7) == 0);
  const int r16 = lid & 15, c4 = lid >> 4;
  const int pcol = wn * WNT + (c4 & 1) * 16 + (c4 >> 1) * 8;  // paired layout, first column
  const uint32_t vp = (uint32_t)((wm * WM + r16) * ldc + pcol) * 2u;
  // One paired store: column blocks 2q and 2q+1 of row block mb.  NT is the
  // cache policy of the 16-byte stores (2: non-temporal).
  auto store_pair = [&](auto nt, int q, int mb) {
    const f32x4 v = acc[2 * q][mb], u = acc[2 * q + 1][mb];
    uint32_t w0 = pack_bf16x2(v[0], v[1]), w1 = pack_bf16x2(v[2], v[3]);
    uint32_t u0 = pack_bf16x2(u[0], u[1]), u1 = pack_bf16x2(u[2], u[3]);
    const auto s0 = __builtin_amdgcn_permlane16_swap(w0, u0, false, false);
    const auto s1 = __builtin_amdgcn_permlane16_swap(w1, u1, false, false);
    w0 = s0[0]; u0 = s0[1];
    w1 = s1[0]; u1 = s1[1];
    const int col = n0 + pcol + 32 * q;
    const int so = (mb * 16 * ldc + 32 * q) * 2;
    if (col + 7 < nN) {
      if (c16) {
        __builtin_amdgcn_raw_buffer_store_b128(v4u{w0, w1, u0, u1}, rsc, vp, so, decltype(nt)::value);
      } else {
        __builtin_amdgcn_raw_buffer_store_b64(v2u{w0, w1}, rsc, vp, so, 0);
        __builtin_amdgcn_raw_buffer_store_b64(v2u{u0, u1}, rsc, vp + 8u, so, 0);
      }
    } else {
      const uint32_t wd[4] = {w0, w1, u0, u1};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const unsigned short h = (unsigned short)(wd[e >> 1] >> (16 * (e & 1)));
        __builtin_amdgcn_raw_buffer_store_b16(h, rsc, col + e < nN ? vp + 2u * e : kOOB, so, 0);
      }
    }
  };
  // The store order and cache policy are chosen by tile width, as measured
  // (8192^3 and 4096 x {14336, 4096, 6144} x {4096, 14336}).  256-wide tiles:
  // column-block pairs outer, non-temporal stores (+1.8% at 8192^3 over the
  // default policy).  Narrower tiles: row blocks outer, so the stores that
  // complete a 128-byte line of C follow each other (+2.7% at
  // 4096x14336x4096), default policy (non-temporal stores cost 1.2% there).
  if constexpr (NBF == 8) {
#pragma unroll
    for (int q = 0; q < NBF / 2; ++q) {
      // keep this pair's accumulators in AGPRs up to here, so that they are
      // copied to VGPRs one pair at a time (not all 256 at the loop exit)
      keep_agprs(acc[2 * q]);
      keep_agprs(acc[2 * q + 1]);
#pragma unroll
      for (int mb = 0; mb < 8; ++mb) store_pair(std::integral_constant<int, 2>{}, q, mb);
      // one pair of column blocks at a time, so their VGPR copies stay few
      __builtin_amdgcn_sched_barrier(0);
    }
  } else {
#pragma unroll
    for (int mb = 0; mb < 8; ++mb) {
      keep_agprs_row<NBF>(acc, mb);
#pragma unroll
      for (int q = 0; q < NBF / 2; ++q) store_pair(std::integral_constant<int, 0>{}, q, mb);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  if constexpr (NBF & 1) {
    constexpr int nb = NBF - 1;
    keep_agprs(acc[nb]);
    const int scol = wn * WNT + nb * 16 + c4 * 4;
    const uint32_t vs = (uint32_t)((wm * WM + r16) * ldc + scol) * 2u;
    const int n = n0 + scol;
#pragma unroll
    for (int mb = 0; mb < 8; ++mb) {
      const f32x4 v = acc[nb][mb];
      const int so = mb * 16 * ldc * 2;
      if (n + 3 < nN) {
        __builtin_amdgcn_raw_buffer_store_b64(v2u{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])}, rsc, vs, so, 0);
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const __bf16 h = (__bf16)v[r];
          __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(unsigned short, h), rsc,
                                                n + r < nN ? vs + 2u * r : kOOB, so, 0);
        }
      }
    }
  }
}

// Another XCD's tile for a workgroup whose own region is exhausted (dynamic
// aware mapping), so every tile is computed whatever the hardware's placement
// of workgroups.  Run by all 64 lanes of wave 0: lane y reads XCD y's counter,
// so one round trip shows which regions still have tiles; those are then
// claimed from in turn, starting after the own XCD.  `q_lane` is region y's
// tile count in lane y.  Returns -1 when every region is exhausted.
__device__ __forceinline__ int steal_aware(const Params& p, int xcc, int q_lane) {
  const int lane = threadIdx.x & 63;
  int left = 0;
  if (lane < p.n_xccs)
    left = q_lane - __hip_atomic_load(&p.ctr[16 + lane], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  unsigned long long open = __ballot(left > 0);
  for (int d = 1; d <= p.n_xccs && open; ++d) {
    const int y = (xcc + d) % p.n_xccs;
    if (!((open >> y) & 1ull)) continue;
    int t = 0;
    if (lane == 0) t = atomicAdd(&p.ctr[16 + y], 1);
    t = __builtin_amdgcn_readfirstlane(t);
    const int q = __builtin_amdgcn_readfirstlane(__shfl(q_lane, y));
    if (t < q) return __builtin_amdgcn_readfirstlane(p.order[p.off[y] + t]);
    open &= ~(1ull << y);
  }
  return -1;
}

// TE = 0: the vector path's direct-to-LDS rings (256 x 32 NBF tiles);
// otherwise the register-staged path with TE x TE tiles.
template <bool VEC, int NBF, int TE>
__device__ __forceinline__ void run_tile(const Params& p, int tile, unsigned char* lds, NextTile& nt) {
  if constexpr (TE == 0) {
    compute_tile_ring<NBF>(p, tile, lds, nt);
  } else {
    compute_tile<VEC, TE>(p, tile, reinterpret_cast<uint16_t*>(lds),
                          reinterpret_cast<uint16_t*>(lds) + 2 * TE * LDP);
    issue_next(nt);
  }
}

// Wave 0's value in box[0] (the first word of LDS) to every wave.  Between
// tiles no load into LDS is in flight and no wave reads it, so the word is
// free; the second barrier keeps the next tile's loads from overwriting it
// before every wave has read it.
__device__ __forceinline__ int read_box(const int* box) {
  __syncthreads();
  const int v = __builtin_amdgcn_readfirstlane(box[0]);
  __syncthreads();
  return v;
}

// Per-workgroup record of a traced launch (TRACE): the constant-rate clock
// (s_memrealtime) when the workgroup starts, when its first tile starts and
// when it leaves, the XCC and hardware IDs it ran on and how many tiles it
// computed.  The traced kernels are separate instantiations, so the untraced
// ones carry none of this.
__device__ __forceinline__ unsigned long long wall_clock() { return __builtin_amdgcn_s_memrealtime(); }
__device__ __forceinline__ unsigned long long core_clock() { return __builtin_amdgcn_s_memtime(); }

__device__ __forceinline__ void trace_record(const Params& p, unsigned long long t0, unsigned long long c0,
                                             unsigned long long t_first, int tiles, int worked) {
  if (threadIdx.x != 0) return;
  uint32_t xr, hw;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xr));
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_HW_ID)" : "=s"(hw));
  asym_wg_record r;
  r.start = t0;
  r.first_tile = t_first;
  r.end = wall_clock();
  r.cycles = core_clock() - c0;
  r.xcc = xr & 0xFu;
  r.hw_id = hw;
  r.tiles = (uint32_t)tiles;
  r.worked = (uint32_t)worked;
  p.trace[blockIdx.x] = r;
}

template <bool VEC, int NBF, int TE = 0, bool TRACE = false>
__global__ void __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(1, 1)))
gemm_bf16_persistent(Params p) {
  __shared__ __attribute__((aligned(1024))) unsigned char lds[TE == 0 ? RING_BYTES : 2 * (2 * TE) * LDP * 2];
  int* const box = reinterpret_cast<int*>(lds);  // tile broadcast, used between tiles only
  const unsigned long long t_start = TRACE ? wall_clock() : 0ull;
  const unsigned long long c_start = TRACE ? core_clock() : 0ull;

  // Static aware assignment: workgroup b belongs to XCD b mod n and is that
  // XCD's (b / n)-th persistent worker (the hardware deals workgroups to XCDs
  // round-robin in launch order, the rule the identity probe measures); worker
  // r of XCD x runs positions r, r + s_x, ... of x's region, and workers
  // r >= s_x leave at once.  It covers every tile whatever the actual
  // placement, which decides only the L2 a tile is served from.  It is used
  // when every XCD has at least as many CUs in the stream's set as workgroups
  // are dealt to it, so no workgroup waits behind a full XCD.  Otherwise
  // (uneven CU sets) the dynamic form: a workgroup reads the XCD it runs on,
  // takes a rank ticket there (ranks past the XCD's CU count leave), and
  // claims tiles of that XCD's region from a counter, then of other regions.
  // Oblivious: every workgroup walks the whole order statically.
  const int lane = threadIdx.x & 63;
  const bool aware = p.mapping == ASYM_MAP_AWARE;
  const bool dyn = aware && p.dynamic;
  int xcc = 0, q_lane = 0;
  NextTile nt;
  nt.order = p.order;
  nt.counter = nullptr;
  nt.own_off = 0;
  nt.own_q = 0;
  nt.v = -1;
  if (dyn) {
    uint32_t xr;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xr));
    xcc = (int)(xr & 0xFu);
    const int own = xcc < p.n_xccs ? xcc : 0;
    nt.own_off = __builtin_amdgcn_readfirstlane(p.off[own]);
    nt.own_q = __builtin_amdgcn_readfirstlane(p.off[own + 1] - p.off[own]);
    nt.counter = &p.ctr[16 + own];
    q_lane = lane < p.n_xccs ? p.off[lane + 1] - p.off[lane] : 0;
    nt.i_next = 0;
    nt.step = 0;
    nt.end = 0;
  } else if (aware) {
    const int x = (int)blockIdx.x % p.n_xccs, r = (int)blockIdx.x / p.n_xccs;
    const int s_x = p.slots[x];
    if (r >= s_x) {  // the whole workgroup, before any barrier
      if constexpr (TRACE) trace_record(p, t_start, c_start, 0ull, 0, 0);
      return;
    }
    nt.i_next = p.off[x] + r;
    nt.step = s_x;
    nt.end = p.off[x + 1];
  } else {
    nt.i_next = blockIdx.x;
    nt.step = gridDim.x;
    nt.end = p.n_tiles;
  }
  int tile;
  if (dyn) {
    if (threadIdx.x < 64) {
      int first = -1;
      bool active = xcc < p.n_xccs && p.slots[xcc] > 0;  // no ticket on an XCD outside the set
      if (active) {
        int r = 0;
        if (lane == 0) r = atomicAdd(&p.ctr[xcc], 1);
        active = __builtin_amdgcn_readfirstlane(r) < p.slots[xcc];
      }
      if (active) {
        int idx = 0;
        if (lane == 0) idx = atomicAdd(nt.counter, 1);
        idx = __builtin_amdgcn_readfirstlane(idx);
        first = idx < nt.own_q ? __builtin_amdgcn_readfirstlane(p.order[nt.own_off + idx])
                               : steal_aware(p, xcc, q_lane);
      }
      if (lane == 0) box[0] = first;
    }
    tile = read_box(box);
  } else {
    tile = nt.i_next < nt.end ? __builtin_amdgcn_readfirstlane(p.order[nt.i_next]) : -1;
  }
  const unsigned long long t_first = TRACE ? wall_clock() : 0ull;
  int n_tiles_done = 0;
  while (tile >= 0) {
    nt.i_next += nt.step;
    if constexpr (TRACE) ++n_tiles_done;
    run_tile<VEC, NBF, TE>(p, tile, lds, nt);
    if (threadIdx.x < 64) {
      const int nxt = take_next(p, nt, xcc, q_lane);
      if (lane == 0) box[0] = nxt;
    }
    tile = read_box(box);
  }
  if constexpr (TRACE) trace_record(p, t_start, c_start, t_first, n_tiles_done, n_tiles_done > 0);
  if (dyn && threadIdx.x == 0) {
    // the last workgroup to leave resets the counters for the next launch
    __threadfence();
    const int done = atomicAdd(&p.ctr[32], 1);
    if (done == (int)gridDim.x - 1) {
      for (int c = 0; c < 33; ++c) atomicExch(&p.ctr[c], 0);
      __threadfence();
    }
  }
}

template <bool TRACE>
int launch_gemm_kind(const GemmLaunch& g, const Params& p, hipStream_t s) {
  if (g.bm == 128 && g.bn == 128) {
    if (g.vec)
      hipLaunchKernelGGL((gemm_bf16_persistent<true, 8, 128, TRACE>), dim3(g.grid), dim3(NT), 0, s, p);
    else
      hipLaunchKernelGGL((gemm_bf16_persistent<false, 8, 128, TRACE>), dim3(g.grid), dim3(NT), 0, s, p);
  } else if (g.bm != 256) {
    return fail(ASYM_EINVAL, "gemm: unsupported tile height");
  } else if (!g.vec)
    hipLaunchKernelGGL((gemm_bf16_persistent<false, 8, 256, TRACE>), dim3(g.grid), dim3(NT), 0, s, p);
  else if (g.bn == 256)
    hipLaunchKernelGGL((gemm_bf16_persistent<true, 8, 0, TRACE>), dim3(g.grid), dim3(NT), 0, s, p);
  else if (g.bn == 224)
    hipLaunchKernelGGL((gemm_bf16_persistent<true, 7, 0, TRACE>), dim3(g.grid), dim3(NT), 0, s, p);
  else if (g.bn == 192)
    hipLaunchKernelGGL((gemm_bf16_persistent<true, 6, 0, TRACE>), dim3(g.grid), dim3(NT), 0, s, p);
  else
    return fail(ASYM_EINVAL, "gemm: unsupported tile width");
  ASYM_HIP(hipGetLastError());
  return ASYM_OK;
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
  p.dynamic = g.dynamic ? 1 : 0;
  p.desc = static_cast<const int4*>(g.d_desc);
  p.trace = static_cast<asym_wg_record*>(g.d_trace);
  return g.d_trace ? launch_gemm_kind<true>(g, p, s) : launch_gemm_kind<false>(g, p, s);
}

int gemm_tile_m() { return BM; }
int gemm_tile_n() { return BN; }

}  // namespace asym
