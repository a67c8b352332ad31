// Multi-head latent attention, decode (the MLA workloads of Section 7.1;
// Appendix F counts one compressed row of 512 + 64 values per token).  Each
// request caches one 576-wide row per token, Kc[t] = [c_t (512) ; r_t (64)];
// every query head h has a 576-wide query (the projections absorbed into it):
//
//   O[b, h] = softmax_t(scale * <q[b, h], Kc[b, t]>) . Kc[b, t, 0:512]
//
// All query heads read the same rows, so the rows are the data a placement
// can share: the paper's topology-plus-locality experiment is MLA decode.
//
// Work is split along the sequence (flash-decoding).  A task is one
// (request, split, block of 16 query heads) and runs on one wave:
//   * scores S^T (16 tokens x 16 heads) = K . Q^T on the matrix cores
//     (v_mfma_f32_16x16x32_bf16, 18 steps over the 576 values): the key
//     fragment of a lane is 16 contiguous bytes of one row, loaded from memory
//     straight into operand registers; the 16 query rows stay in registers
//     for the whole task;
//   * an online softmax per head (a lane's accumulators all belong to one
//     head, so the rescaling is a per-lane factor);
//   * O^T (512 x 16 heads) += V^T . P^T on the matrix cores
//     (v_mfma_f32_16x16x16_bf16): a lane's probabilities (4 consecutive
//     tokens, one head) are already the B operand of that product; the
//     values are written to a per-wave LDS tile as they are, one 16-byte
//     store per key fragment already loaded (the latent part of the row is
//     the value, so the rows are read from memory once), and the A operand
//     V^T comes out of it through gfx950's transposing LDS read
//     (ds_read_b64_tr_b16), one per 16 values; token rows are padded by 32
//     bytes so that the reads of 16 rows spread over the banks;
//   * 16-token blocks; the next block's rows go out as soon as a block's
//     fragments are consumed (scores computed, values written), and the
//     output is rescaled only when a head's block maximum exceeds the
//     reference maximum by more than a fixed gap (the reference then follows;
//     below the gap the stale reference keeps the result exact);
//   * multiples of 64 heads run in the workgroup form instead: four waves on
//     four head blocks share each block's rows through one LDS tile.
// Each task writes its unnormalised output, max and sum (fp32); a second
// kernel merges the splits of each (request, head) in an order fixed by the
// split count (several waves per row when there are many splits), so the
// result does not depend on which wave ran which task.
//
// Placement.  Tasks are numbered in one of two orders.  Aware: request-split
// major, the head blocks of one (request, split) consecutive; each XCD gets a
// share of that list in proportion to its CUs in the stream's set, and its
// workgroups claim groups of 4 tasks from it, then from the other shares, so
// the head blocks that read the same rows run on one XCD, close in time (the
// rows cross into its L2 once).  Oblivious: head-block major (a grid over
// heads, then requests and splits), 4 tasks per workgroup in order; the
// hardware deals workgroups round-robin, so the head blocks of one split
// land on different XCDs and each XCD gets the same share whatever its CUs.
#include <hip/hip_runtime.h>

#include "internal.h"
#include "split_merge.h"

namespace asym {
namespace {

constexpr int MD = 576;            // query / key width
constexpr int MV = 512;            // value (latent) width
constexpr int MW = 4;              // tasks per workgroup, one per wave
constexpr int MT = 16;             // tokens per block
constexpr int MSTEPS = MD / 32;    // 18 MFMA steps for the scores
constexpr int VSTEPS = MV / 32;    // 16 of them cover the latent part
constexpr int V_ROW = MV * 2 + 32;  // bytes of one token's values in the per-wave tile, padded
constexpr int V_BYTES = MT * V_ROW;  // 16.5 KiB per wave
constexpr int MG = 4;              // workgroup form: head blocks per workgroup, one per wave
constexpr int MT2 = 32;            // workgroup form: tokens per block
constexpr int K_ROW = MD * 2 + 32; // workgroup form: bytes of one token's row in the shared tile
constexpr int K_BYTES = MT2 * K_ROW;  // 37 KiB per tile, two tiles
constexpr int WG_CHUNKS = (MT2 * (MD / 8) + 64 * MG - 1) / (64 * MG);  // 16-byte loads per thread per block
constexpr int KB = 6;              // workgroup form: score steps per batch of key-fragment reads
constexpr int MG2 = 8;             // 128-head form: head blocks per workgroup, two per wave
constexpr int T2_ROWSLOTS = K_ROW / 16;  // 16-byte slots of a tile row (72 of them data)
constexpr int T2_DMA = 10;         // 128-head form: 1 KiB direct-to-LDS loads per wave per block
constexpr int T2_BYTES = 4 * T2_DMA * 1024;  // 40 KiB per tile (2368 slots used), three tiles
constexpr int T2_TILES = 3;
constexpr int KB2 = 2;             // 128-head form: score steps per batch of key-fragment reads
static_assert(4 * T2_DMA * 64 >= MT2 * T2_ROWSLOTS, "a block's slots must fit the loads");
constexpr uint32_t kMlOOB = 0x80000000u;
constexpr int kMlClaimStride = 64;  // ints between claim counters (256-byte lines)

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned v4u __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) unsigned char lds_u8;
typedef __attribute__((address_space(3))) const bf16x8 lds_bf16x8;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

struct MlaParams {
  const uint16_t* q;     // [B][Hq][576]
  const uint16_t* kv;    // [B][S][576]
  float* part_o;         // [B][Hq][n_splits][512]
  float* part_ml;        // [B][Hq][n_splits][2]: max, sum
  const int* quota_off;  // aware: [n_x + 1] start of each XCD's share (tasks); null = oblivious
  int* claim;            // aware: groups of 4 claimed from share y at claim[y * kMlClaimStride]
  uint32_t allow;        // aware: XCDs whose workgroups may work
  int B, Hq, S, split, n_splits, hblocks, tasks, n_x;
  float scale;
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t ml_rsrc(const void* base, uint32_t bytes) {
  const unsigned long long a = (unsigned long long)base;
  const unsigned long long u = ((unsigned long long)__builtin_amdgcn_readfirstlane((uint32_t)(a >> 32)) << 32) |
                               (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)a);
  return __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<void*>(u), (short)0,
                                           (int)__builtin_amdgcn_readfirstlane(bytes), 0x00020000);
}

__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// (request, split, head block) of task i in either order.
__device__ __forceinline__ void mla_task_of(const MlaParams& p, bool aware, int i, int& b, int& split, int& hb) {
  if (aware) {
    hb = i % p.hblocks;
    const int r = i / p.hblocks;
    split = r % p.n_splits;
    b = r / p.n_splits;
  } else {
    const int bs = p.B * p.n_splits;
    hb = i / bs;
    const int r = i - hb * bs;
    split = r % p.n_splits;
    b = r / p.n_splits;
  }
}

// The maximum over the four lanes l, l ^ 16, l ^ 32, l ^ 48: each row swap
// (v_permlane16_swap, v_permlane32_swap) of a value with itself leaves every
// lane the pair {x[l], x[l ^ 16]} (then ^ 32) in its two results; in the
// vector unit, with no LDS round trip.  A maximum is exact in any order.
__device__ __forceinline__ float ml_max4(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

// ---- the arithmetic of one 16-token block, shared by both forms ----------
// Scores S^T (16 tokens x 16 heads) = K . Q^T: lane (lr, lq) gets tokens
// 4 lq .. 4 lq + 3 of the block, head lr.
__device__ __forceinline__ f32x4 mla_scores(const bf16x8 (&kf)[MSTEPS], const bf16x8 (&qf)[MSTEPS]) {
  f32x4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int c = 0; c < MSTEPS; ++c) s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[c], qf[c], s, 0, 0, 0);
  return s;
}

// Online softmax of a block (tokens past t1 masked): updates the reference
// max and the sum, rescales the output when some head's block maximum exceeds
// its reference by more than kRescaleGap (the factor is exactly 1 elsewhere)
// and returns the probabilities, relative to the reference, as the B operand
// of P.V.  A reference below the true maximum leaves the result exact (the
// output, the sum and the max that the merge receives all use it); it only
// lets probabilities reach e^kRescaleGap, and saves the 128-multiply rescale
// on most blocks (with the exact maximum, a random sequence raised some head's
// maximum on about 60% of the blocks of a 1024-token split).
constexpr float kRescaleGap = 8.f;
__device__ __forceinline__ i16x4 mla_softmax(f32x4 s, int tok0, int t1, float scale, int lq, f32x4 (&o)[MV / 16],
                                             float& m_run, float& l_part) {
  float v[4];
  float bm = -INFINITY;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int tok = tok0 + 4 * lq + i;
    v[i] = tok < t1 ? s[i] * scale : -INFINITY;
    bm = fmaxf(bm, v[i]);
  }
  bm = ml_max4(bm);
  // bm is finite (every block has a token); the first block always raises
  const bool raise = bm > m_run + kRescaleGap;
  const float m_new = raise ? bm : m_run;
  const float alpha = raise ? __expf(m_run - m_new) : 1.f;
  m_run = m_new;
  float pr[4];
  float ps = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    pr[i] = __expf(v[i] - m_new);
    ps += pr[i];
  }
  l_part = l_part * alpha + ps;
  i16x4 pb;
#pragma unroll
  for (int i = 0; i < 4; ++i) pb[i] = __builtin_bit_cast(short, (__bf16)pr[i]);
  if (__ballot(raise)) {
#pragma unroll
    for (int j = 0; j < MV / 16; ++j) o[j] *= alpha;
  }
  return pb;
}

// O^T (512 values x 16 heads) += V^T . P^T from a row-major tile (token rows
// of `pitch` bytes, the latent values first).  The A operand
// V^T[16 j + lr][4 lq .. 4 lq + 3] comes from a transposing read: in each
// group of 16 lanes, result lane r takes element r % 4 of the 8 bytes that
// lanes 4 i + r / 4 address, i = 0 .. 3; lane (lr, lq) addresses token
// 4 lq + lr / 4, values 16 j + 4 (lr % 4) .. + 3.  In batches of 8, the next
// batch's reads in flight while a batch's MFMAs run (an empty asm that takes a
// whole batch keeps the compiler from placing each read next to its use).
__device__ __forceinline__ void mla_pv(const unsigned char* tile, uint32_t pitch, i16x4 pb, int lr, int lq,
                                       f32x4 (&o)[MV / 16]) {
  const uint32_t tr0 = (uint32_t)(4 * lq + (lr >> 2)) * pitch + 8u * (lr & 3);
  auto read_batch = [&](int jb, i16x4 (&a)[8]) {
#pragma unroll
    for (int u = 0; u < 8; ++u)
      a[u] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (__attribute__((address_space(3))) i16x4*)(tile + tr0 + 32u * (jb + u)));
  };
  i16x4 ab[2][8];
  read_batch(0, ab[0]);
#pragma unroll
  for (int jb = 0; jb < MV / 16; jb += 8) {
    i16x4 (&cur)[8] = ab[(jb / 8) & 1];
    asm volatile("" : "+v"(cur[0]), "+v"(cur[1]), "+v"(cur[2]), "+v"(cur[3]), "+v"(cur[4]), "+v"(cur[5]),
                 "+v"(cur[6]), "+v"(cur[7]));
    if (jb + 8 < MV / 16) read_batch(jb + 8, ab[((jb / 8) + 1) & 1]);
#pragma unroll
    for (int u = 0; u < 8; ++u) o[jb + u] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(cur[u], pb, o[jb + u], 0, 0, 0);
  }
}

// The workgroup form's block of 32 tokens, as two 16-token halves: s0 and
// s1 give lane (lr, lq) tokens 4 lq .. 4 lq + 3 and 16 + 4 lq .. 16 + 4 lq + 3
// of head lr.  The softmax step is that of mla_softmax over the 32 tokens;
// the probabilities come back as the B operand of a 32-deep product whose
// k index 8 lq + i stands for the first group's token 4 lq + i (i < 4) and
// the second group's token 16 + 4 lq + i - 4 (i >= 4).
// The probabilities and the statistics; `alpha` is the factor the output
// takes when the wave's ballot of `raise` is set (exactly 1 on other lanes).
__device__ __forceinline__ bf16x8 mla_softmax32_core(f32x4 s0, f32x4 s1, int tok0, int t1, float scale, int lq,
                                                     float& m_run, float& l_part, float& alpha, bool& raise) {
  float v[8];
  float bm = -INFINITY;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int tok = tok0 + (i < 4 ? 0 : 16) + 4 * lq + (i & 3);
    v[i] = tok < t1 ? (i < 4 ? s0[i] : s1[i - 4]) * scale : -INFINITY;
    bm = fmaxf(bm, v[i]);
  }
  bm = ml_max4(bm);
  // bm is finite (every block has a token); the first block always raises
  raise = bm > m_run + kRescaleGap;
  const float m_new = raise ? bm : m_run;
  alpha = raise ? __expf(m_run - m_new) : 1.f;
  m_run = m_new;
  float pr[8];
  float ps = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    pr[i] = __expf(v[i] - m_new);
    ps += pr[i];
  }
  l_part = l_part * alpha + ps;
  bf16x8 pb;
#pragma unroll
  for (int i = 0; i < 8; ++i) pb[i] = (__bf16)pr[i];
  return pb;
}

__device__ __forceinline__ bf16x8 mla_softmax32(f32x4 s0, f32x4 s1, int tok0, int t1, float scale, int lq,
                                                f32x4 (&o)[MV / 16], float& m_run, float& l_part) {
  float alpha;
  bool raise;
  const bf16x8 pb = mla_softmax32_core(s0, s1, tok0, t1, scale, lq, m_run, l_part, alpha, raise);
  if (__ballot(raise)) {
#pragma unroll
    for (int j = 0; j < MV / 16; ++j) o[j] *= alpha;
  }
  return pb;
}

// O^T += V^T . P^T over a 32-token block of the shared tile with
// v_mfma_f32_16x16x32_bf16: the A operand of lane (lr, lq) joins the
// transposing reads of the two 16-row halves (values 16 j + lr, tokens
// 4 lq .. 4 lq + 3 of each half), in the k order of mla_softmax32.  Batches of
// 8 products, the next batch's 16 reads in flight while a batch runs.
__device__ __forceinline__ void mla_pv32(const unsigned char* tile, bf16x8 pb, int lr, int lq, f32x4 (&o)[MV / 16]) {
  const uint32_t tr0 = (uint32_t)(4 * lq + (lr >> 2)) * K_ROW + 8u * (lr & 3);
  auto read_batch = [&](int jb, i16x4 (&a)[16]) {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      a[2 * u] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (__attribute__((address_space(3))) i16x4*)(tile + tr0 + 32u * (jb + u)));
      a[2 * u + 1] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (__attribute__((address_space(3))) i16x4*)(tile + tr0 + 16u * K_ROW + 32u * (jb + u)));
    }
  };
  i16x4 ab[2][16];
  read_batch(0, ab[0]);
#pragma unroll
  for (int jb = 0; jb < MV / 16; jb += 8) {
    i16x4 (&cur)[16] = ab[(jb / 8) & 1];
    asm volatile("" : "+v"(cur[0]), "+v"(cur[1]), "+v"(cur[2]), "+v"(cur[3]), "+v"(cur[4]), "+v"(cur[5]),
                 "+v"(cur[6]), "+v"(cur[7]), "+v"(cur[8]), "+v"(cur[9]), "+v"(cur[10]), "+v"(cur[11]),
                 "+v"(cur[12]), "+v"(cur[13]), "+v"(cur[14]), "+v"(cur[15]));
    if (jb + 8 < MV / 16) read_batch(jb + 8, ab[((jb / 8) + 1) & 1]);
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const bf16x8 a = __builtin_bit_cast(bf16x8, __builtin_shufflevector(cur[2 * u], cur[2 * u + 1], 0, 1, 2, 3,
                                                                          4, 5, 6, 7));
      o[jb + u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pb, o[jb + u], 0, 0, 0);
    }
  }
}

// The 16 query rows of head block hb (rows past H_q read as zero).
__device__ __forceinline__ void mla_load_q(const MlaParams& p, int b, int hb, int lr, int lq, bf16x8 (&qf)[MSTEPS]) {
  const int h0 = hb * 16;
  const __amdgpu_buffer_rsrc_t rq =
      ml_rsrc(p.q + ((size_t)b * p.Hq + h0) * MD, (uint32_t)min(16, p.Hq - h0) * MD * 2u);
#pragma unroll
  for (int c = 0; c < MSTEPS; ++c)
    qf[c] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(
                                           rq, (uint32_t)(lr * MD + 32 * c + 8 * lq) * 2u, 0, 0));
}

// A task's unnormalised output, max and sum; lane (lr, lq) holds
// O^T[16 j + 4 lq + i][head 16 hb + lr].
__device__ __forceinline__ void mla_store(const MlaParams& p, int b, int split, int hb, int lr, int lq,
                                          const f32x4 (&o)[MV / 16], float m_run, float l_part) {
  l_part += __shfl_xor(l_part, 16);  // the four token groups of a head's sum
  l_part += __shfl_xor(l_part, 32);
  const int h = hb * 16 + lr;
  if (h < p.Hq) {
    const size_t row = ((size_t)b * p.Hq + h) * p.n_splits + split;
    float* dst = p.part_o + row * MV + 4 * lq;
#pragma unroll
    for (int j = 0; j < MV / 16; ++j) *reinterpret_cast<f32x4*>(dst + 16 * j) = o[j];
    if (lq == 0) {
      p.part_ml[row * 2] = m_run;
      p.part_ml[row * 2 + 1] = l_part;
    }
  }
}

// ---- wave form: one (request, split, head block) per wave ---------------
__device__ void mla_task(const MlaParams& p, int b, int split, int hb, unsigned char* __restrict__ vt) {
  const int lane = threadIdx.x & 63;
  const int lr = lane & 15, lq = lane >> 4;
  const int t0 = split * p.split;
  const int t1 = min(p.S, t0 + p.split);
  const int nblk = (t1 - t0 + MT - 1) / MT;
  const __amdgpu_buffer_rsrc_t rk = ml_rsrc(p.kv + (size_t)b * p.S * MD, (uint32_t)p.S * MD * 2u);
  bf16x8 qf[MSTEPS];
  mla_load_q(p, b, hb, lr, lq, qf);
  f32x4 o[MV / 16];
#pragma unroll
  for (int j = 0; j < MV / 16; ++j) o[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_part = 0.f;

  // key fragments of a block (16 tokens): step c holds values 32 c .. 32 c + 31
  bf16x8 kf[MSTEPS];
  auto load_block = [&](int blk) {
    const int tok = t0 + blk * MT + lr;
    const uint32_t base = tok < t1 ? (uint32_t)(tok * MD + 8 * lq) * 2u : kMlOOB;
#pragma unroll
    for (int c = 0; c < MSTEPS; ++c)
      kf[c] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(rk, base, 64 * c, 0));
  };
  load_block(0);
  for (int blk = 0; blk < nblk; ++blk) {
    const f32x4 s = mla_scores(kf, qf);
    // the latent values of the block into the tile as they are (row: token,
    // 16 contiguous bytes per lane and step); this wave's reads of the
    // previous block are complete (its LDS accesses run in order)
#pragma unroll
    for (int c = 0; c < VSTEPS; ++c)
      *reinterpret_cast<v4u*>(vt + (uint32_t)lr * V_ROW + (uint32_t)(32 * c + 8 * lq) * 2u) =
          __builtin_bit_cast(v4u, kf[c]);
    // the next block's rows go out now (the fragments are consumed)
    if (blk + 1 < nblk) load_block(blk + 1);
    const i16x4 pb = mla_softmax(s, t0 + blk * MT, t1, p.scale, lq, o, m_run, l_part);
    wave_sync();  // the tile writes of every lane before any lane reads
    mla_pv(vt, V_ROW, pb, lr, lq, o);
    wave_sync();  // every lane's reads of the tile before the next block's writes
  }
  mla_store(p, b, split, hb, lr, lq, o, m_run, l_part);
}

// ---- workgroup form: one (request, split, group of 4 head blocks) per
// workgroup, wave w on head block 4 g + w.  Each 32-token block's rows are
// loaded once per workgroup into a shared LDS tile (two tiles, the next
// block's loads in flight in registers) and read by all four waves: the keys
// as score operands (the two 16-row halves as two independent MFMA chains),
// the values through the transposing read.  The softmax runs once per
// 32 tokens and P.V takes 32-deep products, so this form rounds differently
// from the wave form (16-token blocks); neither depends on the placement.
__device__ void mla_wg_task(const MlaParams& p, int b, int split, int hg, unsigned char* __restrict__ tiles) {
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int lr = lane & 15, lq = lane >> 4;
  const int t0 = split * p.split;
  const int t1 = min(p.S, t0 + p.split);
  const int nblk = (t1 - t0 + MT2 - 1) / MT2;
  const int hb = hg * MG + wave;
  const __amdgpu_buffer_rsrc_t rk = ml_rsrc(p.kv + (size_t)b * p.S * MD, (uint32_t)p.S * MD * 2u);
  bf16x8 qf[MSTEPS];
  mla_load_q(p, b, hb, lr, lq, qf);
  f32x4 o[MV / 16];
#pragma unroll
  for (int j = 0; j < MV / 16; ++j) o[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_part = 0.f;

  // a block is 32 rows of 72 chunks of 16 bytes; thread t carries chunks
  // t, t + 256, ... (tokens past the split read as zero)
  auto gload = [&](int blk, v4u (&r)[WG_CHUNKS]) {
#pragma unroll
    for (int e = 0; e < WG_CHUNKS; ++e) {
      const int c = threadIdx.x + 64 * MG * e;
      const int tok = t0 + blk * MT2 + c / (MD / 8);
      const bool in = c < MT2 * (MD / 8) && tok < t1;
      r[e] = __builtin_amdgcn_raw_buffer_load_b128(
          rk, in ? (uint32_t)(tok * MD + (c % (MD / 8)) * 8) * 2u : kMlOOB, 0, 0);
    }
  };
  auto swrite = [&](int buf, const v4u (&r)[WG_CHUNKS]) {
#pragma unroll
    for (int e = 0; e < WG_CHUNKS; ++e) {
      const int c = threadIdx.x + 64 * MG * e;
      if (c < MT2 * (MD / 8))
        *reinterpret_cast<v4u*>(tiles + buf * K_BYTES + (uint32_t)(c / (MD / 8)) * K_ROW + (c % (MD / 8)) * 16u) =
            r[e];
    }
  };
  // at the top of iteration blk, tile blk % 2 holds block blk and the
  // staging registers block blk + 1
  v4u ra[WG_CHUNKS];
  gload(0, ra);
  swrite(0, ra);
  if (nblk > 1) gload(1, ra);
  __syncthreads();
  for (int blk = 0; blk < nblk; ++blk) {
    const unsigned char* tile = tiles + (blk & 1) * K_BYTES;
    // scores of the two halves: key fragments of KB steps of both halves
    // per batch, a batch's reads all issued (the empty asm) before the
    // previous batch's MFMAs
    const unsigned char* krow = tile + (uint32_t)lr * K_ROW + 16u * lq;
    f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
    bf16x8 kf[2][2 * KB];
    auto kread = [&](int c0, bf16x8 (&k)[2 * KB]) {
#pragma unroll
      for (int c = 0; c < KB; ++c) {
        k[2 * c] = *reinterpret_cast<const bf16x8*>(krow + 64u * (c0 + c));
        k[2 * c + 1] = *reinterpret_cast<const bf16x8*>(krow + 16u * K_ROW + 64u * (c0 + c));
      }
    };
    kread(0, kf[0]);
#pragma unroll
    for (int c0 = 0; c0 < MSTEPS; c0 += KB) {
      bf16x8 (&k)[2 * KB] = kf[(c0 / KB) & 1];
      asm volatile("" : "+v"(k[0]), "+v"(k[1]), "+v"(k[2]), "+v"(k[3]), "+v"(k[4]), "+v"(k[5]), "+v"(k[6]),
                   "+v"(k[7]), "+v"(k[8]), "+v"(k[9]), "+v"(k[10]), "+v"(k[11]));
      if (c0 + KB < MSTEPS) kread(c0 + KB, kf[((c0 / KB) + 1) & 1]);
#pragma unroll
      for (int c = 0; c < KB; ++c) {
        s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k[2 * c], qf[c0 + c], s0, 0, 0, 0);
        s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k[2 * c + 1], qf[c0 + c], s1, 0, 0, 0);
      }
    }
    const bf16x8 pb = mla_softmax32(s0, s1, t0 + blk * MT2, t1, p.scale, lq, o, m_run, l_part);
    mla_pv32(tile, pb, lr, lq, o);
    // block blk + 1 into the other tile (its last readers, block blk - 1,
    // finished before the previous barrier), then block blk + 2's loads
    if (blk + 1 < nblk) {
      swrite((blk + 1) & 1, ra);
      if (blk + 2 < nblk) gload(blk + 2, ra);
    }
    __syncthreads();
  }
  mla_store(p, b, split, hb, lr, lq, o, m_run, l_part);
}

// ---- 128-head form: one (request, split, group of 8 head blocks) per
// workgroup, wave w on head blocks 8 g + 2 w and 8 g + 2 w + 1.  Every key
// fragment read from the tile feeds both head blocks' score chains and every
// joined value fragment both P.V products, half the LDS reads per head of the
// 64-head form.  The 256 output accumulators stay in AGPRs (inline-asm
// MFMAs, with the wait states around their VALU accesses padded explicitly);
// the rows go from memory straight into three LDS tiles (buffer_load ... lds,
// two blocks ahead), so no registers stage them.  Per head the operations and
// their order are those of the 64-head form, so the bits are the same.

// buffer descriptor words (uniform) for the asm loads
__device__ __forceinline__ i32x4 ml_rsrc_words(const void* base, uint32_t bytes) {
  const unsigned long long a = (unsigned long long)base;
  return i32x4{(int)__builtin_amdgcn_readfirstlane((uint32_t)a), (int)__builtin_amdgcn_readfirstlane((uint32_t)(a >> 32)),
               (int)__builtin_amdgcn_readfirstlane(bytes), 0x00020000};
}

// 16 bytes per lane from memory into LDS: lane L's bytes land at lds + 16 L.
// The compiler does not see these loads; their completion is waited for
// explicitly (ml_vmwait) before the barrier that publishes the tile.
__device__ __forceinline__ void ml_dma16(uint32_t lds, i32x4 rs, uint32_t voff) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds" : : "s"(lds), "v"(voff), "s"(rs)
               : "memory", "m0");
}
template <int N>
__device__ __forceinline__ void ml_vmwait() {
  asm volatile("s_waitcnt vmcnt(%0)" : : "i"(N) : "memory");
}

// acc += a . b with the accumulator in AGPRs
__device__ __forceinline__ void ml_mfma_acc(f32x4& acc, const bf16x8& a, const bf16x8& b) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
}
// wait states between the asm MFMAs and vector accesses of their accumulators
// (covers the longest dependency of the 16x16x32 shape)
__device__ __forceinline__ void ml_mfma_fence() {
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
}
// the accumulators materialised in AGPRs at this point of the program
__device__ __forceinline__ void ml_pin(f32x4 (&o)[2][MV / 16]) {
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int j = 0; j < MV / 16; ++j) asm volatile("" : "+a"(o[h][j]));
}

__device__ void mla_wg2_task(const MlaParams& p, int b, int split, int hg, unsigned char* __restrict__ tiles) {
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int lr = lane & 15, lq = lane >> 4;
  const int t0 = split * p.split;
  const int t1 = min(p.S, t0 + p.split);
  const int nblk = (t1 - t0 + MT2 - 1) / MT2;
  const int hb0 = hg * MG2 + 2 * wave;
  // the request's rows; a split is a multiple of 32 tokens, so only the
  // request's last block is partial and its rows past S_k read as zero
  const i32x4 rk = ml_rsrc_words(p.kv + (size_t)b * p.S * MD, (uint32_t)p.S * MD * 2u);
  bf16x8 qf[2][MSTEPS];
  mla_load_q(p, b, hb0, lr, lq, qf[0]);
  mla_load_q(p, b, hb0 + 1, lr, lq, qf[1]);
  f32x4 o[2][MV / 16];
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int j = 0; j < MV / 16; ++j) o[h][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  ml_pin(o);
  ml_mfma_fence();
  float m_run[2] = {-INFINITY, -INFINITY}, l_part[2] = {0.f, 0.f};

  // load e of this wave fills slots 64 (w + 4 e) .. + 63 of the tile; slot s
  // is row s / 74, 16-byte chunk s % 74 (chunks 72, 73 and slots past row 31
  // are padding and read as zero)
  uint32_t rel[T2_DMA];
#pragma unroll
  for (int e = 0; e < T2_DMA; ++e) {
    const int sl = 64 * (wave + 4 * e) + lane;
    const int row = sl / T2_ROWSLOTS, ch = sl - row * T2_ROWSLOTS;
    rel[e] = (row < MT2 && ch < MD / 8) ? (uint32_t)(row * MD + ch * 8) * 2u : kMlOOB;
  }
  const uint32_t lds_base = (uint32_t)(size_t)tiles;  // a shared address's low word is its LDS address
  const uint32_t lds0 = lds_base + 1024u * (uint32_t)wave;
  auto dma = [&](int blk) {
    const uint32_t base = (uint32_t)(t0 + blk * MT2) * (uint32_t)(MD * 2);
    const uint32_t dst = lds0 + (uint32_t)(blk % T2_TILES) * (uint32_t)T2_BYTES;
#pragma unroll
    for (int e = 0; e < T2_DMA; ++e) ml_dma16(dst + 4096u * e, rk, rel[e] == kMlOOB ? kMlOOB : base + rel[e]);
  };
  dma(0);
  if (nblk > 1) {
    dma(1);
    ml_vmwait<T2_DMA>();
  } else {
    ml_vmwait<0>();
  }
  __syncthreads();
  const uint32_t tr0 = (uint32_t)(4 * lq + (lr >> 2)) * K_ROW + 8u * (lr & 3);
  for (int blk = 0; blk < nblk; ++blk) {
    // block blk + 2 into the tile block blk - 1 left (every wave passed the
    // barrier after reading it)
    if (blk + 2 < nblk) dma(blk + 2);
    // the tile as an LDS address, so that the constant parts of the fragment
    // addresses fold into the instructions' offsets
    lds_u8* tile = reinterpret_cast<lds_u8*>((size_t)(lds_base + (uint32_t)(blk % T2_TILES) * (uint32_t)T2_BYTES));
    // scores: s[h][half] for the two head blocks and the two 16-row halves;
    // key fragments in batches of KB2 steps of both halves, three batches
    // deep (a batch's reads issued two batches before its MFMAs)
    lds_u8* krow = tile + (uint32_t)lr * K_ROW + 16u * lq;
    f32x4 sc[2][2];
#pragma unroll
    for (int h = 0; h < 2; ++h) sc[h][0] = sc[h][1] = f32x4{0.f, 0.f, 0.f, 0.f};
    bf16x8 kf[3][2 * KB2];
    auto kread = [&](int c0, bf16x8 (&k)[2 * KB2]) {
#pragma unroll
      for (int c = 0; c < KB2; ++c) {
        k[2 * c] = *reinterpret_cast<lds_bf16x8*>(krow + 64u * (c0 + c));
        k[2 * c + 1] = *reinterpret_cast<lds_bf16x8*>(krow + 16u * K_ROW + 64u * (c0 + c));
      }
    };
    kread(0, kf[0]);
    kread(KB2, kf[1]);
#pragma unroll
    for (int c0 = 0; c0 < MSTEPS; c0 += KB2) {
      bf16x8 (&k)[2 * KB2] = kf[(c0 / KB2) % 3];
      static_assert(KB2 == 2, "the empty asm below names the batch's four fragments");
      asm volatile("" : "+v"(k[0]), "+v"(k[1]), "+v"(k[2]), "+v"(k[3]));
      if (c0 + 2 * KB2 < MSTEPS) kread(c0 + 2 * KB2, kf[((c0 / KB2) + 2) % 3]);
#pragma unroll
      for (int c = 0; c < KB2; ++c)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          sc[h][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k[2 * c], qf[h][c0 + c], sc[h][0], 0, 0, 0);
          sc[h][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k[2 * c + 1], qf[h][c0 + c], sc[h][1], 0, 0, 0);
        }
    }
    bf16x8 pb[2];
    float alpha[2];
    bool raise[2];
#pragma unroll
    for (int h = 0; h < 2; ++h)
      pb[h] = mla_softmax32_core(sc[h][0], sc[h][1], t0 + blk * MT2, t1, p.scale, lq, m_run[h], l_part[h], alpha[h],
                                 raise[h]);
    if (__ballot(raise[0] || raise[1])) {
      ml_mfma_fence();
      // one accumulator at a time through 4 VGPRs: each read is ordered
      // after the previous write-back by the empty asms
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int j = 0; j < MV / 16; ++j) {
          asm volatile("" : "+a"(o[h][j]));
          f32x4 t = o[h][j];
          asm volatile("" : "+v"(t));
          t *= alpha[h];
          o[h][j] = t;
          asm volatile("" : "+a"(o[h][j]));
        }
    }
    ml_mfma_fence();
    // P.V: batches of 4 value tiles (8 transposing reads), each joined
    // fragment used by both head blocks; the next two batches' reads in
    // flight while a batch's 8 MFMAs run
    auto tread = [&](int jb, i16x4 (&a)[8]) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        a[2 * u] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(reinterpret_cast<lds_i16x4*>(tile + tr0 + 32u * (jb + u)));
        a[2 * u + 1] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            reinterpret_cast<lds_i16x4*>(tile + tr0 + 16u * K_ROW + 32u * (jb + u)));
      }
    };
    i16x4 ab[3][8];
    tread(0, ab[0]);
    tread(4, ab[1]);
#pragma unroll
    for (int jb = 0; jb < MV / 16; jb += 4) {
      i16x4 (&cur)[8] = ab[(jb / 4) % 3];
      asm volatile("" : "+v"(cur[0]), "+v"(cur[1]), "+v"(cur[2]), "+v"(cur[3]), "+v"(cur[4]), "+v"(cur[5]),
                   "+v"(cur[6]), "+v"(cur[7]));
      if (jb + 8 < MV / 16) tread(jb + 8, ab[((jb / 4) + 2) % 3]);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const bf16x8 a = __builtin_bit_cast(bf16x8, __builtin_shufflevector(cur[2 * u], cur[2 * u + 1], 0, 1, 2, 3,
                                                                            4, 5, 6, 7));
        ml_mfma_acc(o[0][jb + u], a, pb[0]);
        ml_mfma_acc(o[1][jb + u], a, pb[1]);
      }
    }
    // block blk + 1 has landed (block blk + 2's loads may still be in flight)
    if (blk + 2 < nblk)
      ml_vmwait<T2_DMA>();
    else
      ml_vmwait<0>();
    __syncthreads();
  }
  ml_mfma_fence();
  mla_store(p, b, split, hb0, lr, lq, o[0], m_run[0], l_part[0]);
  mla_store(p, b, split, hb0 + 1, lr, lq, o[1], m_run[1], l_part[1]);
}

__global__ void __launch_bounds__(64 * MW) mla_decode_split(MlaParams p) {
  __shared__ __attribute__((aligned(16))) unsigned char vt_all[MW][V_BYTES];
  __shared__ int box[2];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const bool aware = p.quota_off != nullptr;
  int own = 0;
  if (aware) {
    uint32_t xr;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xr));
    own = (int)(xr & 0xFu);
    if (own >= p.n_x || !((p.allow >> own) & 1u)) return;  // an XCD outside the set
  }
  // Oblivious: one group of 4 tasks, workgroup i's.  Aware: claims, own share
  // first, then the others in turn; wave 0 reads every counter in one round
  // trip and only adds to shares that still have groups; the loop ends when
  // each counter has passed its share.  One call site of the task body.
  for (int round = 0;; ++round) {
    int base, end;
    if (!aware) {
      if (round > 0) break;
      base = blockIdx.x * MW;
      end = p.tasks;
    } else {
      if (wave == 0) {
        int rem = 0, y = 0, b0 = 0, b1 = 0;
        if (lane < p.n_x) {
          y = (own + lane) % p.n_x;
          b0 = p.quota_off[y];
          b1 = p.quota_off[y + 1];
          const int taken =
              __hip_atomic_load(&p.claim[y * kMlClaimStride], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          rem = (b1 - b0 + MW - 1) / MW - taken;
        }
        unsigned long long open = __ballot(lane < p.n_x && rem > 0);
        int got_base = -1, got_end = 0;
        while (open && got_base < 0) {
          const int l = __builtin_ctzll(open);
          open &= open - 1;
          int got = -1;
          if (lane == l) {
            const int g = atomicAdd(&p.claim[y * kMlClaimStride], 1);
            if (b0 + g * MW < b1) got = b0 + g * MW;
          }
          got = __shfl(got, l);
          if (got >= 0) {
            got_base = got;
            got_end = __shfl(b1, l);
          }
        }
        if (lane == 0) {
          box[0] = got_base;
          box[1] = got_end;
        }
      }
      __syncthreads();
      base = box[0];
      end = box[1];
      __syncthreads();
      if (base < 0) break;
    }
    if (base + wave < end) {
      int b, split, hb;
      mla_task_of(p, aware, base + wave, b, split, hb);
      mla_task(p, b, split, hb, vt_all[wave]);
    }
  }
}

// Workgroup form: tasks (request, split, group of 4 head blocks), numbered
// with the group fastest (aware) or group major (oblivious).  Oblivious: task
// i on workgroup i.  Aware: claims of one task, own share first, then the
// others, as in the wave form.
template <int FORM>
__global__ void __launch_bounds__(256) mla_decode_split_wg(MlaParams p) {
  __shared__ __attribute__((aligned(1024))) unsigned char tiles[FORM == 2 ? T2_TILES * T2_BYTES : 2 * K_BYTES];
  __shared__ int box[1];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const bool aware = p.quota_off != nullptr;
  const int groups = p.hblocks / (FORM == 2 ? MG2 : MG);
  int own = 0;
  if (aware) {
    uint32_t xr;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xr));
    own = (int)(xr & 0xFu);
    if (own >= p.n_x || !((p.allow >> own) & 1u)) return;  // an XCD outside the set
  }
  for (int round = 0;; ++round) {
    int task;
    if (!aware) {
      if (round > 0 || (int)blockIdx.x >= p.tasks) break;
      task = blockIdx.x;
    } else {
      if (wave == 0) {
        int rem = 0, y = 0, b0 = 0, b1 = 0;
        if (lane < p.n_x) {
          y = (own + lane) % p.n_x;
          b0 = p.quota_off[y];
          b1 = p.quota_off[y + 1];
          const int taken =
              __hip_atomic_load(&p.claim[y * kMlClaimStride], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          rem = (b1 - b0) - taken;
        }
        unsigned long long open = __ballot(lane < p.n_x && rem > 0);
        int got_task = -1;
        while (open && got_task < 0) {
          const int l = __builtin_ctzll(open);
          open &= open - 1;
          int got = -1;
          if (lane == l) {
            const int g = atomicAdd(&p.claim[y * kMlClaimStride], 1);
            if (b0 + g < b1) got = b0 + g;
          }
          got_task = __shfl(got, l);
        }
        if (lane == 0) box[0] = got_task;
      }
      __syncthreads();
      task = box[0];
      __syncthreads();
      if (task < 0) break;
    }
    int b, split, hg;
    if (aware) {
      hg = task % groups;
      const int r = task / groups;
      split = r % p.n_splits;
      b = r / p.n_splits;
    } else {
      const int bs = p.B * p.n_splits;
      hg = task / bs;
      const int r = task - hg * bs;
      split = r % p.n_splits;
      b = r / p.n_splits;
    }
    if constexpr (FORM == 2)
      mla_wg2_task(p, b, split, hg, tiles);
    else
      mla_wg_task(p, b, split, hg, tiles);
  }
}

// Merge of the splits of every (request, head) row (split_merge.h); also
// clears the aware form's claim counters (the split launch is complete).
template <int CH>
__global__ void __launch_bounds__(64 * kMergeWaves) mla_decode_merge(const float* __restrict__ part_o,
                                                                     const float* __restrict__ part_ml, int rows,
                                                                     int n_splits, int wpr, uint16_t* __restrict__ o,
                                                                     float* __restrict__ lse, int* claim,
                                                                     int n_claim) {
  if (claim && blockIdx.x == 0 && blockIdx.y == 0 && (int)threadIdx.x < n_claim) claim[threadIdx.x * kMlClaimStride] = 0;
  merge_split_rows<MV, CH>(part_o, part_ml, rows, n_splits, wpr, o, lse);
}

}  // namespace

int launch_mla_decode(const MlaLaunch& a, hipStream_t s) {
  MlaParams p;
  p.q = static_cast<const uint16_t*>(a.q);
  p.kv = static_cast<const uint16_t*>(a.kv);
  p.part_o = a.part_o;
  p.part_ml = a.part_ml;
  p.quota_off = a.d_quota_off;
  p.claim = a.d_claim;
  p.allow = a.allow;
  p.B = a.B;
  p.Hq = a.Hq;
  p.S = a.S;
  p.split = a.split;
  p.n_splits = a.n_splits;
  p.hblocks = (a.Hq + 15) / 16;
  if (a.form < 0 || a.form > 2) return fail(ASYM_EINVAL, "mla: unknown kernel form");
  const int per_task = mla_form_head_blocks(a.form);
  if (p.hblocks % per_task) return fail(ASYM_EINVAL, "mla: the head count does not suit the kernel form");
  p.tasks = a.B * a.n_splits * (p.hblocks / per_task);
  p.n_x = a.n_x;
  p.scale = a.scale;
  if (a.d_quota_off && (!a.d_claim || a.n_x > 64)) return fail(ASYM_EINVAL, "mla: aware launch without claim counters");
  if (a.grid < 1) return fail(ASYM_EINVAL, "mla: empty grid");
  if (a.form == 2)
    hipLaunchKernelGGL(mla_decode_split_wg<2>, dim3((unsigned)a.grid), dim3(256), 0, s, p);
  else if (a.form == 1)
    hipLaunchKernelGGL(mla_decode_split_wg<1>, dim3((unsigned)a.grid), dim3(256), 0, s, p);
  else
    hipLaunchKernelGGL(mla_decode_split, dim3((unsigned)a.grid), dim3(64 * MW), 0, s, p);
  ASYM_HIP(hipGetLastError());
  const int rows = a.B * a.Hq;
  const int wpr = merge_waves_per_row(a.n_splits), rows_per_wg = kMergeWaves / wpr;
  const int groups = (rows + rows_per_wg - 1) / rows_per_wg;
  const int ch = merge_column_chunks(groups, MV / 64);
  auto merge = ch == 8 ? mla_decode_merge<8> : ch == 4 ? mla_decode_merge<4> : ch == 2 ? mla_decode_merge<2>
                                                                                      : mla_decode_merge<1>;
  hipLaunchKernelGGL(merge, dim3((unsigned)groups, (unsigned)ch), dim3(64 * kMergeWaves), 0, s, a.part_o, a.part_ml,
                     rows, a.n_splits, wpr, static_cast<uint16_t*>(a.o), a.lse, a.d_quota_off ? a.d_claim : nullptr,
                     a.n_x);
  ASYM_HIP(hipGetLastError());
  return ASYM_OK;
}

int mla_tasks_per_workgroup() { return MW; }

int mla_form_head_blocks(int form) { return form == 2 ? MG2 : form == 1 ? MG : 1; }

}  // namespace asym
