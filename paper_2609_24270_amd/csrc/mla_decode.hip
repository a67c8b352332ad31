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
//     tokens, one head) are already the B operand of that product, and V^T
//     is written to a per-wave LDS tile from the key fragments already loaded
//     (the latent part of the row is the value), so the rows are read from
//     memory once; the tile's rows are padded to 40 bytes so that the four
//     lane groups of a write land in different banks;
//   * 16-token blocks; the next block's rows go out as soon as a block's
//     fragments are consumed (scores computed, values written), and the
//     output is rescaled only when a head's running maximum rises (a factor
//     of exactly 1 is skipped, so the result is the same).
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
constexpr int VT_ROW = 40;         // bytes of one V^T row: 16 tokens, padded
constexpr int VT_BYTES = MV * VT_ROW;  // 20 KiB per wave
constexpr uint32_t kMlOOB = 0x80000000u;
constexpr int kMlClaimStride = 64;  // ints between claim counters (256-byte lines)

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned v4u __attribute__((ext_vector_type(4)));

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

__device__ void mla_task(const MlaParams& p, int b, int split, int hb, unsigned char* __restrict__ vt) {
  const int lane = threadIdx.x & 63;
  const int lr = lane & 15, lq = lane >> 4;
  const int t0 = split * p.split;
  const int t1 = min(p.S, t0 + p.split);
  const int nblk = (t1 - t0 + MT - 1) / MT;

  // the 16 query rows (rows past H_q are outside the resource and read as zero)
  const int h0 = hb * 16;
  const __amdgpu_buffer_rsrc_t rq =
      ml_rsrc(p.q + ((size_t)b * p.Hq + h0) * MD, (uint32_t)min(16, p.Hq - h0) * MD * 2u);
  const __amdgpu_buffer_rsrc_t rk = ml_rsrc(p.kv + (size_t)b * p.S * MD, (uint32_t)p.S * MD * 2u);
  bf16x8 qf[MSTEPS];
#pragma unroll
  for (int c = 0; c < MSTEPS; ++c)
    qf[c] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(
                                           rq, (uint32_t)(lr * MD + 32 * c + 8 * lq) * 2u, 0, 0));

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
    // scores: lane (lr, lq) gets tokens 4 lq .. 4 lq + 3 of the block, head h0 + lr
    f32x4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < MSTEPS; ++c) s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[c], qf[c], s, 0, 0, 0);
    // the latent values of the block into V^T (row: value index, column:
    // token); this wave's reads of the previous block are complete (its LDS
    // accesses run in order)
#pragma unroll
    for (int c = 0; c < VSTEPS; ++c) {
      const v4u w = __builtin_bit_cast(v4u, kf[c]);
      const uint32_t at = (uint32_t)(32 * c + 8 * lq) * VT_ROW + 2u * lr;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        *reinterpret_cast<uint16_t*>(vt + at + (2 * e) * VT_ROW) = (uint16_t)(w[e] & 0xFFFFu);
        *reinterpret_cast<uint16_t*>(vt + at + (2 * e + 1) * VT_ROW) = (uint16_t)(w[e] >> 16);
      }
    }
    // the next block's rows go out now (the fragments are consumed)
    if (blk + 1 < nblk) load_block(blk + 1);
    // mask tokens past the split, scale, block max per head
    float v[4];
    float bm = -INFINITY;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int tok = t0 + blk * MT + 4 * lq + i;
      v[i] = tok < t1 ? s[i] * p.scale : -INFINITY;
      bm = fmaxf(bm, v[i]);
    }
    bm = fmaxf(bm, __shfl_xor(bm, 16));
    bm = fmaxf(bm, __shfl_xor(bm, 32));
    const float m_new = fmaxf(m_run, bm);  // finite: every block has a token
    const float alpha = __expf(m_run - m_new);
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
    // rescale only where some head's maximum rose (alpha is exactly 1 elsewhere)
    if (__ballot(alpha != 1.f)) {
#pragma unroll
      for (int j = 0; j < MV / 16; ++j) o[j] *= alpha;
    }
    wave_sync();  // the V^T writes of every lane before any lane reads
#pragma unroll
    for (int j = 0; j < MV / 16; ++j) {
      const i16x4 a = *reinterpret_cast<const i16x4*>(vt + (uint32_t)(16 * j + lr) * VT_ROW + 8u * lq);
      o[j] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, pb, o[j], 0, 0, 0);
    }
    wave_sync();  // every lane's reads of the tile before the next block's writes
  }
  // the four token groups of a head's sum
  l_part += __shfl_xor(l_part, 16);
  l_part += __shfl_xor(l_part, 32);
  // lane (lr, lq) holds O^T[16 j + 4 lq + i][head h0 + lr]
  const int h = h0 + lr;
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

__global__ void __launch_bounds__(64 * MW) mla_decode_split(MlaParams p) {
  __shared__ __attribute__((aligned(16))) unsigned char vt_all[MW][VT_BYTES];
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

// Merge of the splits of every (request, head) row (split_merge.h); also
// clears the aware form's claim counters (the split launch is complete).
__global__ void __launch_bounds__(64 * kMergeWaves) mla_decode_merge(const float* __restrict__ part_o,
                                                                     const float* __restrict__ part_ml, int rows,
                                                                     int n_splits, int wpr, uint16_t* __restrict__ o,
                                                                     float* __restrict__ lse, int* claim,
                                                                     int n_claim) {
  if (claim && blockIdx.x == 0 && (int)threadIdx.x < n_claim) claim[threadIdx.x * kMlClaimStride] = 0;
  merge_split_rows<MV>(part_o, part_ml, rows, n_splits, wpr, o, lse);
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
  p.tasks = a.B * a.n_splits * p.hblocks;
  p.n_x = a.n_x;
  p.scale = a.scale;
  if (a.d_quota_off && (!a.d_claim || a.n_x > 64)) return fail(ASYM_EINVAL, "mla: aware launch without claim counters");
  if (a.grid < 1) return fail(ASYM_EINVAL, "mla: empty grid");
  hipLaunchKernelGGL(mla_decode_split, dim3((unsigned)a.grid), dim3(64 * MW), 0, s, p);
  ASYM_HIP(hipGetLastError());
  const int rows = a.B * a.Hq;
  const int wpr = merge_waves_per_row(a.n_splits), rows_per_wg = kMergeWaves / wpr;
  hipLaunchKernelGGL(mla_decode_merge, dim3((unsigned)((rows + rows_per_wg - 1) / rows_per_wg)),
                     dim3(64 * kMergeWaves), 0, s, a.part_o, a.part_ml, rows, a.n_splits, wpr,
                     static_cast<uint16_t*>(a.o), a.lse, a.d_quota_off ? a.d_claim : nullptr, a.n_x);
  ASYM_HIP(hipGetLastError());
  return ASYM_OK;
}

int mla_tasks_per_workgroup() { return MW; }

}  // namespace asym
