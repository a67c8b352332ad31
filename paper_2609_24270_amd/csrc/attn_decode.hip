// Decode attention with grouped key/value heads (the attention workloads of
// Section 7.1, decode case: one query token per request; Appendix F gives the
// head dimension 128 and 32 or 8 key/value heads).
//
//   O[b, h] = softmax_t(scale * <q[b, h], K[b, g, t]>) . V[b, g, :],  g = h / G
//
// Work is split along the key/value sequence (flash-decoding): a task is one
// (request, key/value head, sequence split) and serves the G query heads that
// read that head, so every K and V byte is read once.  One wave runs one task:
//   * scores of 16 tokens x 16 query-head rows come from four
//     v_mfma_f32_16x16x32_bf16, K fragments loaded straight from HBM into
//     operand registers (a lane's 8 bf16 are 16 contiguous bytes of one key);
//   * an online softmax per head keeps the running max and sum;
//   * P.V runs on the vector ALU: a lane owns 8 of the 128 dimensions and a
//     quarter of the block's tokens, value rows are 16-byte loads, and the
//     probabilities reach it through a per-wave LDS tile (V's layout puts the
//     token index across rows, which an MFMA operand would need transposed);
//   * the next block's K and V are in flight while a block is computed.
// Each task writes its unnormalised output, max and sum (fp32); a second
// kernel merges the splits of each (request, head) in an order fixed by the
// split count (several waves per row when there are many splits), so the
// result is the same for every assignment of tasks to workgroups.
//
// Assignment.  A task's bytes are read by exactly one wave, so there is no
// cache reuse for a placement to exploit; what the topology decides is how
// many tasks each XCD gets.  Oblivious: tasks 4i .. 4i+3 go to workgroup i;
// the hardware deals workgroups to XCDs round-robin, so every XCD gets the
// same share whatever its CU count.  Aware: each XCD's share of the task list
// is proportional to its CU count in the stream's CU set; a workgroup reads
// the XCD it runs on (XCC_ID) and claims groups of 4 tasks of that XCD's share
// from a counter, then of the other shares, until none are left (which XCD a
// block index is dealt to is not fixed: the starting XCD differs between
// streams, so claims, not block indices, decide).
//
// Paged keys and values (the placed form, Appendix E's memory remapping).
// The caller's K and V live in pools of 8 KiB pages (32 tokens of one head),
// and an int32 table per pool gives the pool page of every (request, head,
// 32-token page).  With the aware mapping each task's share, and so the XCD
// that reads it, is known before launch; the table lets the caller put a
// task's pages in memory homed on that XCD's die.  A task loads its split's
// page numbers once (one per lane) and reads each block's page with a lane
// read; a 16-token block never crosses a page.  The pools are read through
// buffer descriptors sized to them, so a table entry past the pool reads
// zeros or other pool bytes, never memory outside it.
#include <hip/hip_runtime.h>

#include "internal.h"
#include "split_merge.h"

namespace asym {
namespace {

constexpr int AD = 128;            // head dimension
constexpr int AT_WAVES = 4;        // tasks per workgroup, one per wave
constexpr uint32_t kAtOOB = 0x80000000u;
constexpr int kClaimStride = 64;   // ints between claim counters: one 256-byte line each

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned v4u __attribute__((ext_vector_type(4)));

struct AttnParams {
  const uint16_t* q;   // [B][Hq][128]
  const uint16_t* k;   // [B][Hkv][S][128]
  const uint16_t* v;   // [B][Hkv][S][128]
  float* part_o;       // [B][Hq][n_splits][128]
  float* part_ml;      // [B][Hq][n_splits][2]: max, sum
  const int* quota_off;  // aware: [n_x + 1] start of each XCD's share (tasks), null = oblivious
  int* claim;            // aware: groups of 4 claimed from share y at claim[y * kClaimStride] (zero at launch)
  uint32_t allow;        // aware: XCDs whose workgroups may work (the others leave)
  int B, Hq, Hkv, S, split, n_splits, tasks, n_x;
  float scale;
  int pages_per_head;    // paged form: ceil(S / 32)
  const int* k_page;     // paged form: pool page of (request, head, page) [B][Hkv][pages_per_head]
  const int* v_page;
  uint32_t pool_bytes;   // each pool's size (at most 2^31, so the out-of-range offset reads zero)
};

constexpr int kPageTokens = 32;  // 8 KiB of one head's keys (or values)

__device__ __forceinline__ __amdgpu_buffer_rsrc_t at_rsrc(const void* base, uint32_t bytes) {
  const unsigned long long a = (unsigned long long)base;
  const unsigned long long u = ((unsigned long long)__builtin_amdgcn_readfirstlane((uint32_t)(a >> 32)) << 32) |
                               (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)a);
  return __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<void*>(u), (short)0,
                                           (int)__builtin_amdgcn_readfirstlane(bytes), 0x00020000);
}

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// One task on one wave.  G: query heads per key/value head (1 .. 16);
// PAGED: K and V through the page tables.
template <int G, bool PAGED>
__device__ void attn_task(const AttnParams& p, int task, float* __restrict__ sp) {
  const int lane = threadIdx.x & 63;
  const int split = task % p.n_splits;
  const int bh = task / p.n_splits;          // b * Hkv + kv head
  const int b = bh / p.Hkv, hk = bh - b * p.Hkv;
  const int t0 = split * p.split;
  const int t1 = min(p.S, t0 + p.split);
  const int nblk = (t1 - t0 + 15) >> 4;

  // q rows of the G heads; rows past G read as zero
  const __amdgpu_buffer_rsrc_t rq = at_rsrc(p.q + ((size_t)b * p.Hq + (size_t)hk * G) * AD, G * AD * 2u);
  const __amdgpu_buffer_rsrc_t rk =
      PAGED ? at_rsrc(p.k, p.pool_bytes) : at_rsrc(p.k + (size_t)bh * p.S * AD, (uint32_t)p.S * AD * 2u);
  const __amdgpu_buffer_rsrc_t rv =
      PAGED ? at_rsrc(p.v, p.pool_bytes) : at_rsrc(p.v + (size_t)bh * p.S * AD, (uint32_t)p.S * AD * 2u);
  const int lr = lane & 15, lq = lane >> 4;
  // paged: lane j holds the pool pages of the split's j-th page (at most 64)
  const int p0 = t0 / kPageTokens;
  int kpg = 0, vpg = 0;
  if constexpr (PAGED) {
    const int npg = (t1 - 1) / kPageTokens - p0 + 1;
    if (lane < npg) {
      const size_t e = (size_t)bh * p.pages_per_head + p0 + lane;
      kpg = p.k_page[e];
      vpg = p.v_page[e];
    }
  }
  // byte offset of block blk's first row in its buffer
  auto blk_off = [&](int blk, int pg) -> uint32_t {
    const int bt = t0 + blk * 16;
    if constexpr (PAGED)
      return (uint32_t)__builtin_amdgcn_readlane(pg, bt / kPageTokens - p0) * (kPageTokens * AD * 2u) +
             (uint32_t)(bt % kPageTokens) * (AD * 2u);
    return (uint32_t)bt * (AD * 2u);
  };
  bf16x8 qf[4];
#pragma unroll
  for (int c = 0; c < 4; ++c)
    qf[c] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(
                                           rq, (uint32_t)(lr * AD + lq * 8 + 32 * c) * 2u, 0, 0));

  // score lanes: head lr, tokens 4 lq .. 4 lq + 3 of a block;
  // value lanes: dimensions 8 lr .. 8 lr + 7, tokens lq, lq + 4, lq + 8, lq + 12
  float m_run = -INFINITY, l_part = 0.f;
  float o[G][8];
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int e = 0; e < 8; ++e) o[g][e] = 0.f;

  auto load_k = [&](int blk, bf16x8 (&kf)[4]) {
    const int tok = t0 + blk * 16 + lr;
    const uint32_t base = tok < t1 ? blk_off(blk, kpg) + (uint32_t)(lr * AD + lq * 8) * 2u : kAtOOB;
#pragma unroll
    for (int c = 0; c < 4; ++c)
      kf[c] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(rk, base, 64 * c, 0));
  };
  auto load_v = [&](int blk, v4u (&vf)[4]) {
    const uint32_t r0 = blk_off(blk, vpg);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int tok = t0 + blk * 16 + 4 * i + lq;
      vf[i] = __builtin_amdgcn_raw_buffer_load_b128(
          rv, tok < t1 ? r0 + (uint32_t)((4 * i + lq) * AD + lr * 8) * 2u : kAtOOB, 0, 0);
    }
  };

  bf16x8 kc[4], kn[4];
  v4u vc[4], vn[4];
  load_k(0, kc);
  load_v(0, vc);
  for (int blk = 0; blk < nblk; ++blk) {
    const bool more = blk + 1 < nblk;
    if (more) {
      load_k(blk + 1, kn);
      load_v(blk + 1, vn);
    }
    f32x4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < 4; ++c) s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kc[c], qf[c], s, 0, 0, 0);
    // mask tokens past the split, scale, block max per head
    float bm = -INFINITY;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int tok = t0 + blk * 16 + 4 * lq + r;
      s[r] = tok < t1 ? s[r] * p.scale : -INFINITY;
      bm = fmaxf(bm, s[r]);
    }
    bm = fmaxf(bm, __shfl_xor(bm, 16));
    bm = fmaxf(bm, __shfl_xor(bm, 32));
    const float m_new = fmaxf(m_run, bm);   // finite: every block has a token
    const float alpha = __expf(m_run - m_new);
    m_run = m_new;
    float ps = 0.f;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float e = __expf(s[r] - m_new);
      ps += e;
      if (lr < G) sp[(4 * lq + r) * 16 + lr] = e;
    }
    l_part = l_part * alpha + ps;
    if (lane < G) sp[256 + lane] = alpha;
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    // P.V on the value lanes
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float a = sp[256 + g];
#pragma unroll
      for (int e = 0; e < 8; ++e) o[g][e] *= a;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int t = 4 * i + lq;
      float vx[8];
      vx[0] = bf_lo(vc[i].x); vx[1] = bf_hi(vc[i].x);
      vx[2] = bf_lo(vc[i].y); vx[3] = bf_hi(vc[i].y);
      vx[4] = bf_lo(vc[i].z); vx[5] = bf_hi(vc[i].z);
      vx[6] = bf_lo(vc[i].w); vx[7] = bf_hi(vc[i].w);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float pg = sp[t * 16 + g];
#pragma unroll
        for (int e = 0; e < 8; ++e) o[g][e] = fmaf(pg, vx[e], o[g][e]);
      }
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    if (more) {
#pragma unroll
      for (int c = 0; c < 4; ++c) kc[c] = kn[c];
#pragma unroll
      for (int i = 0; i < 4; ++i) vc[i] = vn[i];
    }
  }
  // the four token groups of a dimension chunk, and of a head's sum
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      o[g][e] += __shfl_xor(o[g][e], 16);
      o[g][e] += __shfl_xor(o[g][e], 32);
    }
  l_part += __shfl_xor(l_part, 16);
  l_part += __shfl_xor(l_part, 32);
  const size_t row0 = ((size_t)b * p.Hq + (size_t)hk * G) * p.n_splits + split;  // (b, h = hk G, split)
  if (lq == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float* dst = p.part_o + (row0 + (size_t)g * p.n_splits) * AD + lr * 8;
      *reinterpret_cast<f32x4*>(dst) = f32x4{o[g][0], o[g][1], o[g][2], o[g][3]};
      *reinterpret_cast<f32x4*>(dst + 4) = f32x4{o[g][4], o[g][5], o[g][6], o[g][7]};
    }
    if (lr < G) {
      float* ml = p.part_ml + (row0 + (size_t)lr * p.n_splits) * 2;
      ml[0] = m_run;
      ml[1] = l_part;
    }
  }
}

template <int G, bool PAGED>
__global__ void __launch_bounds__(64 * AT_WAVES) attn_decode_split(AttnParams p) {
  __shared__ float sp_all[AT_WAVES][256 + 16];
  __shared__ int box[2];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (!p.quota_off) {
    const int task = blockIdx.x * AT_WAVES + wave;
    if (task < p.tasks) attn_task<G, PAGED>(p, task, sp_all[wave]);
    return;
  }
  uint32_t xr;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xr));
  const int own = (int)(xr & 0xFu);
  if (own >= p.n_x || !((p.allow >> own) & 1u)) return;  // an XCD outside the set
  // claims: own share first, then the others in turn.  Wave 0 reads every
  // counter in one round trip and only adds to shares that still have groups;
  // the loop ends when each counter has passed its share.
  const int lane = threadIdx.x & 63;
  for (;;) {
    if (wave == 0) {
      int rem = 0, y = 0, b0 = 0, b1 = 0;
      if (lane < p.n_x) {
        y = (own + lane) % p.n_x;
        b0 = p.quota_off[y];
        b1 = p.quota_off[y + 1];
        const int taken = __hip_atomic_load(&p.claim[y * kClaimStride], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        rem = (b1 - b0 + AT_WAVES - 1) / AT_WAVES - taken;
      }
      unsigned long long open = __ballot(lane < p.n_x && rem > 0);
      int base = -1, end = 0;
      while (open && base < 0) {
        const int l = __builtin_ctzll(open);
        open &= open - 1;
        int got = -1;
        if (lane == l) {
          const int g = atomicAdd(&p.claim[y * kClaimStride], 1);
          if (b0 + g * AT_WAVES < b1) got = b0 + g * AT_WAVES;
        }
        got = __shfl(got, l);
        if (got >= 0) {
          base = got;
          end = __shfl(b1, l);
        }
      }
      if (lane == 0) {
        box[0] = base;
        box[1] = end;
      }
    }
    __syncthreads();
    const int base = box[0], end = box[1];
    __syncthreads();
    if (base < 0) break;
    if (base + wave < end) attn_task<G, PAGED>(p, base + wave, sp_all[wave]);
  }
}



// Merge of the splits of every (request, head) row (split_merge.h).  It also
// clears the aware form's claim counters for the next split launch on the
// stream (the split launch is complete when the merge runs).
template <int CH>
__global__ void __launch_bounds__(64 * kMergeWaves) attn_decode_merge(const float* __restrict__ part_o,
                                                                      const float* __restrict__ part_ml, int rows,
                                                                      int n_splits, int wpr, uint16_t* __restrict__ o,
                                                                      float* __restrict__ lse, int* claim,
                                                                      int n_claim) {
  if (claim && blockIdx.x == 0 && blockIdx.y == 0 && (int)threadIdx.x < n_claim) claim[threadIdx.x * kClaimStride] = 0;
  merge_split_rows<AD, CH>(part_o, part_ml, rows, n_splits, wpr, o, lse);
}

}  // namespace

int launch_attn_decode(const AttnLaunch& a, hipStream_t s) {
  AttnParams p;
  p.q = static_cast<const uint16_t*>(a.q);
  p.k = static_cast<const uint16_t*>(a.k);
  p.v = static_cast<const uint16_t*>(a.v);
  p.part_o = a.part_o;
  p.part_ml = a.part_ml;
  p.quota_off = a.d_quota_off;
  p.claim = a.d_claim;
  p.allow = a.allow;
  p.B = a.B;
  p.Hq = a.Hq;
  p.Hkv = a.Hkv;
  p.S = a.S;
  p.split = a.split;
  p.n_splits = a.n_splits;
  p.tasks = a.B * a.Hkv * a.n_splits;
  p.n_x = a.n_x;
  p.scale = a.scale;
  p.k_page = a.k_page;
  p.v_page = a.v_page;
  p.pages_per_head = (a.S + kPageTokens - 1) / kPageTokens;
  p.pool_bytes = a.pool_bytes;
  const int G = a.Hq / a.Hkv;
  const dim3 grid((unsigned)a.grid), block(64 * AT_WAVES);
  if (a.d_quota_off && (!a.d_claim || a.n_x > 64))
    return fail(ASYM_EINVAL, "attention: aware launch without claim counters");
  const bool paged = a.k_page != nullptr;
  if (paged && (!a.v_page || a.pool_bytes == 0 || a.pool_bytes > (1u << 31) || a.split > 64 * kPageTokens))
    return fail(ASYM_EINVAL, "attention: a paged launch needs both tables, pools of at most 2 GiB, splits of <= 2048");
#define ASYM_ATTN_CASE(g)                                                      \
  case g:                                                                      \
    if (paged)                                                                 \
      hipLaunchKernelGGL((attn_decode_split<g, true>), grid, block, 0, s, p);  \
    else                                                                       \
      hipLaunchKernelGGL((attn_decode_split<g, false>), grid, block, 0, s, p); \
    break;
  switch (G) {
    ASYM_ATTN_CASE(1)
    ASYM_ATTN_CASE(2)
    ASYM_ATTN_CASE(4)
    ASYM_ATTN_CASE(8)
    ASYM_ATTN_CASE(16)
    default: return fail(ASYM_EUNSUPPORTED, "attention: query heads per key/value head must be 1, 2, 4, 8 or 16");
  }
#undef ASYM_ATTN_CASE
  ASYM_HIP(hipGetLastError());
  const int rows = a.B * a.Hq;
  const int wpr = merge_waves_per_row(a.n_splits), rows_per_wg = kMergeWaves / wpr;
  const int groups = (rows + rows_per_wg - 1) / rows_per_wg;
  const int ch = merge_column_chunks(groups, AD / 64);
  auto merge = ch == 2 ? attn_decode_merge<2> : attn_decode_merge<1>;
  hipLaunchKernelGGL(merge, dim3((unsigned)groups, (unsigned)ch), dim3(64 * kMergeWaves), 0, s, a.part_o, a.part_ml,
                     rows, a.n_splits, wpr, static_cast<uint16_t*>(a.o), a.lse, a.d_quota_off ? a.d_claim : nullptr,
                     a.n_x);
  ASYM_HIP(hipGetLastError());
  return ASYM_OK;
}

int attn_tasks_per_workgroup() { return AT_WAVES; }

int attn_page_tokens() { return kPageTokens; }

int attn_claim_ints() { return ASYM_MAX_XCDS * kClaimStride; }

}  // namespace asym
