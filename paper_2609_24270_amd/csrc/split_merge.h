// Merge of a split sequence's partial results (flash-decoding's second pass),
// shared by the decode-attention kernels.  A split s of a (request, head) row
// left its unnormalised output o_s (D floats), its running max m_s and its sum
// l_s; the row's result is
//   M = max_s m_s,  L = sum_s exp(m_s - M) l_s,
//   O = (sum_s exp(m_s - M) o_s) / L,  lse = M + log L.
// `wpr` waves work on one row (1, 2, 4, 8 or 16, from the split count): wave
// j of a row takes splits j, j + wpr, j + 2 wpr, ... and eight of them at a
// time, so that many partial loads are in flight; the waves' sums are added in
// wave order.  A row's D columns may be cut into CH chunks, one per workgroup
// (the grid's second dimension), so that rows with many splits are read by
// more CUs; every workgroup of a row computes M and L the same way, and each
// output element is summed over the same splits in the same order whatever
// CH is.  The order depends only on the split count, so every assignment of
// the splits to workgroups gives the same bits.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

namespace asym {
namespace {

constexpr int kMergeWaves = 16;        // waves per merge workgroup
constexpr int kMergeTargetGroups = 256;  // merge workgroups wanted (one per CU of the chip)

// a lane's values: a vector of N floats, or one float (an asm operand cannot
// be a one-element vector)
template <int N>
struct MergeVec {
  typedef float type __attribute__((ext_vector_type(N)));
};
template <>
struct MergeVec<1> {
  typedef float type;
};
template <int N>
__device__ __forceinline__ float vget(const typename MergeVec<N>::type& v, int e) {
  if constexpr (N == 1)
    return v;
  else
    return v[e];
}
template <int N>
__device__ __forceinline__ void vset(typename MergeVec<N>::type& v, int e, float f) {
  if constexpr (N == 1)
    v = f;
  else
    v[e] = f;
}

// D: floats per row (128 or 512), CH: column chunks per row; lane l holds
// D / (64 CH) consecutive values of its chunk.
template <int D, int CH>
__device__ __forceinline__ void merge_split_rows(const float* __restrict__ part_o, const float* __restrict__ part_ml,
                                                 int rows, int n_splits, int wpr, uint16_t* __restrict__ o,
                                                 float* __restrict__ lse) {
  constexpr int DC = D / CH;  // columns of this workgroup's chunk
  constexpr int DPL = DC / 64;
  static_assert(DPL == 1 || DPL == 2 || DPL == 4 || DPL == 8, "1 to 8 values per lane");
  __shared__ float red[kMergeWaves][DC];
  __shared__ float red_m[kMergeWaves], red_l[kMergeWaves];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int rows_per_wg = kMergeWaves / wpr;
  const int row = blockIdx.x * rows_per_wg + wave / wpr;
  const int c0 = (int)blockIdx.y * DC + DPL * lane;  // this lane's first column
  const int sub = wave % wpr;
  const int lead = wave - sub;  // first wave of this row
  const bool valid = row < rows;
  const float* ml = part_ml + (size_t)(valid ? row : 0) * n_splits * 2;
  const float* po = part_o + (size_t)(valid ? row : 0) * n_splits * D + c0;

  // the row's max over every split: the lanes of a wave read 64 of its
  // splits at a time, then the waves' maxima are combined
  float m = -INFINITY;
  if (valid)
    for (int s = sub + wpr * lane; s < n_splits; s += 64 * wpr) m = fmaxf(m, ml[2 * s]);
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) m = fmaxf(m, __shfl_xor(m, d));
  if (lane == 0) red_m[wave] = m;
  __syncthreads();
  float M = -INFINITY;
  for (int j = 0; j < wpr; ++j) M = fmaxf(M, red_m[lead + j]);

  typedef typename MergeVec<DPL>::type vrow;
  vrow acc = {};
  float L = 0.f;
  auto load = [&](int s, vrow& x, float2& q) {
    x = *reinterpret_cast<const vrow*>(po + (size_t)s * D);
    q = *reinterpret_cast<const float2*>(ml + 2 * s);
  };
  auto add = [&](const vrow& x, float2 q) {
    const float w = __expf(q.x - M);
    L = fmaf(q.y, w, L);
#pragma unroll
    for (int e = 0; e < DPL; ++e) vset<DPL>(acc, e, fmaf(vget<DPL>(x, e), w, vget<DPL>(acc, e)));
  };
  if (valid) {
    int s = sub;
    for (; s + 7 * wpr < n_splits; s += 8 * wpr) {
      vrow x[8];
      float2 q[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) load(s + u * wpr, x[u], q[u]);
      // one empty asm that takes the whole batch: every load is issued before
      // the first of them is waited for (the compiler would otherwise place
      // each load next to its use, one memory latency per split)
      asm volatile("" : "+v"(x[0]), "+v"(x[1]), "+v"(x[2]), "+v"(x[3]), "+v"(x[4]), "+v"(x[5]), "+v"(x[6]),
                   "+v"(x[7]), "+v"(q[0]), "+v"(q[1]), "+v"(q[2]), "+v"(q[3]), "+v"(q[4]), "+v"(q[5]), "+v"(q[6]),
                   "+v"(q[7]));
#pragma unroll
      for (int u = 0; u < 8; ++u) add(x[u], q[u]);
    }
    for (; s < n_splits; s += wpr) {
      vrow x0;
      float2 q0;
      load(s, x0, q0);
      add(x0, q0);
    }
  }
  if (wpr > 1) {
#pragma unroll
    for (int e = 0; e < DPL; ++e) red[wave][DPL * lane + e] = vget<DPL>(acc, e);
    if (lane == 0) red_l[wave] = L;
  }
  __syncthreads();
  if (!valid || sub != 0) return;
  if (wpr > 1) {
#pragma unroll
    for (int e = 0; e < DPL; ++e) vset<DPL>(acc, e, red[lead][DPL * lane + e]);
    L = red_l[lead];
    for (int j = 1; j < wpr; ++j) {
#pragma unroll
      for (int e = 0; e < DPL; ++e) vset<DPL>(acc, e, vget<DPL>(acc, e) + red[lead + j][DPL * lane + e]);
      L += red_l[lead + j];
    }
  }
  const float inv = 1.f / L;
  uint16_t* dst = o + (size_t)row * D + c0;
  if constexpr (DPL == 1) {
    *dst = __builtin_bit_cast(unsigned short, (__bf16)(vget<DPL>(acc, 0) * inv));
  } else {
    uint32_t packed[DPL / 2];
#pragma unroll
    for (int e = 0; e < DPL / 2; ++e) {
      const __bf16 lo = (__bf16)(vget<DPL>(acc, 2 * e) * inv), hi = (__bf16)(vget<DPL>(acc, 2 * e + 1) * inv);
      packed[e] = (uint32_t)__builtin_bit_cast(unsigned short, lo) |
                  ((uint32_t)__builtin_bit_cast(unsigned short, hi) << 16);
    }
    if constexpr (DPL == 8)
      *reinterpret_cast<uint4*>(dst) = uint4{packed[0], packed[1], packed[2], packed[3]};
    else if constexpr (DPL == 4)
      *reinterpret_cast<uint2*>(dst) = uint2{packed[0], packed[1]};
    else
      *reinterpret_cast<uint32_t*>(dst) = packed[0];
  }
  if (lse && blockIdx.y == 0 && lane == 0) lse[row] = M + __logf(L);
}

// waves per row for a split count: enough that each wave merges about 8 splits
inline int merge_waves_per_row(int n_splits) {
  int w = 1;
  while (w < kMergeWaves && w * 8 < n_splits) w *= 2;
  return w;
}

// column chunks per row (a power of two, at most max_chunks): enough that the
// merge's workgroups number about kMergeTargetGroups
inline int merge_column_chunks(int row_groups, int max_chunks) {
  int ch = 1;
  while (ch < max_chunks && row_groups * ch < kMergeTargetGroups) ch *= 2;
  return ch;
}

}  // namespace
}  // namespace asym
