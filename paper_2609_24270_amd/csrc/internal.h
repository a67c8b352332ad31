// Internal declarations of libasym (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>
#include <vector>

#include "../../include/asym.h"

namespace asym {

// ---- errors: thread-local message, status codes from asym.h ---------------
int fail(int status, const std::string& msg);
int hip_fail(hipError_t e, const char* what);
#define ASYM_HIP(call)                                   \
  do {                                                   \
    hipError_t e_ = (call);                              \
    if (e_ != hipSuccess) return ::asym::hip_fail(e_, #call); \
  } while (0)

// ---- topology ---------------------------------------------------------------
struct CuRecord {
  int xcc, se, sh, cu;
  int mask_bit;  // -1 if unknown
};

struct Topology {
  int device = -1;
  int n_xccs = 0;
  int n_cus = 0;
  std::vector<CuRecord> cus;             // dense order: sorted (xcc, se, sh, cu)
  std::vector<int> cus_per_xcd;          // [n_xccs]
  std::vector<int> bit_to_cu;            // mask bit -> dense CU index, -1 unknown
  bool has_maskmap = false;
  double rr_fraction = -1.0;             // round-robin dispatch agreement
  bool has_latency = false;
  asym_latency_summary lat{};
  unsigned flags = 0;                    // what was probed (asym_probe_flags)
  std::string compute_partition = "unknown", memory_partition = "unknown";
  std::string key;                       // chip and configuration it was probed on
};

// The chip and configuration a probe result belongs to (PCI bus id, UUID,
// runtime and driver versions, architecture, partition modes, counts), as one
// line of text; a cached topology is reused only under the same key.
int device_key(int device, std::string* key, asym_device_info* info);
// Cache file of a topology (text; host only).  load: ASYM_ENOCACHE with the
// reason when the file is missing, made under another key, lacks a requested
// probe, or is malformed or breaks an invariant.
int topology_save(const Topology& t, const char* path);
// The driver's current compute and memory partition modes of the PCI function
// (sysfs), or "unknown"; each written as a C string of at most len bytes.
int read_partition_modes(const char* pci_bus_id, char* compute, char* memory, size_t len);
int topology_load(const char* path, const std::string& key, unsigned flags, Topology* out);

// Fields of the HW_ID hardware register (GCN/CDNA layout).
inline int hwid_cu(uint32_t h) { return (h >> 8) & 0xF; }
inline int hwid_sh(uint32_t h) { return (h >> 12) & 0x1; }
inline int hwid_se(uint32_t h) { return (h >> 13) & 0x7; }
inline int xccid(uint32_t x) { return x & 0xF; }

// Build the dense map from raw identity records {xcc reg, hw_id reg, block, _}.
int build_topology(const int32_t* rec, int n, int n_cus_expected,
                   int n_xccs_expected, const int32_t* mask_bit_record,
                   Topology& out);
// Exact invariants: every CU once, per-XCD counts sum to n_cus, bijective map.
int check_invariants(const Topology& t);
// Per-XCD CU counts of a mask; needs the mask map unless the mask is full.
int mask_counts(const Topology& t, const uint32_t* mask, std::vector<int>& per_xcd);

// Default per-device topology (identity probe on first use).
int default_topology(int device, const Topology** out);

// ---- schedule ---------------------------------------------------------------
struct Schedule {
  int tiles_m = 0, tiles_n = 0, n_xcds = 0;
  std::vector<int> order;   // tile ids
  std::vector<int> off;     // [n_xcds + 1]
  std::vector<int> quota;   // [n_xcds]
};
int build_schedule(int tiles_m, int tiles_n, int n_xcds, const int* slots,
                   int mapping, int band, Schedule& s);
std::vector<int> largest_remainder_quotas(int total, const std::vector<int>& w);
int build_grouped_schedule(int G, const int* tiles_m, int tiles_n, int n_xcds, const int* slots,
                           int mapping, Schedule& s);

// ---- device entry points (implemented in .hip files) -------------------------
struct GemmLaunch {
  const void* A; const void* B; void* C;
  int M, N, K, lda, ldb, ldc;
  int mapping;                 // asym_mapping
  const int* d_order;          // device tile order
  const int* d_off;            // device [ASYM_MAX_XCDS+1]
  const int* d_slots;          // device [ASYM_MAX_XCDS]
  int* d_ctr;                  // device counters of the dynamic form (self-resetting)
  bool dynamic;                // aware mapping on an uneven CU set: claims, not static
  int grid;                    // workgroups
  int tiles_m, tiles_n;
  int n_xccs;
  bool vec;                    // aligned vector path
  int bn;                      // tile width: 256, or 224 / 192 on the vector path; 128 with bm = 128
  int bm = 256;                // tile height: 256, or 128 (128 x 128 tiles, register-staged path)
  const void* d_desc = nullptr; // grouped GEMM: device int4 per tile {row, rows, group B row, column}
  void* d_trace = nullptr;      // traced launch: device asym_wg_record per workgroup
};
int launch_gemm(const GemmLaunch& g, hipStream_t s);

// Small-M path (at most 64 rows per row tile; vector-path alignment).
struct SmallMLaunch {
  const void* A; const void* B; void* C;
  int M, N, K, lda, ldb, ldc;
  int mb;                       // 16-row blocks per row tile: 1, 2 or 4
  int row_tiles = 1;            // plain GEMM: row tiles of 16 mb rows
  int order = 0;                // plain GEMM: 0 aware, 1 column-major, 2 row-major
  int n_x = 8;                  // XCDs
  long long grid = 0;           // workgroups
  const void* d_desc = nullptr; // grouped: device int4 per workgroup {row, rows, B row, column}
  int tile_cols = 64;           // columns per column tile: a multiple of 8 up to 64 (plain, unsplit)
  int ksplit = 1;               // plain, one row tile: K ranges per column tile
  float* part = nullptr;        // ksplit > 1: [column tiles][ksplit][16 mb][64] fp32
};
int launch_gemm_small_m(const SmallMLaunch& g, hipStream_t s);
int small_m_blocks(int max_rows);  // 1, 2, 4, or 0 above 64 rows
int small_m_tile_cols();           // the widest column tile (64)
int small_m_cols(int N, int mb, int row_tiles, int ksplit, int device_cus);  // the width a plain launch takes

// Decode attention (head dimension 128).
struct AttnLaunch {
  const void *q, *k, *v;
  void* o;
  float* lse;                 // nullable
  float* part_o;              // [B][Hq][n_splits][128]
  float* part_ml;             // [B][Hq][n_splits][2]
  const int* d_quota_off;     // aware: device [n_x + 1]; null = oblivious
  int* d_claim = nullptr;     // aware: claim counters, zero at launch (the merge clears them)
  uint32_t allow = 0xFFFFFFFFu; // aware: XCDs whose workgroups work
  int B, Hq, Hkv, S, split, n_splits, n_x, grid;
  float scale;
  const int* k_page = nullptr;  // paged form: device tables [B][Hkv][ceil(S / 32)]; null = dense K, V
  const int* v_page = nullptr;
  uint32_t pool_bytes = 0;      // paged form: bytes of each pool (<= 2^31)
};
int launch_attn_decode(const AttnLaunch& a, hipStream_t s);
int attn_tasks_per_workgroup();
int attn_page_tokens();  // tokens per page of the paged form (8 KiB of one head)

// Multi-head latent attention, decode (576-wide cache rows, 512-wide values).
struct MlaLaunch {
  const void *q, *kv;
  void* o;
  float* lse;                 // nullable
  float* part_o;              // [B][Hq][n_splits][512]
  float* part_ml;             // [B][Hq][n_splits][2]
  const int* d_quota_off;     // aware: device [n_x + 1]; null = oblivious
  int* d_claim = nullptr;     // aware: claim counters, zero at launch (the merge clears them)
  uint32_t allow = 0xFFFFFFFFu;
  int B, Hq, S, split, n_splits, n_x, grid;
  float scale;
  int form = 0;               // 0: a task is one head block on one wave; 1, 2: 4 or 8 head blocks on one workgroup
};
int launch_mla_decode(const MlaLaunch& a, hipStream_t s);
int mla_tasks_per_workgroup();  // wave form: tasks (head blocks) per workgroup
int mla_form_head_blocks(int form);  // head blocks per task of a kernel form
int attn_claim_ints();  // ints of the aware form's claim counters

int probe_identity_run(int device, hipStream_t s, int n_blocks,
                       std::vector<int32_t>& rec, int pre_blocks = 0);
// Dispatch of n workgroups (block index block[i] ran on XCC xcc[i]): the share
// of workgroups on the XCC holding most of their residue class (block mod n_x),
// and the rotation k for which xcc = (block + k) mod n_x fits most (host only).
void dispatch_stats(const int* block, const int* xcc, int n, int n_x, double* class_fraction, int* rotation);
int probe_latency_run(int device, Topology& t);
int latency_probe(int device, const asym_latency_params& p, uint32_t* lat_out,
                  asym_latency_summary& out);
// One latency measurement over explicit line offsets of a fresh allocation of
// `alloc` bytes (2 MiB aligned): per XCD and pass, the HBM regime over every
// offset, the L2 regime over the first l2_samples and (if mall) the
// memory-side-cache regime over every offset; best = per-(regime, XCD,
// offset) minima, [3][n_x][offs.size()], regimes L2, MALL, HBM (UINT32_MAX
// where not timed).  Each timed load is preceded by a load of the line at
// offset ^ touch_delta (translation warm-up; must stay in the allocation).
struct LatencyMeasure {
  size_t alloc = 0;
  std::vector<uint64_t> offs;
  int passes = 8;
  int l2_samples = 0;
  bool mall = true;
  uint64_t touch_delta = 1ull << 20;
  const void* ext_base = nullptr;  // time lines of this caller allocation of `alloc`
                                   // bytes (read only) instead of a fresh one
  int n_x = 0;                     // out
  std::vector<uint32_t> best;      // out
  double timer_overhead = -1.0;    // out
  double clock_mhz = -1.0;         // out
  uint64_t base_align = 0;         // out: largest power of two dividing the base address
};
int latency_measure(int device, LatencyMeasure& m);
// home map analysis (numa_host.cpp): the homes of every chunk from the timed page and verification lines
int home_map_analyze(const uint32_t* L, int n_x, int n_pages, const uint64_t* voffs, int n_verify,
                     const int* grp, uint64_t hash_mask, int chunk_log2, double tie, int8_t* chunk_home,
                     asym_home_map_info& info);
// Affinity groups and home groups from HBM latencies [n_x][n_s] (host only);
// home (nullable, n_s entries) receives each address's home group, -1 if tied.
int analyze_latency(const uint32_t* lat, int n_x, int n_s, double threshold, double tie,
                    asym_latency_summary& out, int8_t* home = nullptr);

// Partition-hash analysis of HBM latencies [n_x][n_a] over offsets in blocks (host only).
int analyze_interleave(const uint32_t* L, int n_x, int n_a, const uint64_t* offs, int block,
                       double threshold, double tie, double decide, int8_t* home_out,
                       asym_interleave_result& r);

// Bandwidth-bound co-runner: `passes` reads of a whole buffer (sink: grid x
// 256 x 16 bytes).
// reading CUs per XCD cus[n_x] (0 = no share) -> a grid whose workgroups all fit at once
int stream_read_grid(const int* cus, int n_x);
int launch_stream_read(const void* src, size_t n_bytes, int passes, void* sink, int grid, const int* cus,
                       int n_x, hipStream_t s);

// Streaming copy: `passes` passes of dst = src over n_bytes (a multiple of 16),
// the buffer cut into per-XCD slices in proportion to cus[n_x] (0 = no slice);
// stop_flag (nullable) is read before every pass after the first.
int copy_grid(const int* cus, int n_x);
int launch_copy(void* dst, const void* src, size_t n_bytes, int passes, const int* stop_flag,
                const int* cus, int n_x, int grid, hipStream_t s);
// dst[c][r] = src[r][c] (bf16; row pitches lds >= cols and ldd >= rows)
int launch_transpose_bf16(const void* src, int rows, int cols, int lds, void* dst, int ldd, hipStream_t s);
// zero n 4-byte words at p, ordered on stream s
int launch_zero_words(void* p, size_t n, hipStream_t s);
// dst[0 .. n) = host[0 .. n) (4-byte words), ordered on stream s, carried in
// kernel arguments: no staging buffer, no allocation
int launch_put_words(int* dst, const int* host, size_t n, hipStream_t s);

// GEMM with every device buffer beyond A, B and C (tile schedule, claim
// counters, split-K partials) in the caller's scratch area of `bytes` bytes
// at device address `scratch` (layout below); allocates no device memory.
// Calls that share one scratch area and overlap in time race.
constexpr size_t kScratchCtrOff = 0;              // 64 ints: claim counters
constexpr size_t kScratchOffOff = 256;            // ASYM_MAX_XCDS + 1 ints: region offsets
constexpr size_t kScratchSlotsOff = 384;          // ASYM_MAX_XCDS ints: workers per XCD
constexpr size_t kScratchOrderOff = 512;          // the tile order
constexpr size_t kScratchPartOff = 1u << 20;      // fp32 partial tiles of a split K
constexpr size_t kScratchPartBytes = 16u << 20;  // split K: fewer than 4 x CUs (tile, range) pairs of 16 KiB
constexpr size_t kScratchBytes = kScratchPartOff + kScratchPartBytes;
constexpr int kScratchMaxTiles = (int)((kScratchPartOff - kScratchOrderOff) / sizeof(int));
// the checks that need no device: a topology given, [N][K] storage, a tile
// count within the array's schedule
int gemm_noalloc_check(const asym_topology* topo, int M, int N, int b_layout);
int gemm_bf16_scratch(const asym_topology* topo, int M, int N, int K, const void* A, int lda, const void* B,
                      int ldb, int b_layout, void* C, int ldc, int mapping, uint32_t xcd_mask,
                      hipStream_t stream, unsigned char* scratch, size_t bytes);
void release_workspace(hipStream_t s);

// Stream CU mask -> CU set seen by the scheduler.
int stream_cu_mask(hipStream_t s, int n_cus, uint32_t* mask /*ASYM_MASK_WORDS*/);

}  // namespace asym
