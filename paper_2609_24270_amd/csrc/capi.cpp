// C ABI of libasym: argument checking, device discovery, per-stream device
// workspaces, schedule caching, masked streams, and the co-run harness.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cctype>

#include <algorithm>
#include <cmath>
#include <atomic>
#include <chrono>
#include <cstring>
#include <map>
#include <memory>
#include <mutex>
#include <thread>
#include <tuple>

#include "internal.h"

struct asym_topology;

namespace asym {

const Topology* unwrap(const asym_topology* p);
asym_topology* wrap_topology(Topology&& t);
int gemm_tile_m();
int gemm_tile_n();

static thread_local std::string g_last_error;

int fail(int status, const std::string& msg) {
  g_last_error = msg;
  return status;
}

int hip_fail(hipError_t e, const char* what) {
  g_last_error = std::string(what) + ": " + hipGetErrorString(e);
  return ASYM_EHIP;
}

// ---- process-wide state, guarded by one mutex --------------------------------
namespace {

std::mutex g_mu;

struct ScheduleKey {
  int device, tiles_m, tiles_n, mapping;
  std::vector<int> slots;
  bool operator<(const ScheduleKey& o) const {
    return std::tie(device, tiles_m, tiles_n, mapping, slots) <
           std::tie(o.device, o.tiles_m, o.tiles_n, o.mapping, o.slots);
  }
};
struct DeviceSchedule {
  int* d_order = nullptr;
  int* d_off = nullptr;    // [ASYM_MAX_XCDS + 1]
  int* d_slots = nullptr;  // [ASYM_MAX_XCDS]
};
std::map<ScheduleKey, DeviceSchedule> g_schedules;  // never freed: kernels may still read them

// One grouped problem's device tables: tile descriptors, and the schedule
// (order [T], off [MAX_XCDS + 1], slots [MAX_XCDS]).
struct GroupedTables {
  std::vector<int> key;   // row counts, N, tile width, mapping, slots
  int4* desc = nullptr;
  int* sched = nullptr;
  int T = 0;
};
constexpr size_t kGroupedCache = 8;

// Device counters per (device, stream): launches on one stream run in order
// and the kernels leave their counters zeroed, so one block per stream does.
struct Workspace {
  int* gemm_ctr = nullptr;                  // 64 ints (dynamic aware GEMM)
  // grouped GEMM: device copies of recent tile tables and schedules, most
  // recent first (a repeated call reuses its tables), and a pinned host
  // staging buffer with an event recorded after the copies out of it: the
  // next upload waits for it before writing the staging again
  std::vector<GroupedTables> g_tables;
  void* g_host = nullptr;
  size_t g_host_bytes = 0;
  hipEvent_t g_copied = nullptr;
  bool g_pending = false;
  // decode attention: split partials (grown on demand) and the per-XCD task
  // offsets of recent aware plans (key: tasks, per-XCD slots), most recent first
  float* attn_buf = nullptr;
  size_t attn_bytes = 0;
  int* attn_claim = nullptr;  // claim counters of the aware form, one 256-byte line each
  // small-M GEMM with a split K: fp32 partial tiles (grown on demand)
  float* sm_part = nullptr;
  size_t sm_part_bytes = 0;
  // B stored [K][N]: its transpose, [N][K rounded up to 8] (grown on demand)
  void* kn_buf = nullptr;
  size_t kn_bytes = 0;
  std::vector<std::pair<std::vector<int>, int*>> attn_off;
};

std::map<std::pair<int, hipStream_t>, Workspace> g_ws;

std::map<int, std::unique_ptr<Topology>> g_default_topo;

}  // namespace

// A stream's workspace, created at its first use.  Nothing here waits for
// other streams: the counters are cleared by a kernel ordered on s (a blocking
// hipMemset would run on the null stream, which waits for every other stream,
// and so would hold a launch back until a co-running kernel ended).
static int get_workspace(int device, hipStream_t s, Workspace** out) {
  auto key = std::make_pair(device, s);
  auto it = g_ws.find(key);
  if (it == g_ws.end()) {
    Workspace w;
    ASYM_HIP(hipMalloc(&w.gemm_ctr, 64 * sizeof(int)));
    int rc = launch_zero_words(w.gemm_ctr, 64, s);
    if (rc != ASYM_OK) {
      (void)hipFree(w.gemm_ctr);
      return rc;
    }
    it = g_ws.emplace(key, w).first;
  }
  *out = &it->second;
  return ASYM_OK;
}

int default_topology(int device, const Topology** out) {
  auto it = g_default_topo.find(device);
  if (it == g_default_topo.end()) {
    asym_topology* t = nullptr;
    int rc = asym_probe_topology(device, ASYM_PROBE_IDENTITY, nullptr, &t);
    if (rc != ASYM_OK) return rc;
    const Topology* tt = unwrap(t);
    g_default_topo[device] = std::make_unique<Topology>(*tt);
    asym_topology_free(t);
    it = g_default_topo.find(device);
  }
  *out = it->second.get();
  return ASYM_OK;
}

int stream_cu_mask(hipStream_t s, int n_cus, uint32_t* mask) {
  std::memset(mask, 0, sizeof(uint32_t) * ASYM_MASK_WORDS);
  uint32_t m[ASYM_MASK_WORDS] = {0};
  hipError_t e = hipExtStreamGetCUMask(s, ASYM_MASK_WORDS, m);
  if (e != hipSuccess) {
    // streams without a queue of their own (the null stream) report no mask:
    // they run on the whole device
    (void)hipGetLastError();
    std::memset(m, 0, sizeof m);
  }
  int pop = 0;
  for (int b = 0; b < n_cus; ++b)
    if ((m[b >> 5] >> (b & 31)) & 1u) {
      mask[b >> 5] |= 1u << (b & 31);
      ++pop;
    }
  if (pop == 0)  // no mask reported: the whole device
    for (int b = 0; b < n_cus; ++b) mask[b >> 5] |= 1u << (b & 31);
  return ASYM_OK;
}

static int current_device(int* dev) {
  ASYM_HIP(hipGetDevice(dev));
  return ASYM_OK;
}

// The device copy of a schedule, built and uploaded at its first use.  The
// copies are ordered on the launch stream, and only that stream is waited for
// (the host arrays are then free): a blocking hipMemcpy would wait for every
// other stream too.
static int upload_schedule(int device, int tiles_m, int tiles_n, int mapping,
                           const std::vector<int>& slots, hipStream_t stream, const DeviceSchedule** out) {
  ScheduleKey key{device, tiles_m, tiles_n, mapping, slots};
  auto it = g_schedules.find(key);
  if (it == g_schedules.end()) {
    Schedule s;
    int rc = build_schedule(tiles_m, tiles_n, (int)slots.size(), slots.data(), mapping, 0, s);
    if (rc != ASYM_OK) return rc;
    std::vector<int> off(ASYM_MAX_XCDS + 1, s.off.back()), sl(ASYM_MAX_XCDS, 0);
    for (size_t x = 0; x < s.off.size(); ++x) off[x] = s.off[x];
    for (size_t x = 0; x < slots.size(); ++x) sl[x] = slots[x];
    DeviceSchedule d;
    ASYM_HIP(hipMalloc(&d.d_order, sizeof(int) * s.order.size()));
    ASYM_HIP(hipMalloc(&d.d_off, sizeof(int) * off.size()));
    ASYM_HIP(hipMalloc(&d.d_slots, sizeof(int) * sl.size()));
    ASYM_HIP(hipMemcpyAsync(d.d_order, s.order.data(), sizeof(int) * s.order.size(), hipMemcpyHostToDevice,
                            stream));
    ASYM_HIP(hipMemcpyAsync(d.d_off, off.data(), sizeof(int) * off.size(), hipMemcpyHostToDevice, stream));
    ASYM_HIP(hipMemcpyAsync(d.d_slots, sl.data(), sizeof(int) * sl.size(), hipMemcpyHostToDevice, stream));
    ASYM_HIP(hipStreamSynchronize(stream));
    it = g_schedules.emplace(key, d).first;
  }
  *out = &it->second;
  return ASYM_OK;
}

static bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// Tile width of the vector path (the height is always 256): the one with the
// least time per launch in the model  ceil(tiles / workers) x width / eff,
// i.e. whole waves of tiles, each as long as its width, with eff the measured
// relative MFMA efficiency of the narrower tiles.  Decoder shapes gain most:
// 4096 x 6144 is 1.5 waves of 256-wide tiles on 256 CUs but 2 waves of
// 192-wide ones; 4096 x 14336 is 3.5 waves at 256 but 4 at 224.
static int choose_tile_width(int M, int N, int workers) {
  static const int widths[3] = {256, 224, 192};
  static const double eff[3] = {1.0, 0.97, 0.94};
  const int64_t tm = (M + 255) / 256;
  int best = 256;
  double best_cost = 0;
  for (int i = 0; i < 3; ++i) {
    const int64_t tiles = tm * ((N + widths[i] - 1) / widths[i]);
    const int64_t waves = (tiles + workers - 1) / workers;
    const double cost = (double)waves * widths[i] / eff[i];
    if (i == 0 || cost < best_cost * (1.0 - 1e-9)) {
      best = widths[i];
      best_cost = cost;
    }
  }
  return best;
}

// Everything a launch decides before it touches the device: arguments checked,
// the CU set read off the stream, the tile width and the aware form chosen.
// Called with g_mu held.
struct GemmPlan {
  const Topology* t = nullptr;
  int device = 0;
  std::vector<int> per, slots;
  int total = 0, smax = 0;
  bool vec = false, dynamic = false, whole = true;
  bool vec_ab = false;  // A and B alone meet the vector-path alignment
  int bn = 0, bm = 256, tiles_m = 0, tiles_n = 0, grid = 0;
  int small_mb = 0;  // > 0: the small-M kernel with this many 16-row blocks
  bool b_transposed = false;  // B stored [K][N]: transposed into a library buffer first
};

// Row pitch (elements) of the transposed copy of a [K][N] operand.
static int kn_pitch(int K) { return (K + 7) / 8 * 8; }

// The small-M kernel serves row tiles of at most 64 rows when A and B meet the
// vector-path alignment (C may have any stride) and the GEMM runs on every XCD
// of its CU set (a whole-XCD restriction needs
// the persistent kernel, whose workers leave the excluded XCDs).
std::atomic<bool> g_small_m{true};
// latent-attention decode: which kernel forms may run (0: waves only; 1: up to
// the 64-head workgroup form; 2: also the 128-head form where it has enough
// tasks; 3: the 128-head form wherever the head count allows)
std::atomic<int> g_mla_form{2};

// Up to 64 rows (per group) the small-M kernel always wins (measured: decode
// projections and 20-row expert groups).  From 65 to kSmallMMaxRows rows it
// runs 64-row tiles, and each of them re-reads the shared A fragments from LDS
// in every wave, so it only wins while its workgroups fit about two per CU
// (where the persistent kernel's 256-row tiles leave most CUs idle); with more
// work the persistent kernel is faster (measured: 4096- and 14336-column
// products of 64 to 512 rows, the 192-row expert groups).
constexpr int kSmallMMaxRows = 256;

int small_m_for(const GemmPlan& P, int max_rows, long long wgs_at_64_rows) {
  if (!g_small_m.load() || !P.vec_ab || !P.whole || max_rows > kSmallMMaxRows) return 0;
  if (max_rows <= 64) return small_m_blocks(max_rows);
  return wgs_at_64_rows <= 2ll * P.total ? 4 : 0;
}

// Workgroups of a plain small-M launch: the aware order pads the column tiles
// to a multiple of the XCD count.
long long small_m_grid(int row_tiles, int tiles_n, int order, int n_x) {
  if (order == 0) return (long long)((tiles_n + n_x - 1) / n_x) * row_tiles * n_x;
  return (long long)row_tiles * tiles_n;
}

int small_m_order(int mapping) {
  return mapping == ASYM_MAP_AWARE ? 0 : mapping == ASYM_MAP_OBLIVIOUS_GROUPED ? 1 : 2;
}

// A CU reads HBM at about 20-24 GB/s at most, so a single row tile with fewer
// 64-column tiles than the device has CUs splits K into ranges, one workgroup
// each (up to 8, each range at least two stages of k-steps); a second launch
// adds the ranges' fp32 tiles in range order (the launch boundary makes the
// partial tiles of every XCD visible; a hand-off inside the kernel needs
// device-scope fences that write back and invalidate whole L2s, and measured
// slower than no split).  The count depends only on the shape and the device,
// not on the stream's CU set, so a product has the same bits on every CU set
// it runs on with the small-M kernel.  A whole-XCD restriction sends it to the
// persistent kernel instead (one MFMA chain over all of K per output), whose
// fp32 sums can differ in the last bits from a split product's; without a
// split the two kernels agree bitwise.
int small_m_ksplit(int M, int N, int K, int mb, int device_cus) {
  if (M > 64) return 1;
  const int tiles = (N + small_m_tile_cols() - 1) / small_m_tile_cols();
  const int steps = (K + 31) / 32;
  const int u = mb == 4 ? 4 : 8;
  // only when the column tiles leave half the CUs idle, then about two
  // workgroups per CU in a power of two of ranges, each at least two stages
  // (measured on the decode shapes: 96 column tiles ran 18.6 us in 2 ranges
  // and 15.4 us in 8; 224 tiles gained nothing, a 23.8 us split kernel plus a
  // 4.5 us reduction against 28.7 us unsplit)
  if (2 * tiles > device_cus) return 1;
  int ks = 1;
  while (ks < 8 && (long long)ks * tiles < 2ll * device_cus) ks *= 2;
  while (ks > 1 && ks * 2 * u > steps) ks /= 2;
  return ks;
}

// An unsplit product takes the column-tile width, a multiple of 8 up to 64,
// that minimises what the busiest CU reads: ceil(workgroups / CUs) x (the
// tile's 16 mb rows of A + its columns of B, per k), since a CU reads at about
// 20-24 GB/s at most.  A narrower width is taken only when that saves at least
// 7% over 64 columns (the widest on ties; measured: 32 x 14336 x 4096, 256
// tiles of 56 columns instead of 224 of 64, 8% less read and 4% faster;
// 32 x 10240 x 4096 in 40 columns, 1.08x; 128 x 4096 x 4096 in 32 columns,
// 1.25x; 128 x 14336 x 4096 in 56 columns would save 6% and ran 1.4% slower).
// A wave with no columns at a tile's edge computes nothing; a narrower wave is
// the same case as the product's edge, and each output is still one wave's
// MFMA chain over all of K: the bits do not change.
int small_m_cols(int N, int mb, int row_tiles, int ksplit, int device_cus) {
  const int w = small_m_tile_cols();
  if (ksplit != 1 || device_cus < 1 || row_tiles < 1) return w;
  auto cost = [&](int c) {
    const long long wgs = (long long)row_tiles * ((N + c - 1) / c);
    return (wgs + device_cus - 1) / device_cus * (16 * mb + c);
  };
  const long long wide = cost(w);
  int best = w;
  long long best_cost = wide;
  for (int c = w - 8; c >= 8; c -= 8) {
    const long long k = cost(c);
    if (k < best_cost && k * 100 <= wide * 93) {
      best_cost = k;
      best = c;
    }
  }
  return best;
}

// The CU set a launch on `stream` may use: the device's topology (probed on
// first use unless given), the stream's per-XCD CU counts, and the workers per
// XCD after an optional whole-XCD restriction (one per CU).
struct CuSet {
  const Topology* t = nullptr;
  int device = 0;
  std::vector<int> per, slots;
  int total = 0, smax = 0;
  bool whole = true;
};

static int cu_set_for(const asym_topology* topo_in, int mapping, uint32_t xcd_mask, hipStream_t stream,
                      const char* what, CuSet* cs) {
  const std::string w(what);
  int device = 0;
  int rc = current_device(&device);
  if (rc != ASYM_OK) return rc;
  const Topology* t = unwrap(topo_in);
  if (!t) {
    rc = default_topology(device, &t);
    if (rc != ASYM_OK) return rc;
  } else if (t->device != device && t->device >= 0) {
    return fail(ASYM_EINVAL, w + ": topology was probed on another device");
  }
  uint32_t mask[ASYM_MASK_WORDS];
  rc = stream_cu_mask(stream, t->n_cus, mask);
  if (rc != ASYM_OK) return rc;
  std::vector<int> per;
  rc = mask_counts(*t, mask, per);
  if (rc != ASYM_OK) return rc;
  const uint32_t all = (t->n_xccs >= 32) ? 0xFFFFFFFFu : ((1u << t->n_xccs) - 1u);
  const uint32_t xm = xcd_mask == 0 ? all : (xcd_mask & all);
  if (xcd_mask != 0 && (xcd_mask & ~all)) return fail(ASYM_EINVAL, w + ": xcd_mask names XCDs the device does not have");
  if (mapping != ASYM_MAP_AWARE && xm != all)
    return fail(ASYM_EUNSUPPORTED, w + ": XCD restriction needs the aware mapping (oblivious mappings place work statically)");
  for (int x = 0; x < t->n_xccs; ++x)
    if (per[x] == 0)
      return fail(ASYM_EUNSUPPORTED, w + ": the stream's CU mask leaves XCD " + std::to_string(x) +
                                         " without a CU; workgroups dealt to it could never run");
  std::vector<int> slots(t->n_xccs, 0);
  int total = 0, smax = 0;
  for (int x = 0; x < t->n_xccs; ++x) {
    slots[x] = ((xm >> x) & 1u) ? per[x] : 0;
    total += slots[x];
    smax = std::max(smax, slots[x]);
  }
  if (total == 0) return fail(ASYM_EINVAL, w + ": the CU set is empty");
  cs->t = t;
  cs->device = device;
  cs->per = std::move(per);
  cs->slots = std::move(slots);
  cs->total = total;
  cs->smax = smax;
  cs->whole = xm == all;
  return ASYM_OK;
}

static int plan_gemm(const asym_topology* topo_in, int M, int N, int K, const void* A, int lda,
                     const void* B, int ldb, int b_layout, const void* C, int ldc, int mapping,
                     uint32_t xcd_mask, hipStream_t stream, GemmPlan* P, bool small_tiles = true) {
  if (M < 1 || N < 1 || K < 1) return fail(ASYM_EINVAL, "gemm: M, N, K must be >= 1");
  if (!A || !B || !C) return fail(ASYM_EINVAL, "gemm: null matrix pointer");
  if (lda < K || ldc < N) return fail(ASYM_EINVAL, "gemm: leading dimension too small");
  if (b_layout == ASYM_B_KN) {
    // B stored [K][ldb]: the kernels read its transpose, written to a
    // library buffer [N][kn_pitch(K)] (16-byte aligned rows); plan for that
    if (ldb < N) return fail(ASYM_EINVAL, "gemm: leading dimension too small");
    if ((int64_t)K * ldb * 2 >= (1ll << 40)) return fail(ASYM_EUNSUPPORTED, "gemm: B too large");
    P->b_transposed = true;
    ldb = kn_pitch(K);
    B = reinterpret_cast<const void*>((uintptr_t)256);  // a 16-byte aligned stand-in for the buffer
  } else if (b_layout != ASYM_B_NK) {
    return fail(ASYM_EINVAL, "gemm: unknown B layout");
  }
  if (ldb < K) return fail(ASYM_EINVAL, "gemm: leading dimension too small");
  if (mapping != ASYM_MAP_AWARE && mapping != ASYM_MAP_OBLIVIOUS_GROUPED &&
      mapping != ASYM_MAP_OBLIVIOUS_ROWMAJOR)
    return fail(ASYM_EINVAL, "gemm: unknown mapping");
  // one tile's rows must be addressable by a 32-bit buffer offset
  const int64_t BMr = gemm_tile_m(), BNr = gemm_tile_n();
  if ((int64_t)BMr * lda * 2 >= (1ll << 31) || (int64_t)BNr * ldb * 2 >= (1ll << 31) ||
      (int64_t)BMr * ldc * 2 >= (1ll << 31))
    return fail(ASYM_EUNSUPPORTED, "gemm: leading dimension too large for 32-bit tile offsets");

  CuSet cs;
  int rc = cu_set_for(topo_in, mapping, xcd_mask, stream, "gemm", &cs);
  if (rc != ASYM_OK) return rc;
  const Topology* t = cs.t;
  const int device = cs.device, total = cs.total, smax = cs.smax;
  std::vector<int> per = cs.per, slots = cs.slots;

  const bool vec_ab = aligned16(A) && aligned16(B) && (K % 8 == 0) && (lda % 8 == 0) && (ldb % 8 == 0);
  const bool vec = vec_ab && (((uintptr_t)C & 7u) == 0) && (ldc % 4 == 0);
  P->t = t;
  P->device = device;
  P->total = total;
  P->smax = smax;
  P->vec = vec;
  P->vec_ab = vec_ab;
  P->bm = (int)BMr;
  P->bn = vec ? choose_tile_width(M, N, total) : (int)BNr;
  // A product whose 256 x 256 tiles would leave three quarters of the workers
  // idle takes 128 x 128 tiles on the register-staged path: four times the
  // tiles, at most one round (512^3: 16 tiles instead of 4).  Each output is
  // the same MFMA chain either way, so the bits do not change.
  if (small_tiles && ((int64_t)(M + BMr - 1) / BMr) * ((N + BNr - 1) / BNr) * 4 <= total) {
    P->bm = 128;
    P->bn = 128;
  }
  P->tiles_m = (M + P->bm - 1) / P->bm;
  P->tiles_n = (N + P->bn - 1) / P->bn;
  P->grid = mapping == ASYM_MAP_AWARE ? t->n_xccs * smax : total;
  // The aware grid deals smax workgroups to every XCD.  Where an XCD has fewer
  // CUs in the stream's set, the surplus there waits for a CU and holds up the
  // dispatch behind it, so the static assignment (which needs every worker to
  // run) gives way to claims.
  P->dynamic = false;
  for (int x = 0; x < t->n_xccs; ++x)
    if (per[x] < smax) P->dynamic = true;
  // A whole-XCD restriction also takes claims: the static form's workers of
  // XCD x are the workgroups with block index x mod n, which the hardware
  // deals to one XCD but not always to XCD x (the XCD that dealing starts on
  // differs between streams), so the static form could run the work on an
  // XCD outside the set; claims read XCC_ID.
  if (!cs.whole) P->dynamic = true;
  P->whole = cs.whole;
  P->per = std::move(per);
  P->slots = std::move(slots);
  P->small_mb = small_m_for(*P, M, (long long)((M + 63) / 64) * ((N + small_m_tile_cols() - 1) / small_m_tile_cols()));
  return ASYM_OK;
}

// The small-M launch a plan asks for (everything but the partials buffer of
// a split K, which the caller provides).
static SmallMLaunch small_m_launch(const GemmPlan& P, const void* A, const void* B, void* C, int M, int N, int K,
                                   int lda, int ldb, int ldc, int mapping) {
  SmallMLaunch sm;
  sm.A = A; sm.B = B; sm.C = C;
  sm.M = M; sm.N = N; sm.K = K; sm.lda = lda; sm.ldb = ldb; sm.ldc = ldc;
  sm.mb = P.small_mb;
  sm.row_tiles = (M + 16 * P.small_mb - 1) / (16 * P.small_mb);
  sm.order = small_m_order(mapping);
  sm.n_x = P.t->n_xccs;
  sm.ksplit = small_m_ksplit(M, N, K, P.small_mb, P.t->n_cus);
  sm.tile_cols = small_m_cols(N, P.small_mb, sm.row_tiles, sm.ksplit, P.t->n_cus);
  const int tiles_n = (N + sm.tile_cols - 1) / sm.tile_cols;
  sm.grid = small_m_grid(sm.row_tiles, tiles_n, sm.order, sm.n_x);
  if (sm.ksplit > 1) sm.grid = (long long)tiles_n * sm.ksplit;
  return sm;
}

// fp32 partial tiles of a split K: [column tiles][ranges][16 mb rows][64 columns]
static size_t small_m_part_bytes(const SmallMLaunch& sm) {
  const int tiles_n = (sm.N + small_m_tile_cols() - 1) / small_m_tile_cols();
  return (size_t)tiles_n * sm.ksplit * 16 * sm.mb * 64 * sizeof(float);
}

static int gemm_bf16_locked(const asym_topology* topo_in, int M, int N, int K, const void* A, int lda,
                            const void* B, int ldb, int b_layout, void* C, int ldc, int mapping,
                            uint32_t xcd_mask, hipStream_t stream);

int gemm_bf16(const asym_topology* topo_in, int M, int N, int K, const void* A, int lda,
              const void* B, int ldb, int b_layout, void* C, int ldc, int mapping,
              uint32_t xcd_mask, hipStream_t stream) {
  std::lock_guard<std::mutex> lock(g_mu);
  if (b_layout != ASYM_B_KN)
    return gemm_bf16_locked(topo_in, M, N, K, A, lda, B, ldb, b_layout, C, ldc, mapping, xcd_mask, stream);
  // [K][N] storage: check everything first, then transpose B into the
  // stream's buffer (an exact copy) and run the [N][K] path on it
  GemmPlan P;
  int rc = plan_gemm(topo_in, M, N, K, A, lda, B, ldb, b_layout, C, ldc, mapping, xcd_mask, stream, &P);
  if (rc != ASYM_OK) return rc;
  Workspace* ws = nullptr;
  rc = get_workspace(P.device, stream, &ws);
  if (rc != ASYM_OK) return rc;
  const int ldt = kn_pitch(K);
  const size_t need = (size_t)N * ldt * sizeof(uint16_t);
  if (ws->kn_bytes < need) {
    // a buffer in use by launches on this stream is freed after they finish
    ASYM_HIP(hipStreamSynchronize(stream));
    if (ws->kn_buf) ASYM_HIP(hipFree(ws->kn_buf));
    ws->kn_buf = nullptr;
    ws->kn_bytes = 0;
    ASYM_HIP(hipMalloc(&ws->kn_buf, need));
    ws->kn_bytes = need;
  }
  rc = launch_transpose_bf16(B, K, N, ldb, ws->kn_buf, ldt, stream);
  if (rc != ASYM_OK) return rc;
  return gemm_bf16_locked(topo_in, M, N, K, A, lda, ws->kn_buf, ldt, ASYM_B_NK, C, ldc, mapping, xcd_mask,
                          stream);
}

static int gemm_bf16_locked(const asym_topology* topo_in, int M, int N, int K, const void* A, int lda,
                            const void* B, int ldb, int b_layout, void* C, int ldc, int mapping,
                            uint32_t xcd_mask, hipStream_t stream) {
  GemmPlan P;
  int rc = plan_gemm(topo_in, M, N, K, A, lda, B, ldb, b_layout, C, ldc, mapping, xcd_mask, stream, &P);
  if (rc != ASYM_OK) return rc;
  if (P.small_mb) {
    SmallMLaunch sm = small_m_launch(P, A, B, C, M, N, K, lda, ldb, ldc, mapping);
    if (sm.ksplit > 1) {
      Workspace* ws = nullptr;
      rc = get_workspace(P.device, stream, &ws);
      if (rc != ASYM_OK) return rc;
      const size_t part_bytes = small_m_part_bytes(sm);
      if (ws->sm_part_bytes < part_bytes) {
        // a buffer in use by launches on this stream is freed after they finish
        ASYM_HIP(hipStreamSynchronize(stream));
        if (ws->sm_part) ASYM_HIP(hipFree(ws->sm_part));
        ws->sm_part = nullptr;
        ws->sm_part_bytes = 0;
        const size_t pb = std::max<size_t>(part_bytes, 4 << 20);
        ASYM_HIP(hipMalloc(&ws->sm_part, pb));
        ws->sm_part_bytes = pb;
      }
      sm.part = ws->sm_part;
    }
    return launch_gemm_small_m(sm, stream);
  }
  const DeviceSchedule* ds = nullptr;
  rc = upload_schedule(P.device, P.tiles_m, P.tiles_n, mapping, P.slots, stream, &ds);
  if (rc != ASYM_OK) return rc;
  Workspace* ws = nullptr;
  rc = get_workspace(P.device, stream, &ws);
  if (rc != ASYM_OK) return rc;

  GemmLaunch g;
  g.A = A; g.B = B; g.C = C;
  g.M = M; g.N = N; g.K = K; g.lda = lda; g.ldb = ldb; g.ldc = ldc;
  g.mapping = mapping;
  g.d_order = ds->d_order; g.d_off = ds->d_off; g.d_slots = ds->d_slots;
  g.tiles_m = P.tiles_m; g.tiles_n = P.tiles_n;
  g.n_xccs = P.t->n_xccs;
  g.grid = P.grid;
  g.d_ctr = ws->gemm_ctr;
  g.dynamic = P.dynamic;
  g.vec = P.vec;
  g.bn = P.bn;
  g.bm = P.bm;
  return launch_gemm(g, stream);
}

// ---- the GEMM without allocation: every buffer in the caller's scratch ------
// Which schedule each device's scratch area holds (written by the last call
// that needed a different one); guarded by g_mu.
std::map<int, ScheduleKey> g_scratch_schedule;

int gemm_noalloc_check(const asym_topology* topo_in, int M, int N, int b_layout) {
  if (!topo_in)
    return fail(ASYM_EINVAL, "gemm (no allocation): needs a probed topology (a first-use probe would allocate)");
  if (b_layout == ASYM_B_KN)
    return fail(ASYM_EUNSUPPORTED, "gemm (no allocation): B stored [K][N] needs a transposed copy; store B as [N][K]");
  // every tile width is at most 256, so this bound holds before the plan picks one
  if (M >= 1 && N >= 1 && (int64_t)((M + 255) / 256) * ((N + 255) / 256) > kScratchMaxTiles)
    return fail(ASYM_EINVAL, "gemm (no allocation): more than " + std::to_string(kScratchMaxTiles) +
                                 " output tiles; the scratch area holds no larger schedule");
  return ASYM_OK;
}

int gemm_bf16_scratch(const asym_topology* topo_in, int M, int N, int K, const void* A, int lda, const void* B,
                      int ldb, int b_layout, void* C, int ldc, int mapping, uint32_t xcd_mask,
                      hipStream_t stream, unsigned char* scratch, size_t bytes) {
  int rc = gemm_noalloc_check(topo_in, M, N, b_layout);
  if (rc != ASYM_OK) return rc;
  if (!scratch || bytes < kScratchBytes) return fail(ASYM_EINVAL, "gemm (no allocation): scratch area too small");
  std::lock_guard<std::mutex> lock(g_mu);
  GemmPlan P;
  rc = plan_gemm(topo_in, M, N, K, A, lda, B, ldb, b_layout, C, ldc, mapping, xcd_mask, stream, &P);
  if (rc != ASYM_OK) return rc;
  if (P.small_mb) {
    SmallMLaunch sm = small_m_launch(P, A, B, C, M, N, K, lda, ldb, ldc, mapping);
    if (sm.ksplit > 1) {
      if (small_m_part_bytes(sm) > kScratchPartBytes)
        return fail(ASYM_EINVAL, "gemm (no allocation): split-K partials exceed the scratch area");
      sm.part = reinterpret_cast<float*>(scratch + kScratchPartOff);
    }
    return launch_gemm_small_m(sm, stream);
  }
  const int64_t T = (int64_t)P.tiles_m * P.tiles_n;
  if (T > kScratchMaxTiles)
    return fail(ASYM_EINVAL, "gemm (no allocation): more than " + std::to_string(kScratchMaxTiles) +
                                 " output tiles; the scratch area holds no larger schedule");
  int* d_ctr = reinterpret_cast<int*>(scratch + kScratchCtrOff);
  int* d_off = reinterpret_cast<int*>(scratch + kScratchOffOff);
  int* d_slots = reinterpret_cast<int*>(scratch + kScratchSlotsOff);
  int* d_order = reinterpret_cast<int*>(scratch + kScratchOrderOff);
  ScheduleKey key{P.device, P.tiles_m, P.tiles_n, mapping, P.slots};
  auto it = g_scratch_schedule.find(P.device);
  if (it == g_scratch_schedule.end() || it->second < key || key < it->second) {
    if (it != g_scratch_schedule.end()) g_scratch_schedule.erase(it);
    Schedule sch;
    rc = build_schedule(P.tiles_m, P.tiles_n, (int)P.slots.size(), P.slots.data(), mapping, 0, sch);
    if (rc != ASYM_OK) return rc;
    std::vector<int> off(ASYM_MAX_XCDS + 1, sch.off.back()), sl(ASYM_MAX_XCDS, 0);
    for (size_t x = 0; x < sch.off.size(); ++x) off[x] = sch.off[x];
    for (size_t x = 0; x < P.slots.size(); ++x) sl[x] = P.slots[x];
    rc = launch_put_words(d_off, off.data(), off.size(), stream);
    if (rc == ASYM_OK) rc = launch_put_words(d_slots, sl.data(), sl.size(), stream);
    if (rc == ASYM_OK) rc = launch_put_words(d_order, sch.order.data(), sch.order.size(), stream);
    if (rc != ASYM_OK) return rc;
    g_scratch_schedule[P.device] = key;
  }
  // the claiming form needs its counters at zero (its last workgroup leaves
  // them so, but the area keeps whatever the last call on it left)
  if (mapping == ASYM_MAP_AWARE && P.dynamic) {
    rc = launch_zero_words(d_ctr, 64, stream);
    if (rc != ASYM_OK) return rc;
  }
  GemmLaunch g;
  g.A = A; g.B = B; g.C = C;
  g.M = M; g.N = N; g.K = K; g.lda = lda; g.ldb = ldb; g.ldc = ldc;
  g.mapping = mapping;
  g.d_order = d_order; g.d_off = d_off; g.d_slots = d_slots;
  g.tiles_m = P.tiles_m; g.tiles_n = P.tiles_n;
  g.n_xccs = P.t->n_xccs;
  g.grid = P.grid;
  g.d_ctr = d_ctr;
  g.dynamic = P.dynamic;
  g.vec = P.vec;
  g.bn = P.bn;
  g.bm = P.bm;
  return launch_gemm(g, stream);
}

static_assert(sizeof(asym_wg_record) == 48, "the trace record layout is part of the ABI");

int gemm_bf16_trace(const asym_topology* topo_in, int M, int N, int K, const void* A, int lda, const void* B,
                    int ldb, int b_layout, void* C, int ldc, int mapping, uint32_t xcd_mask, hipStream_t stream,
                    asym_wg_record* records, int capacity, int* n_records) {
  if (!records || !n_records) return fail(ASYM_EINVAL, "gemm trace: null records");
  if (b_layout == ASYM_B_KN) return fail(ASYM_EUNSUPPORTED, "gemm trace: B stored [K][N] is not traced");
  std::lock_guard<std::mutex> lock(g_mu);
  const bool prev = g_small_m.exchange(false);  // the persistent kernel, whatever the shape
  GemmPlan P;
  int rc = plan_gemm(topo_in, M, N, K, A, lda, B, ldb, b_layout, C, ldc, mapping, xcd_mask, stream, &P);
  g_small_m.store(prev);
  if (rc != ASYM_OK) return rc;
  if (capacity < P.grid) return fail(ASYM_EINVAL, "gemm trace: capacity below the grid (" + std::to_string(P.grid) + ")");
  const DeviceSchedule* ds = nullptr;
  rc = upload_schedule(P.device, P.tiles_m, P.tiles_n, mapping, P.slots, stream, &ds);
  if (rc != ASYM_OK) return rc;
  Workspace* ws = nullptr;
  rc = get_workspace(P.device, stream, &ws);
  if (rc != ASYM_OK) return rc;
  GemmLaunch g;
  g.A = A; g.B = B; g.C = C;
  g.M = M; g.N = N; g.K = K; g.lda = lda; g.ldb = ldb; g.ldc = ldc;
  g.mapping = mapping;
  g.d_order = ds->d_order; g.d_off = ds->d_off; g.d_slots = ds->d_slots;
  g.tiles_m = P.tiles_m; g.tiles_n = P.tiles_n;
  g.n_xccs = P.t->n_xccs;
  g.grid = P.grid;
  g.d_ctr = ws->gemm_ctr;
  g.dynamic = P.dynamic;
  g.vec = P.vec;
  g.bn = P.bn;
  g.bm = P.bm;
  g.d_trace = records;
  *n_records = P.grid;
  return launch_gemm(g, stream);
}

int gemm_grouped_bf16(const asym_topology* topo_in, int G, const int* Ms, int N, int K, const void* A,
                      int lda, const void* B, int ldb, void* C, int ldc, int mapping, uint32_t xcd_mask,
                      hipStream_t stream) {
  if (G < 1) return fail(ASYM_EINVAL, "grouped gemm: G must be >= 1");
  if (!Ms) return fail(ASYM_EINVAL, "grouped gemm: null row counts");
  int64_t rows = 0;
  for (int g = 0; g < G; ++g) {
    if (Ms[g] < 0) return fail(ASYM_EINVAL, "grouped gemm: negative row count");
    rows += Ms[g];
  }
  if (rows > (1ll << 30)) return fail(ASYM_EINVAL, "grouped gemm: too many rows");
  if ((int64_t)G * N > (1ll << 31) - 1) return fail(ASYM_EINVAL, "grouped gemm: G * N too large");
  std::vector<int> tm(G);
  int64_t trows = 0;
  for (int g = 0; g < G; ++g) {
    tm[g] = (Ms[g] + gemm_tile_m() - 1) / gemm_tile_m();
    trows += tm[g];
  }
  if (rows == 0) {
    // nothing to compute; A and C may be empty (null) buffers
    if (N < 1 || K < 1) return fail(ASYM_EINVAL, "grouped gemm: N, K must be >= 1");
    if (!B) return fail(ASYM_EINVAL, "grouped gemm: null weights");
    if (mapping != ASYM_MAP_AWARE && mapping != ASYM_MAP_OBLIVIOUS_GROUPED &&
        mapping != ASYM_MAP_OBLIVIOUS_ROWMAJOR)
      return fail(ASYM_EINVAL, "grouped gemm: unknown mapping");
    return ASYM_OK;
  }
  std::lock_guard<std::mutex> lock(g_mu);
  // the checks, CU set, path and tile width of a GEMM with as many tile rows
  // (the weights: G * N rows of B)
  GemmPlan P;
  const int virt_m = (int)std::max<int64_t>(1, trows * gemm_tile_m());
  int rc = plan_gemm(topo_in, virt_m, N, K, A, lda, B, ldb, ASYM_B_NK, C, ldc, mapping, xcd_mask, stream, &P,
                     false);
  if (rc != ASYM_OK) return rc;
  const int max_rows = *std::max_element(Ms, Ms + G);
  long long wgs64 = 0;
  for (int g = 0; g < G; ++g) wgs64 += (long long)((Ms[g] + 63) / 64) * ((N + small_m_tile_cols() - 1) / small_m_tile_cols());
  const int small_mb = small_m_for(P, max_rows, wgs64);
  // the small-M path's column-tile width, by the rule of a plain product over
  // all the groups' row tiles
  int small_w = small_m_tile_cols();
  if (small_mb) {
    long long rts = 0;
    for (int g = 0; g < G; ++g) rts += (Ms[g] + 16 * small_mb - 1) / (16 * small_mb);
    small_w = small_m_cols(N, small_mb, (int)std::min<long long>(rts, 1 << 30), 1, P.t->n_cus);
  }
  const int tiles_n = small_mb ? (N + small_w - 1) / small_w : (N + P.bn - 1) / P.bn;
  Workspace* ws = nullptr;
  rc = get_workspace(P.device, stream, &ws);
  if (rc != ASYM_OK) return rc;
  std::vector<int> key(Ms, Ms + G);
  key.push_back(N);
  key.push_back(small_mb ? -small_mb : P.bn);
  key.push_back(small_mb ? small_w : 0);
  key.push_back(mapping);
  key.insert(key.end(), P.slots.begin(), P.slots.end());
  auto hit = std::find_if(ws->g_tables.begin(), ws->g_tables.end(),
                          [&](const GroupedTables& t) { return t.key == key; });
  if (hit != ws->g_tables.end()) {
    std::rotate(ws->g_tables.begin(), hit, hit + 1);  // most recent first
  } else {
    Schedule sch;
    std::vector<int4> small_desc;
    if (small_mb) {
      // one workgroup per (group, row tile, column tile), in the mapping's
      // order; the aware order runs a column's row tiles one after another on
      // one XCD (each group's run padded to a multiple of the XCD count with
      // empty entries, so the XCD of an entry is its column mod n)
      const int n_x = P.t->n_xccs;
      const int tr = 16 * small_mb;
      const int order = small_m_order(mapping);
      int row0 = 0;
      for (int g = 0; g < G; ++g) {
        const int R = (Ms[g] + tr - 1) / tr;
        auto put = [&](int r, int c) {
          if (c >= tiles_n) {
            small_desc.push_back(int4{0, 0, 0, 0});
            return;
          }
          small_desc.push_back(int4{row0 + r * tr, std::min(tr, Ms[g] - r * tr), g * N, c * small_w});
        };
        if (R > 0) {
          if (order == 0) {
            for (int cb = 0; cb < (tiles_n + n_x - 1) / n_x; ++cb)
              for (int r = 0; r < R; ++r)
                for (int j = 0; j < n_x; ++j) put(r, cb * n_x + j);
          } else if (order == 1) {
            for (int c = 0; c < tiles_n; ++c)
              for (int r = 0; r < R; ++r) put(r, c);
          } else {
            for (int r = 0; r < R; ++r)
              for (int c = 0; c < tiles_n; ++c) put(r, c);
          }
        }
        row0 += Ms[g];
      }
      for (size_t i = 0; i < small_desc.size(); ++i) sch.order.push_back((int)i);
      sch.off.assign(P.t->n_xccs + 1, 0);
    } else {
      rc = build_grouped_schedule(G, tm.data(), tiles_n, P.t->n_xccs, P.slots.data(), mapping, sch);
      if (rc != ASYM_OK) return rc;
    }
    GroupedTables tb;
    tb.key = std::move(key);
    tb.T = (int)sch.order.size();
    const size_t desc_bytes = (size_t)tb.T * sizeof(int4);
    const size_t sched_bytes = ((size_t)tb.T + 2 * ASYM_MAX_XCDS + 1) * sizeof(int);
    if (ws->g_tables.size() >= kGroupedCache) {
      // the oldest tables may still be read by launches on this stream
      ASYM_HIP(hipStreamSynchronize(stream));
      GroupedTables& old = ws->g_tables.back();
      ASYM_HIP(hipFree(old.desc));
      ASYM_HIP(hipFree(old.sched));
      ws->g_tables.pop_back();
    }
    ASYM_HIP(hipMalloc(&tb.desc, desc_bytes));
    ASYM_HIP(hipMalloc(&tb.sched, sched_bytes));
    // the staging buffer is free once the previous upload's copies have run
    if (ws->g_pending) {
      ASYM_HIP(hipEventSynchronize(ws->g_copied));
      ws->g_pending = false;
    }
    if (ws->g_host_bytes < desc_bytes + sched_bytes) {
      if (ws->g_host) ASYM_HIP(hipHostFree(ws->g_host));
      ws->g_host = nullptr;
      ws->g_host_bytes = 0;
      const size_t bytes = std::max<size_t>(desc_bytes + sched_bytes, 64 << 10);
      ASYM_HIP(hipHostMalloc(&ws->g_host, bytes));
      ws->g_host_bytes = bytes;
    }
    if (!ws->g_copied) ASYM_HIP(hipEventCreateWithFlags(&ws->g_copied, hipEventDisableTiming));
    int4* h_desc = static_cast<int4*>(ws->g_host);
    int* h_sched = reinterpret_cast<int*>(static_cast<char*>(ws->g_host) + desc_bytes);
    if (small_mb) {
      std::copy(small_desc.begin(), small_desc.end(), h_desc);
    } else {
      int id = 0, row0 = 0;
      for (int g = 0; g < G; ++g) {
        for (int r = 0; r < tm[g]; ++r)
          for (int c = 0; c < tiles_n; ++c)
            h_desc[id++] = int4{row0 + r * gemm_tile_m(), std::min(gemm_tile_m(), Ms[g] - r * gemm_tile_m()),
                                g * N, c * P.bn};
        row0 += Ms[g];
      }
    }
    std::fill(h_sched, h_sched + sched_bytes / sizeof(int), 0);
    std::copy(sch.order.begin(), sch.order.end(), h_sched);
    for (int x = 0; x <= P.t->n_xccs; ++x) h_sched[tb.T + x] = sch.off[x];
    for (int x = 0; x < P.t->n_xccs; ++x) h_sched[tb.T + ASYM_MAX_XCDS + 1 + x] = P.slots[x];
    ASYM_HIP(hipMemcpyAsync(tb.desc, h_desc, desc_bytes, hipMemcpyHostToDevice, stream));
    ASYM_HIP(hipMemcpyAsync(tb.sched, h_sched, sched_bytes, hipMemcpyHostToDevice, stream));
    ASYM_HIP(hipEventRecord(ws->g_copied, stream));
    ws->g_pending = true;
    ws->g_tables.insert(ws->g_tables.begin(), std::move(tb));
  }
  const GroupedTables& tb = ws->g_tables.front();
  const int T = tb.T;
  if (small_mb) {
    SmallMLaunch sm;
    sm.A = A; sm.B = B; sm.C = C;
    sm.M = (int)rows; sm.N = N; sm.K = K; sm.lda = lda; sm.ldb = ldb; sm.ldc = ldc;
    sm.mb = small_mb;
    sm.n_x = P.t->n_xccs;
    sm.grid = T;
    sm.d_desc = tb.desc;
    sm.tile_cols = small_w;
    return launch_gemm_small_m(sm, stream);
  }

  GemmLaunch gl;
  gl.A = A; gl.B = B; gl.C = C;
  gl.M = virt_m; gl.N = N; gl.K = K; gl.lda = lda; gl.ldb = ldb; gl.ldc = ldc;
  gl.mapping = mapping;
  gl.d_order = tb.sched;
  gl.d_off = tb.sched + T;
  gl.d_slots = tb.sched + T + ASYM_MAX_XCDS + 1;
  gl.tiles_m = (int)trows;
  gl.tiles_n = tiles_n;
  gl.n_xccs = P.t->n_xccs;
  gl.grid = P.grid;
  gl.d_ctr = ws->gemm_ctr;
  gl.dynamic = P.dynamic;
  gl.vec = P.vec;
  gl.bn = P.bn;
  gl.d_desc = tb.desc;
  return launch_gemm(gl, stream);
}

// ---- decode attention -------------------------------------------------------
struct AttnPlan {
  CuSet cs;
  int split = 0, n_splits = 0, tasks = 0, grid = 0;
  std::vector<int> quota;  // aware: tasks per XCD
  size_t ws_bytes = 0;
  bool dense_static = false;  // aware: a dense call deals its tasks statically (below)
};

static int attn_plan(const asym_topology* topo_in, int B, int Hq, int Hkv, int S, int D, int split_in,
                     int mapping, uint32_t xcd_mask, hipStream_t stream, AttnPlan* P) {
  if (B < 1 || Hq < 1 || Hkv < 1 || S < 1) return fail(ASYM_EINVAL, "attention: B, H_q, H_kv, S_k must be >= 1");
  if (Hq % Hkv) return fail(ASYM_EINVAL, "attention: H_kv must divide H_q");
  const int G = Hq / Hkv;
  if (G != 1 && G != 2 && G != 4 && G != 8 && G != 16)
    return fail(ASYM_EUNSUPPORTED, "attention: query heads per key/value head must be 1, 2, 4, 8 or 16");
  if (D != 128) return fail(ASYM_EUNSUPPORTED, "attention: the head dimension must be 128");
  if (S >= (1 << 24)) return fail(ASYM_EUNSUPPORTED, "attention: S_k of 2^24 or more (32-bit offsets into a head's keys)");
  if (split_in < 0 || split_in % 16 || split_in > (1 << 20))
    return fail(ASYM_EINVAL, "attention: split_tokens must be 0 (automatic) or a positive multiple of 16");
  if (mapping != ASYM_MAP_AWARE && mapping != ASYM_MAP_OBLIVIOUS_GROUPED && mapping != ASYM_MAP_OBLIVIOUS_ROWMAJOR)
    return fail(ASYM_EINVAL, "attention: unknown mapping");
  int rc = cu_set_for(topo_in, mapping, xcd_mask, stream, "attention", &P->cs);
  if (rc != ASYM_OK) return rc;
  const int64_t heads = (int64_t)B * Hkv;
  int L = split_in;
  if (!L) {
    // the longest split (up to 1024 tokens) that still gives 2048 tasks
    L = 1024;
    while (L > 64 && heads * ((S + L - 1) / L) < 2048) L /= 2;
  }
  const int64_t n_splits = (S + L - 1) / L;
  const int64_t tasks = heads * n_splits;
  if (tasks > (1ll << 30)) return fail(ASYM_EINVAL, "attention: too many tasks");
  P->split = L;
  P->n_splits = (int)n_splits;
  P->tasks = (int)tasks;
  const int per_wg = attn_tasks_per_workgroup();
  const int n_x = P->cs.t->n_xccs;
  if (mapping == ASYM_MAP_AWARE) {
    P->quota = largest_remainder_quotas(P->tasks, P->cs.slots);
    // claiming workgroups loop until every share is taken: two per CU of the
    // largest XCD on every XCD (the dealing is equal per XCD), but no more
    // than the groups of the largest share
    int most = 0;
    for (int x = 0; x < n_x; ++x) most = std::max(most, (P->quota[x] + per_wg - 1) / per_wg);
    P->grid = std::max(1, std::min(most, 2 * P->cs.smax) * n_x);
    // On a set with equal CUs per XCD, every claiming workgroup holding one
    // group at most and short tasks (at most 128 tokens), the claims can move
    // no work and their round trips are a large part of each task: a dense
    // call then deals its groups as the oblivious grid does (round-robin over
    // the XCDs: equal shares, the proportional ones on this set).  Measured on
    // the full chip, claiming: GQA B=16 S=1024 25.3 against 20.3 us, B=1
    // S=8192 16.6 against 13.7; with longer tasks the claims balance the tail
    // (B=16 S=8192, 512-token splits: 1.03-1.16x the round-robin).  Paged
    // calls always claim: their pages are placed by the physical XCD of each
    // share.
    bool uniform = P->cs.whole;
    for (int x = 0; x < n_x; ++x) uniform = uniform && P->cs.slots[x] == P->cs.smax && P->cs.smax > 0;
    P->dense_static = uniform && most <= 2 * P->cs.smax && L <= 128;
  } else {
    P->grid = (P->tasks + per_wg - 1) / per_wg;
  }
  P->ws_bytes = (size_t)B * Hq * n_splits * (128 + 2) * sizeof(float);
  return ASYM_OK;
}

// The aware attention forms' per-XCD task offsets on the device (cached per
// stream by CU counts, task count and kernel) and the claim counters, zeroed
// at creation (every aware launch's merge leaves them zero again).
static int aware_share_offsets(Workspace* ws, const CuSet& cs, const std::vector<int>& quota, int tasks, int kind,
                               hipStream_t stream, int** d_off_out) {
  const int n_x = cs.t->n_xccs;
  std::vector<int> key(cs.slots);
  key.push_back(tasks);
  key.push_back(kind);
  auto hit = std::find_if(ws->attn_off.begin(), ws->attn_off.end(),
                          [&](const std::pair<std::vector<int>, int*>& e) { return e.first == key; });
  if (hit != ws->attn_off.end()) {
    std::rotate(ws->attn_off.begin(), hit, hit + 1);
  } else {
    if (ws->attn_off.size() >= 8) {
      ASYM_HIP(hipStreamSynchronize(stream));
      ASYM_HIP(hipFree(ws->attn_off.back().second));
      ws->attn_off.pop_back();
    }
    int* dev_off = nullptr;
    ASYM_HIP(hipMalloc(&dev_off, (ASYM_MAX_XCDS + 1) * sizeof(int)));
    if (ws->g_pending) {
      ASYM_HIP(hipEventSynchronize(ws->g_copied));
      ws->g_pending = false;
    }
    if (ws->g_host_bytes < (ASYM_MAX_XCDS + 1) * sizeof(int)) {
      if (ws->g_host) ASYM_HIP(hipHostFree(ws->g_host));
      ws->g_host = nullptr;
      ws->g_host_bytes = 0;
      ASYM_HIP(hipHostMalloc(&ws->g_host, 64 << 10));
      ws->g_host_bytes = 64 << 10;
    }
    if (!ws->g_copied) ASYM_HIP(hipEventCreateWithFlags(&ws->g_copied, hipEventDisableTiming));
    int* h = static_cast<int*>(ws->g_host);
    h[0] = 0;
    for (int x = 0; x < n_x; ++x) h[x + 1] = h[x] + quota[x];
    ASYM_HIP(hipMemcpyAsync(dev_off, h, (n_x + 1) * sizeof(int), hipMemcpyHostToDevice, stream));
    ASYM_HIP(hipEventRecord(ws->g_copied, stream));
    ws->g_pending = true;
    ws->attn_off.insert(ws->attn_off.begin(), std::make_pair(std::move(key), dev_off));
  }
  *d_off_out = ws->attn_off.front().second;
  if (!ws->attn_claim) {
    ASYM_HIP(hipMalloc(&ws->attn_claim, attn_claim_ints() * sizeof(int)));
    int rc = launch_zero_words(ws->attn_claim, attn_claim_ints(), stream);
    if (rc != ASYM_OK) return rc;
  }
  return ASYM_OK;
}

// fp32 partials of the attention forms in the stream's buffer (grown after a
// stream synchronisation: the old buffer may still be read by launches on it)
static int attn_partials(Workspace* ws, size_t bytes_needed, hipStream_t stream) {
  if (ws->attn_bytes >= bytes_needed) return ASYM_OK;
  ASYM_HIP(hipStreamSynchronize(stream));
  if (ws->attn_buf) ASYM_HIP(hipFree(ws->attn_buf));
  ws->attn_buf = nullptr;
  ws->attn_bytes = 0;
  const size_t bytes = std::max<size_t>(bytes_needed, 1 << 20);
  ASYM_HIP(hipMalloc(&ws->attn_buf, bytes));
  ws->attn_bytes = bytes;
  return ASYM_OK;
}

int attn_decode(const asym_topology* topo_in, int B, int Hq, int Hkv, int S, int D, const void* q, const void* k,
                const void* v, void* o, float* lse, float scale, int split_in, int mapping, uint32_t xcd_mask,
                hipStream_t stream, const int* k_pages = nullptr, const int* v_pages = nullptr,
                size_t pool_pages = 0) {
  if (!q || !k || !v || !o) return fail(ASYM_EINVAL, "attention: null pointer");
  const bool paged = k_pages || v_pages;
  if (paged) {
    if (!k_pages || !v_pages) return fail(ASYM_EINVAL, "paged attention: null page table");
    if (((uintptr_t)k_pages & 3u) || ((uintptr_t)v_pages & 3u))
      return fail(ASYM_EINVAL, "paged attention: page tables must be 4-byte aligned");
    const size_t page_bytes = (size_t)attn_page_tokens() * 128 * 2;
    if (pool_pages < 1 || pool_pages > ((size_t)1 << 31) / page_bytes)
      return fail(ASYM_EINVAL, "paged attention: pool_pages must be in [1, 2 GiB / 8 KiB]");
    if (split_in > 64 * attn_page_tokens())
      return fail(ASYM_EINVAL, "paged attention: split_tokens must be at most 2048");
  }
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || ((uintptr_t)o & 3u) || ((uintptr_t)lse & 3u))
    return fail(ASYM_EINVAL, "attention: q, K, V must be 16-byte aligned, O and lse 4-byte aligned");
  if (!std::isfinite(scale)) return fail(ASYM_EINVAL, "attention: scale must be finite");
  std::lock_guard<std::mutex> lock(g_mu);
  AttnPlan P;
  int rc = attn_plan(topo_in, B, Hq, Hkv, S, D, split_in, mapping, xcd_mask, stream, &P);
  if (rc != ASYM_OK) return rc;
  Workspace* ws = nullptr;
  rc = get_workspace(P.cs.device, stream, &ws);
  if (rc != ASYM_OK) return rc;
  rc = attn_partials(ws, P.ws_bytes, stream);
  if (rc != ASYM_OK) return rc;
  const int n_x = P.cs.t->n_xccs;
  int* d_off = nullptr;
  const bool claims = mapping == ASYM_MAP_AWARE && (paged || !P.dense_static);
  if (claims) {
    rc = aware_share_offsets(ws, P.cs, P.quota, P.tasks, 0, stream, &d_off);
    if (rc != ASYM_OK) return rc;
  } else if (mapping == ASYM_MAP_AWARE) {
    P.grid = (P.tasks + attn_tasks_per_workgroup() - 1) / attn_tasks_per_workgroup();
  }
  AttnLaunch a;
  a.q = q; a.k = k; a.v = v; a.o = o; a.lse = lse;
  a.part_o = ws->attn_buf;
  a.part_ml = ws->attn_buf + (size_t)B * Hq * P.n_splits * 128;
  a.d_quota_off = d_off;
  a.d_claim = ws->attn_claim;
  a.allow = 0;
  for (int x = 0; x < n_x; ++x)
    if (P.cs.slots[x] > 0) a.allow |= 1u << x;
  a.B = B; a.Hq = Hq; a.Hkv = Hkv; a.S = S;
  a.split = P.split; a.n_splits = P.n_splits;
  a.n_x = n_x; a.grid = P.grid;
  a.scale = scale;
  if (paged) {
    a.k_page = k_pages;
    a.v_page = v_pages;
    a.pool_bytes = (uint32_t)(pool_pages * (size_t)attn_page_tokens() * 128 * 2);
  }
  return launch_attn_decode(a, stream);
}

int attn_decode_plan(const asym_topology* topo_in, int B, int Hq, int Hkv, int S, int D, int split_in,
                     int mapping, uint32_t xcd_mask, hipStream_t stream, asym_attn_plan_info* out) {
  if (!out) return fail(ASYM_EINVAL, "attention plan: null output");
  std::lock_guard<std::mutex> lock(g_mu);
  AttnPlan P;
  const int rc = attn_plan(topo_in, B, Hq, Hkv, S, D, split_in, mapping, xcd_mask, stream, &P);
  if (rc != ASYM_OK) return rc;
  *out = asym_attn_plan_info{};
  out->split_tokens = P.split;
  out->n_splits = P.n_splits;
  out->tasks = P.tasks;
  out->grid = P.grid;
  out->tasks_per_workgroup = attn_tasks_per_workgroup();
  out->n_xcds = P.cs.t->n_xccs;
  out->workspace_bytes = P.ws_bytes;
  out->dense_static = P.dense_static ? 1 : 0;
  const int per_wg = attn_tasks_per_workgroup();
  for (int x = 0; x < out->n_xcds && x < ASYM_MAX_XCDS; ++x) {
    if (mapping == ASYM_MAP_AWARE) {
      out->tasks_per_xcd[x] = P.quota[x];
    } else {
      // workgroup i lands on XCD i mod n and holds tasks per_wg i .. per_wg i + per_wg - 1
      long long c = 0;
      for (int i = x; i < P.grid; i += out->n_xcds) c += std::min(per_wg, P.tasks - i * per_wg);
      out->tasks_per_xcd[x] = (int)c;
    }
  }
  return ASYM_OK;
}

// ---- multi-head latent attention, decode ------------------------------------
static int mla_plan(const asym_topology* topo_in, int B, int Hq, int S, int split_in, int mapping, uint32_t xcd_mask,
                    hipStream_t stream, AttnPlan* P, int* hblocks, int* form_out) {
  if (B < 1 || Hq < 1 || S < 1) return fail(ASYM_EINVAL, "mla: B, H_q, S_k must be >= 1");
  if (Hq % 16) return fail(ASYM_EUNSUPPORTED, "mla: H_q must be a multiple of 16 (blocks of 16 query heads)");
  if (Hq > 1024) return fail(ASYM_EUNSUPPORTED, "mla: at most 1024 query heads");
  if ((int64_t)S * 576 * 2 >= (1ll << 31)) return fail(ASYM_EUNSUPPORTED, "mla: a request's cache must be below 2 GiB");
  if (split_in < 0 || split_in % 32 || split_in > (1 << 20))
    return fail(ASYM_EINVAL, "mla: split_tokens must be 0 (automatic) or a positive multiple of 32");
  if (mapping != ASYM_MAP_AWARE && mapping != ASYM_MAP_OBLIVIOUS_GROUPED && mapping != ASYM_MAP_OBLIVIOUS_ROWMAJOR)
    return fail(ASYM_EINVAL, "mla: unknown mapping");
  int rc = cu_set_for(topo_in, mapping, xcd_mask, stream, "mla", &P->cs);
  if (rc != ASYM_OK) return rc;
  const int hb = Hq / 16;
  int L = split_in;
  if (!L) {
    // the longest split (up to 1024 tokens) that still gives 1024 tasks (a
    // task is one wave over 16 heads), then no more than 256 splits per row:
    // the merge reads every split's 512-value partial, and with few rows and
    // many splits it is bound by latency (measured at one request: 16 heads,
    // 32K tokens, 1024 splits of 32 took 49 us against 39 us with 256)
    L = 1024;
    while (L > 32 && (int64_t)B * hb * ((S + L - 1) / L) < 1024) L /= 2;
    while (L < 1024 && (S + L - 1) / L > 256) L *= 2;
  }
  int64_t n_splits = (S + L - 1) / L;
  // the workgroup forms share each block's rows among 4 or 8 head blocks
  // (one task per workgroup); the wave form runs one head block per wave.
  // The 128-head form does a task's blocks faster, but has half the 64-head
  // form's tasks: it is taken when those tasks fill more than half the CU set
  // (with fewer, the 64-head form finishes in one round of tasks on every CU;
  // measured at one request, 128 heads, 32K tokens: 47.6 against 37.7 us)
  const int allow = g_mla_form.load();
  const int set_cus = P->cs.total;
  int64_t t128 = (int64_t)B * n_splits * (hb / mla_form_head_blocks(2));
  const bool fits128 = hb % mla_form_head_blocks(2) == 0;
  // An automatic split of 1024 tokens or more is halved when that gives the
  // 128-head form more tasks than half the CU set (the rule below then takes
  // it): 512-token splits keep its tasks long enough (measured at 128 heads,
  // B=8, S=16384: 62.4 us against 73.0 in the 64-head form's 1024-token
  // splits; B=32, S=4096: 65.5 against 73.8), shorter ones do not (B=16,
  // S=4096: 49.0 in 256-token splits against 47.3 for the 64-head form's 512).
  if (!split_in && allow == 2 && fits128 && L >= 1024 && 2 * t128 <= set_cus && 4 * t128 > set_cus) {
    L /= 2;
    n_splits = (S + L - 1) / L;
    t128 = (int64_t)B * n_splits * (hb / mla_form_head_blocks(2));
  }
  const int form = allow >= 3 && fits128                         ? 2
                   : allow >= 2 && fits128 && 2 * t128 > set_cus ? 2
                   : allow >= 1 && hb % mla_form_head_blocks(1) == 0 ? 1
                                                                      : 0;
  // a workgroup-form task is 4 or 8 head blocks: with automatic splits, they
  // are lengthened (up to 8192 tokens) while at least two tasks per CU of
  // the set remain.  The fp32 partials shrink with the split count (at B=64,
  // 128 heads, 32K tokens: 537 MB for 32 splits, beyond the memory-side
  // cache, against 134 MB for 8)
  if (form != 0 && !split_in) {
    const int64_t groups = hb / mla_form_head_blocks(form);
    while (L < 8192 && (int64_t)B * ((S + 2 * L - 1) / (2 * L)) * groups >= 2ll * P->cs.total) L *= 2;
    n_splits = (S + L - 1) / L;
  }
  const int64_t tasks = (int64_t)B * n_splits * (hb / mla_form_head_blocks(form));
  if (tasks > (1ll << 30)) return fail(ASYM_EINVAL, "mla: too many tasks");
  P->split = L;
  P->n_splits = (int)n_splits;
  P->tasks = (int)tasks;
  *hblocks = hb;
  *form_out = form;
  const int per_wg = form ? 1 : mla_tasks_per_workgroup();
  const int n_x = P->cs.t->n_xccs;
  if (mapping == ASYM_MAP_AWARE) {
    P->quota = largest_remainder_quotas(P->tasks, P->cs.slots);
    // one 128 KiB workgroup fits per CU: one per CU of the largest XCD on
    // every XCD (the dealing is equal per XCD), no more than the groups of
    // the largest share
    int most = 0;
    for (int x = 0; x < n_x; ++x) most = std::max(most, (P->quota[x] + per_wg - 1) / per_wg);
    P->grid = std::max(1, std::min(most, P->cs.smax) * n_x);
    // On a set with equal CUs on every XCD, with each claiming workgroup
    // holding one group at most, the claims can move no work: every task runs
    // at once, and the head groups of a split that could share its rows
    // through one L2 read a working set the memory-side cache holds (so few
    // tasks mean few requests and short splits).  Such a call deals its tasks
    // as the oblivious grid does.  Measured on the full chip, claiming
    // against dealing: 128 heads, B=64, S=4096 107.6 against 102.5 us; 16
    // heads, B=1, S=32768 37.1 against 35.7; 128 heads (two head groups per
    // split), B=1, S=32768 35.3 against 34.3.
    bool uniform = P->cs.whole;
    for (int x = 0; x < n_x; ++x) uniform = uniform && P->cs.slots[x] == P->cs.smax && P->cs.smax > 0;
    P->dense_static = uniform && most <= P->cs.smax;
  } else {
    P->grid = (P->tasks + per_wg - 1) / per_wg;
  }
  P->ws_bytes = (size_t)B * Hq * n_splits * (512 + 2) * sizeof(float);
  return ASYM_OK;
}

int mla_decode(const asym_topology* topo_in, int B, int Hq, int S, const void* q, const void* kv, void* o, float* lse,
               float scale, int split_in, int mapping, uint32_t xcd_mask, hipStream_t stream) {
  if (!q || !kv || !o) return fail(ASYM_EINVAL, "mla: null pointer");
  if (!aligned16(q) || !aligned16(kv) || !aligned16(o) || ((uintptr_t)lse & 3u))
    return fail(ASYM_EINVAL, "mla: q, the cache and O must be 16-byte aligned, lse 4-byte aligned");
  if (!std::isfinite(scale)) return fail(ASYM_EINVAL, "mla: scale must be finite");
  std::lock_guard<std::mutex> lock(g_mu);
  AttnPlan P;
  int hblocks = 0;
  int form = 0;
  int rc = mla_plan(topo_in, B, Hq, S, split_in, mapping, xcd_mask, stream, &P, &hblocks, &form);
  if (rc != ASYM_OK) return rc;
  Workspace* ws = nullptr;
  rc = get_workspace(P.cs.device, stream, &ws);
  if (rc != ASYM_OK) return rc;
  rc = attn_partials(ws, P.ws_bytes, stream);
  if (rc != ASYM_OK) return rc;
  const int n_x = P.cs.t->n_xccs;
  int* d_off = nullptr;
  if (mapping == ASYM_MAP_AWARE && !P.dense_static) {
    rc = aware_share_offsets(ws, P.cs, P.quota, P.tasks, 1 + form, stream, &d_off);
    if (rc != ASYM_OK) return rc;
  } else if (mapping == ASYM_MAP_AWARE) {
    const int per_wg = form ? 1 : mla_tasks_per_workgroup();
    P.grid = (P.tasks + per_wg - 1) / per_wg;
  }
  MlaLaunch a;
  a.q = q; a.kv = kv; a.o = o; a.lse = lse;
  a.part_o = ws->attn_buf;
  a.part_ml = ws->attn_buf + (size_t)B * Hq * P.n_splits * 512;
  a.d_quota_off = d_off;
  a.d_claim = ws->attn_claim;
  a.allow = 0;
  for (int x = 0; x < n_x; ++x)
    if (P.cs.slots[x] > 0) a.allow |= 1u << x;
  a.B = B; a.Hq = Hq; a.S = S;
  a.split = P.split; a.n_splits = P.n_splits;
  a.n_x = n_x; a.grid = P.grid;
  a.scale = scale;
  a.form = form;
  return launch_mla_decode(a, stream);
}

int mla_decode_plan(const asym_topology* topo_in, int B, int Hq, int S, int split_in, int mapping, uint32_t xcd_mask,
                    hipStream_t stream, asym_mla_plan_info* out) {
  if (!out) return fail(ASYM_EINVAL, "mla plan: null output");
  std::lock_guard<std::mutex> lock(g_mu);
  AttnPlan P;
  int hblocks = 0;
  int form = 0;
  const int rc = mla_plan(topo_in, B, Hq, S, split_in, mapping, xcd_mask, stream, &P, &hblocks, &form);
  if (rc != ASYM_OK) return rc;
  *out = asym_mla_plan_info{};
  out->split_tokens = P.split;
  out->n_splits = P.n_splits;
  out->head_blocks = hblocks;
  out->tasks = P.tasks;
  out->grid = P.grid;
  const int per_wg = form ? 1 : mla_tasks_per_workgroup();
  out->tasks_per_workgroup = per_wg;
  out->n_xcds = P.cs.t->n_xccs;
  out->workgroup_form = form;
  out->workspace_bytes = P.ws_bytes;
  out->static_deal = P.dense_static ? 1 : 0;
  for (int x = 0; x < out->n_xcds && x < ASYM_MAX_XCDS; ++x) {
    if (mapping == ASYM_MAP_AWARE) {
      out->tasks_per_xcd[x] = P.quota[x];
    } else {
      long long c = 0;
      for (int i = x; i < P.grid; i += out->n_xcds) c += std::min(per_wg, P.tasks - i * per_wg);
      out->tasks_per_xcd[x] = (int)c;
    }
  }
  return ASYM_OK;
}

int gemm_plan(const asym_topology* topo_in, int M, int N, int K, const void* A, int lda,
              const void* B, int ldb, int b_layout, const void* C, int ldc, int mapping,
              uint32_t xcd_mask, hipStream_t stream, asym_gemm_plan_info* out) {
  if (!out) return fail(ASYM_EINVAL, "gemm_plan: null output");
  std::lock_guard<std::mutex> lock(g_mu);
  GemmPlan P;
  const int rc = plan_gemm(topo_in, M, N, K, A, lda, B, ldb, b_layout, C, ldc, mapping, xcd_mask, stream, &P);
  if (rc != ASYM_OK) return rc;
  *out = asym_gemm_plan_info{};
  out->n_xcds = P.t->n_xccs;
  out->b_transposed = P.b_transposed ? 1 : 0;
  out->vector_path = P.vec ? 1 : 0;
  if (P.small_mb) {
    out->vector_path = 1;
    out->tile_m = 16 * P.small_mb;
    out->tiles_m = (M + out->tile_m - 1) / out->tile_m;
    out->k_splits = small_m_ksplit(M, N, K, P.small_mb, P.t->n_cus);
    out->tile_n = small_m_cols(N, P.small_mb, out->tiles_m, out->k_splits, P.t->n_cus);
    out->tiles_n = (N + out->tile_n - 1) / out->tile_n;
    out->grid = (int)small_m_grid(out->tiles_m, out->tiles_n, small_m_order(mapping), P.t->n_xccs);
    if (out->k_splits > 1) out->grid = out->tiles_n * out->k_splits;
    out->workers = out->grid;
    out->claims = 0;
    out->small_m = 1;
    return ASYM_OK;
  }
  out->tile_m = P.bm;
  out->tile_n = P.bn;
  out->tiles_m = P.tiles_m;
  out->tiles_n = P.tiles_n;
  out->grid = P.grid;
  out->workers = P.total;
  out->claims = (mapping == ASYM_MAP_AWARE && P.dynamic) ? 1 : 0;
  for (int x = 0; x < P.t->n_xccs && x < ASYM_MAX_XCDS; ++x) out->workers_per_xcd[x] = P.slots[x];
  out->small_m = 0;
  out->k_splits = 1;
  return ASYM_OK;
}

// Drop the workspace of a stream that is about to be destroyed.
void release_workspace(hipStream_t s) {
  std::lock_guard<std::mutex> lock(g_mu);
  for (auto it = g_ws.begin(); it != g_ws.end();) {
    if (it->first.second == s) {
      (void)hipFree(it->second.gemm_ctr);
      if (it->second.attn_buf) (void)hipFree(it->second.attn_buf);
      if (it->second.attn_claim) (void)hipFree(it->second.attn_claim);
      if (it->second.sm_part) (void)hipFree(it->second.sm_part);
      if (it->second.kn_buf) (void)hipFree(it->second.kn_buf);
      for (auto& t : it->second.attn_off) (void)hipFree(t.second);
      for (auto& t : it->second.g_tables) {
        (void)hipFree(t.desc);
        (void)hipFree(t.sched);
      }
      if (it->second.g_host) (void)hipHostFree(it->second.g_host);
      if (it->second.g_copied) (void)hipEventDestroy(it->second.g_copied);
      it = g_ws.erase(it);
    } else {
      ++it;
    }
  }
}

}  // namespace asym

using asym::fail;

extern "C" int asym_device_query(int device, asym_device_info* out) {
  if (!out) return fail(ASYM_EINVAL, "null out");
  std::memset(out, 0, sizeof *out);
  int n = 0;
  ASYM_HIP(hipGetDeviceCount(&n));
  if (device < 0 || device >= n) return fail(ASYM_EINVAL, "no such device");
  ASYM_HIP(hipDeviceGetAttribute(&out->n_cus, hipDeviceAttributeMultiprocessorCount, device));
  ASYM_HIP(hipDeviceGetAttribute(&out->n_xccs, hipDeviceAttributeNumberOfXccs, device));
  ASYM_HIP(hipDeviceGetAttribute(&out->n_cus_physical, hipDeviceAttributePhysicalMultiProcessorCount, device));
  ASYM_HIP(hipDeviceGetAttribute(&out->clock_khz, hipDeviceAttributeClockRate, device));
  ASYM_HIP(hipDeviceGetAttribute(&out->wall_clock_khz, hipDeviceAttributeWallClockRate, device));
  ASYM_HIP(hipDeviceGetAttribute(&out->lds_bytes_per_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, device));
  ASYM_HIP(hipDeviceGetAttribute(&out->l2_bytes, hipDeviceAttributeL2CacheSize, device));
  hipDeviceProp_t p;
  ASYM_HIP(hipGetDeviceProperties(&p, device));
  out->hbm_bytes = p.totalGlobalMem;
  std::strncpy(out->arch, p.gcnArchName, sizeof(out->arch) - 1);
  if (out->n_xccs < 1) out->n_xccs = 1;
  char bus[sizeof(out->pci_bus_id)] = {0};
  ASYM_HIP(hipDeviceGetPCIBusId(bus, (int)sizeof(bus) - 1, device));
  for (size_t i = 0; i + 1 < sizeof(bus) && bus[i]; ++i) out->pci_bus_id[i] = (char)std::tolower((unsigned char)bus[i]);
  hipUUID u;
  ASYM_HIP(hipDeviceGetUuid(&u, device));
  for (int i = 0; i < 16; ++i)
    std::snprintf(out->uuid + 2 * i, 3, "%02x", (unsigned)(unsigned char)u.bytes[i]);
  ASYM_HIP(hipRuntimeGetVersion(&out->runtime_version));
  ASYM_HIP(hipDriverGetVersion(&out->driver_version));
  return asym::read_partition_modes(out->pci_bus_id, out->compute_partition, out->memory_partition,
                              sizeof(out->compute_partition));
}

extern "C" int asym_gemm_bf16(const asym_topology* topo, int M, int N, int K, const void* A, int lda,
                              const void* B, int ldb, int b_layout, void* C, int ldc, int mapping,
                              uint32_t xcd_mask, void* stream) {
  return asym::gemm_bf16(topo, M, N, K, A, lda, B, ldb, b_layout, C, ldc, mapping, xcd_mask,
                         static_cast<hipStream_t>(stream));
}

extern "C" int asym_gemm_bf16_trace(const asym_topology* topo, int M, int N, int K, const void* A, int lda,
                                    const void* B, int ldb, int b_layout, void* C, int ldc, int mapping,
                                    uint32_t xcd_mask, void* stream, asym_wg_record* records, int capacity,
                                    int* n_records) {
  return asym::gemm_bf16_trace(topo, M, N, K, A, lda, B, ldb, b_layout, C, ldc, mapping, xcd_mask,
                               static_cast<hipStream_t>(stream), records, capacity, n_records);
}

extern "C" int asym_gemm_grouped_bf16(const asym_topology* topo, int G, const int* M, int N, int K,
                                      const void* A, int lda, const void* B, int ldb, void* C, int ldc,
                                      int mapping, uint32_t xcd_mask, void* stream) {
  return asym::gemm_grouped_bf16(topo, G, M, N, K, A, lda, B, ldb, C, ldc, mapping, xcd_mask,
                                 static_cast<hipStream_t>(stream));
}

extern "C" int asym_gemm_plan(const asym_topology* topo, int M, int N, int K, const void* A, int lda,
                              const void* B, int ldb, int b_layout, const void* C, int ldc, int mapping,
                              uint32_t xcd_mask, void* stream, asym_gemm_plan_info* out) {
  return asym::gemm_plan(topo, M, N, K, A, lda, B, ldb, b_layout, C, ldc, mapping, xcd_mask,
                         static_cast<hipStream_t>(stream), out);
}

extern "C" int asym_copy_bf16(const asym_topology* topo, void* dst, const void* src, size_t n_bytes,
                              int passes, const int* stop_flag, uint32_t xcd_mask, void* stream) {
  using namespace asym;
  if (!dst || !src) return fail(ASYM_EINVAL, "copy: null pointer");
  if (n_bytes == 0 || (n_bytes & 15u) || ((uintptr_t)dst & 15u) || ((uintptr_t)src & 15u))
    return fail(ASYM_EINVAL, "copy: size and pointers must be nonzero multiples of 16 bytes");
  if (n_bytes >> 40) return fail(ASYM_EINVAL, "copy: at most 2^40 bytes");
  if (passes < 1) return fail(ASYM_EINVAL, "copy: passes must be >= 1");
  const char* sp = static_cast<const char*>(src);
  const char* dp = static_cast<const char*>(dst);
  if (sp < dp + n_bytes && dp < sp + n_bytes) return fail(ASYM_EINVAL, "copy: source and destination overlap");
  hipStream_t s = static_cast<hipStream_t>(stream);
  std::lock_guard<std::mutex> lock(g_mu);
  // the stream's CU set, less the XCDs outside xcd_mask (their workgroups
  // leave at once); a mask that leaves an XCD without a CU is refused, since
  // the workgroups dealt there could never run
  CuSet cs;
  int rc = cu_set_for(topo, ASYM_MAP_AWARE, xcd_mask, s, "copy", &cs);
  if (rc != ASYM_OK) return rc;
  const int n_x = cs.t->n_xccs;
  return launch_copy(dst, src, n_bytes, passes, stop_flag, cs.slots.data(), n_x,
                     copy_grid(cs.slots.data(), n_x), s);
}

extern "C" int asym_stream_create(const asym_topology* topo, const uint32_t* mask, void** out) {
  using namespace asym;
  if (!out) return fail(ASYM_EINVAL, "null out");
  *out = nullptr;
  hipStream_t s = nullptr;
  if (!mask) {
    ASYM_HIP(hipStreamCreateWithFlags(&s, hipStreamNonBlocking));
    *out = s;
    return ASYM_OK;
  }
  const Topology* t = unwrap(topo);
  if (!t) return fail(ASYM_EINVAL, "stream: a masked stream needs a topology");
  std::vector<int> per;
  int rc = mask_counts(*t, mask, per);
  if (rc != ASYM_OK) return rc;
  for (int x = 0; x < t->n_xccs; ++x)
    if (per[x] == 0)
      return fail(ASYM_EUNSUPPORTED, "stream: the mask leaves XCD " + std::to_string(x) +
                                         " without a CU; workgroups dispatched there could never run "
                                         "(restrict whole XCDs with xcd_mask instead)");
  ASYM_HIP(hipExtStreamCreateWithCUMask(&s, ASYM_MASK_WORDS, mask));
  *out = s;
  return ASYM_OK;
}

extern "C" int asym_stream_destroy(void* stream) {
  if (!stream) return fail(ASYM_EINVAL, "null stream");
  ASYM_HIP(hipStreamSynchronize(static_cast<hipStream_t>(stream)));
  asym::release_workspace(static_cast<hipStream_t>(stream));
  ASYM_HIP(hipStreamDestroy(static_cast<hipStream_t>(stream)));
  return ASYM_OK;
}

extern "C" const char* asym_last_error(void) { return asym::g_last_error.c_str(); }

extern "C" int asym_version(void) { return 1; }

extern "C" int asym_gemm_set_small_m(int enable) {
  return asym::g_small_m.exchange(enable != 0) ? 1 : 0;
}

extern "C" int asym_mla_set_workgroup_form(int level) {
  if (level < 0 || level > 3) return asym::fail(ASYM_EINVAL, "mla: the form level must be 0, 1, 2 or 3");
  return asym::g_mla_form.exchange(level);
}

extern "C" int asym_mla_decode_bf16(const asym_topology* topo, int B, int H_q, int S_k, const void* q,
                                    const void* kv, void* o, float* lse, float scale, int split_tokens, int mapping,
                                    uint32_t xcd_mask, void* stream) {
  return asym::mla_decode(topo, B, H_q, S_k, q, kv, o, lse, scale, split_tokens, mapping, xcd_mask,
                          static_cast<hipStream_t>(stream));
}

extern "C" int asym_mla_decode_plan(const asym_topology* topo, int B, int H_q, int S_k, int split_tokens,
                                    int mapping, uint32_t xcd_mask, void* stream, asym_mla_plan_info* out) {
  return asym::mla_decode_plan(topo, B, H_q, S_k, split_tokens, mapping, xcd_mask, static_cast<hipStream_t>(stream),
                               out);
}

extern "C" int asym_attn_decode_bf16(const asym_topology* topo, int B, int H_q, int H_kv, int S_k, int D,
                                     const void* q, const void* k, const void* v, void* o, float* lse,
                                     float scale, int split_tokens, int mapping, uint32_t xcd_mask,
                                     void* stream) {
  return asym::attn_decode(topo, B, H_q, H_kv, S_k, D, q, k, v, o, lse, scale, split_tokens, mapping, xcd_mask,
                           static_cast<hipStream_t>(stream));
}

extern "C" int asym_attn_decode_paged_bf16(const asym_topology* topo, int B, int H_q, int H_kv, int S_k,
                                           const void* q, const void* k_pool, const void* v_pool, size_t pool_pages,
                                           const int32_t* k_pages, const int32_t* v_pages, void* o, float* lse,
                                           float scale, int split_tokens, int mapping, uint32_t xcd_mask,
                                           void* stream) {
  if (!k_pages || !v_pages) return asym::fail(ASYM_EINVAL, "paged attention: null page table");
  return asym::attn_decode(topo, B, H_q, H_kv, S_k, 128, q, k_pool, v_pool, o, lse, scale, split_tokens, mapping,
                           xcd_mask, static_cast<hipStream_t>(stream), k_pages, v_pages, pool_pages);
}

extern "C" int asym_attn_decode_plan(const asym_topology* topo, int B, int H_q, int H_kv, int S_k, int D,
                                     int split_tokens, int mapping, uint32_t xcd_mask, void* stream,
                                     asym_attn_plan_info* out) {
  return asym::attn_decode_plan(topo, B, H_q, H_kv, S_k, D, split_tokens, mapping, xcd_mask,
                                static_cast<hipStream_t>(stream), out);
}
