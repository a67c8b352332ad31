/*
 * asym: asymmetry-aware scheduling of a persistent bf16 GEMM on MI355X (gfx950).
 *
 * C ABI of libasym.so.  Plain C types only: device buffers are `void*` device
 * pointers, streams are `void*` hipStream_t handles, host arrays are plain
 * pointers with explicit sizes.
 *
 * The calls follow the paper's problem statement ("Dissecting How Die Scaling
 * Breaks GPU Fine-grained Scheduling"):
 *   - discover the chip's hidden compute topology and memory affinity per chip
 *     (Introduction, challenge C-1; Section 5.1 topology discovery;
 *     Section 6.1 latency-based affinity discovery; Appendix G for the
 *     XCD-level variant on AMD parts);
 *   - run a kernel on an allocated set of compute units, assigning work by the
 *     physical unit it lands on (Section 7.1: persistent blocks, affinity-based
 *     static task assignment, work in proportion to each partition's units);
 *   - co-run kernels on partitioned unit sets (Sections 7.2 and 7.3), choosing
 *     which units, not only how many (Section 7.4, lessons).
 *
 * Conventions
 *   Return value: every call returning int returns an asym_status; 0 is
 *   success.  On failure, asym_last_error() returns a message for the calling
 *   thread (valid until that thread's next call into the library).  No call
 *   aborts the process on bad input.
 *   Ownership: the library owns asym_topology objects (free with
 *   asym_topology_free), the streams it creates (destroy with
 *   asym_stream_destroy) and its internal device workspace (schedules,
 *   counters; kept for the life of the process).  All matrix and copy
 *   buffers are owned by the caller; the library never frees them.
 *   Devices: one GPU at a time; `device` is a HIP device ordinal.
 *   Asynchrony: asym_gemm_bf16 and asym_copy_bf16 enqueue work on the given
 *   stream and return; probes and asym_corun synchronise.
 */
#ifndef ASYM_H
#define ASYM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ASYM_MASK_WORDS 8 /* 256 compute units, one bit each */
#define ASYM_MAX_XCDS 16
#define ASYM_MAX_CUS (ASYM_MASK_WORDS * 32)

typedef enum asym_status {
  ASYM_OK = 0,
  ASYM_EINVAL = -1,       /* bad argument (null pointer, size, layout, mask) */
  ASYM_EHIP = -2,         /* a HIP runtime call failed; message has its text */
  ASYM_EUNSUPPORTED = -3, /* valid request the library or device cannot serve */
  ASYM_ETIMEOUT = -4,     /* a watched device wait did not finish in time */
  ASYM_EINVARIANT = -5,   /* a topology map violates its exact invariants */
  ASYM_ENOMEM = -6,       /* host or device allocation failed */
  ASYM_ENOCACHE = -7      /* no usable topology cache: missing, made on another chip
                             or configuration, lacking a requested probe, or malformed */
} asym_status;

/* Tile-to-compute-unit mappings of the persistent GEMM (Section 7.1). */
typedef enum asym_mapping {
  /* Every XCD gets a region of the tile grid: in each band of tile rows, a
   * contiguous run of the band's column-major walk whose length is
   * proportional to the XCD's CUs in the set (largest remainder), so the
   * tiles an XCD runs at once share A rows and B columns in its L2.
   * Workgroup b is XCD (b mod n)'s (b / n)-th worker (the hardware's
   * round-robin dispatch, measured by the identity probe) and runs that
   * region with a stride of the XCD's CU count. */
  ASYM_MAP_AWARE = 0,
  /* Same banded order, tile i to persistent workgroup i mod P: with the
   * hardware's round-robin workgroup-to-XCD dispatch, neighbouring tiles land
   * on different XCDs (the usual single-L2 "grouped" order). */
  ASYM_MAP_OBLIVIOUS_GROUPED = 1,
  /* Row-major tile order, tile i to workgroup i mod P. */
  ASYM_MAP_OBLIVIOUS_ROWMAJOR = 2
} asym_mapping;

/* Storage of the B operand of C = A . B. */
typedef enum asym_b_layout {
  ASYM_B_NK = 0, /* B stored transposed, [N][ldb] row-major, K contiguous */
  ASYM_B_KN = 1  /* B stored [K][ldb] row-major, N contiguous: transposed first
                    (an exact copy into a library buffer), then as ASYM_B_NK */
} asym_b_layout;

/* What asym_probe_topology measures. */
typedef enum asym_probe_flags {
  ASYM_PROBE_IDENTITY = 1, /* XCC/SE/SH/CU of every CU from hardware IDs */
  ASYM_PROBE_MASKMAP = 2,  /* CU-mask bit -> physical CU map (implies IDENTITY) */
  ASYM_PROBE_LATENCY = 4   /* per-XCD L2 / memory-side-cache / HBM latency */
} asym_probe_flags;

/* CU-set policies for asym_cuset_make (Section 7.3; lessons of Section 7.4:
 * tenants state topology requirements, not only counts). */
typedef enum asym_cuset_policy {
  ASYM_CUSET_XCD_ALIGNED = 0,      /* whole XCDs, lowest free XCD ids first */
  ASYM_CUSET_AFFINITY_ALIGNED = 1, /* whole XCDs, filling one affinity group first */
  ASYM_CUSET_STRIPED = 2,          /* the same share of every XCD, SE-balanced */
  ASYM_CUSET_RANDOM = 3            /* seeded uniform choice among free CUs */
} asym_cuset_policy;

/* Device and partition-mode discovery (Section 5.2: topology differs between
 * chips of one product and between configurations, so every probe result is
 * tied to the chip and mode it was measured on). */
typedef struct asym_device_info {
  int n_cus;          /* hipDeviceAttributeMultiprocessorCount */
  int n_xccs;         /* hipDeviceAttributeNumberOfXccs */
  int n_cus_physical; /* hipDeviceAttributePhysicalMultiProcessorCount */
  int clock_khz;      /* peak shader clock */
  int wall_clock_khz; /* rate of the constant-rate counter read by s_memrealtime */
  int lds_bytes_per_cu;
  int l2_bytes;       /* per XCD as reported by the runtime */
  size_t hbm_bytes;
  char arch[64];      /* gcnArchName, e.g. "gfx950:sramecc+:xnack-" */
  char pci_bus_id[32];         /* "dddd:bb:dd.f", lower case */
  char uuid[40];               /* the runtime's device UUID, 32 hex digits */
  int runtime_version;         /* hipRuntimeGetVersion */
  int driver_version;          /* hipDriverGetVersion */
  char compute_partition[16];  /* the driver's current compute partition mode
                                  (e.g. "SPX", "CPX"), "unknown" if not readable */
  char memory_partition[16];   /* current memory partition mode (e.g. "NPS1"),
                                  "unknown" if not readable */
} asym_device_info;

typedef struct asym_topology asym_topology; /* opaque, library-owned */

/* Per-XCD memory latency and affinity (Section 6.1, access latency
 * distribution; Appendix C, the latency kernels; Appendix G, XCD-level probing
 * and XCD grouping on an AMD part).  One lane on one XCD times dependent
 * loads of sampled 128-byte lines, one at a time, with the shader clock
 * (s_memtime).  Three regimes per XCD x:
 *   L2:   the lines were just loaded by x (in x's L2; the sample is far larger
 *         than the per-CU vector cache, so that cache misses);
 *   MALL: all caches flushed, then the lines loaded by another XCD, so they sit
 *         in the memory-side cache but not in x's L2;
 *   HBM:  all caches flushed before every pass.
 * A flush writes a buffer four times the memory-side cache through every XCD.
 * Before each timed load the lane touches another line of the same 2 MiB page,
 * so a translation miss does not enter the timed window.  Every figure is the
 * minimum over `passes` passes per (XCD, address). */
typedef struct asym_latency_params {
  size_t alloc_bytes;     /* sampled allocation; 0 = 32 GiB (less if memory is short);
                             rounded down to a multiple of 2 MiB, at least 64 MiB */
  int n_samples;          /* addresses, uniform 128-byte-aligned lines (<= 1<<22) */
  int passes;             /* 1..64 */
  int l2_samples;         /* the first l2_samples addresses are timed in the L2
                             regime (<= n_samples, <= 8192) */
  uint64_t seed;          /* address sample (splitmix64) */
  double group_threshold; /* XCDs whose HBM latency vectors correlate above this
                             (Pearson) are joined into one affinity group */
  double tie_cycles;      /* an address whose two lowest group means differ by
                             less is left unclassified */
} asym_latency_params;

/* Fill *p with the defaults: 32 GiB, 16384 samples, 8 passes, 4096 L2
 * samples, seed 0, threshold 0.5, tie 20 cycles. */
void asym_latency_params_default(asym_latency_params* p);

/* Results of the latency probe.  Latencies are shader-clock cycles including the timer's
 * own overhead (timer_overhead, reported separately); < 0 = not measured. */
typedef struct asym_latency_summary {
  int n_xcds;
  int n_samples;                   /* addresses per regime (L2: l2_samples) */
  int passes;
  int l2_samples;
  double timer_overhead;           /* cycles of an empty timed window (min) */
  double clock_mhz;                /* shader-clock ticks per microsecond seen by the probe */
  double l2_hit[ASYM_MAX_XCDS];    /* mean latency per XCD, L2 regime */
  double mall_hit[ASYM_MAX_XCDS];  /* mean latency per XCD, memory-side-cache regime */
  double hbm[ASYM_MAX_XCDS];       /* mean latency per XCD, HBM regime */
  int group_of_xcd[ASYM_MAX_XCDS]; /* affinity group of each XCD (0 .. n_groups-1,
                                      numbered by lowest member XCD) */
  int n_groups;
  double home_share[ASYM_MAX_XCDS];/* fraction of addresses whose home is group g */
  double unclassified_share;       /* fraction left unclassified (tie) */
  double corr[ASYM_MAX_XCDS][ASYM_MAX_XCDS];        /* Pearson, HBM regime */
  double hbm_by_home[ASYM_MAX_XCDS][ASYM_MAX_XCDS]; /* [x][g]: mean HBM latency from
                                      XCD x to addresses homed in group g (-1: none) */
} asym_latency_summary;

/* ---- device discovery -------------------------------------------------- */
/* Fill *out from the HIP runtime; the partition modes come from the driver's
 * sysfs files of the device's PCI function (current_compute_partition,
 * current_memory_partition), "unknown" where they cannot be read.
 * Errors: ASYM_EINVAL (null out, no such device), ASYM_EHIP. */
int asym_device_query(int device, asym_device_info* out);

/* The key a probe result of `device` is cached under: one line naming the
 * PCI bus id, UUID, runtime and driver versions, architecture, compute and
 * memory partition modes and CU / XCD counts (Section 5.2: topology is per
 * chip and per configuration).  *needed (nullable) receives the length + 1.
 * Errors: ASYM_EINVAL (null or short buffer), ASYM_EHIP. */
int asym_topology_cache_key(int device, char* buf, size_t len, size_t* needed);

/* ---- topology probe (Section 5.1, Section 6.1, Appendix G) -------------- */
/* Probe `device` and return a new topology map in *out.
 * cache_path (nullable): a per-chip cache file.  If it holds a map made
 * under this device's cache key (asym_topology_cache_key) with at least the
 * requested probes, that map is returned without probing; otherwise the
 * device is probed and the file is (re)written with the result (a failed
 * write is not an error: the probed map is returned).
 * IDENTITY launches an oversubscribed kernel whose workgroups record
 * XCC_ID and HW_ID; the distinct (xcc, se, sh, cu) tuples, sorted, are the
 * CU records with dense indices 0..n-1.  MASKMAP launches the same kernel once
 * per mask bit on a stream whose CU mask has every bit but that one, and maps
 * the bit to the one CU that never appears.  LATENCY runs asym_latency_probe
 * with default parameters and keeps its summary (affinity groups).
 * The map is checked against its exact invariants (every CU once, per-XCD
 * counts summing to the device CU count, mask map a bijection); a violation
 * returns ASYM_EINVARIANT and no map.  Synchronous.
 * Errors: ASYM_EINVAL, ASYM_EHIP, ASYM_EINVARIANT, ASYM_ETIMEOUT. */
int asym_probe_topology(int device, unsigned flags, const char* cache_path,
                        asym_topology** out);

/* Write `topo` to the cache file `path` (text: the key, the probes made,
 * every CU record with its mask bit, the latency summary), replacing it
 * atomically.  `key` (nullable) overrides the key the map was probed under
 * (for maps built from records).  Host only.
 * Errors: ASYM_EINVAL (null argument, unwritable path). */
int asym_topology_save(const asym_topology* topo, const char* path, const char* key);

/* Read a cache file written by asym_topology_save into a new map in *out,
 * accepting it only if its key equals `key` and it holds every probe in
 * `flags`; the map is checked against its exact invariants.  Host only.
 * Errors: ASYM_EINVAL (null argument), ASYM_ENOCACHE (missing file, other
 * key, missing probe, malformed file or broken invariant; the message says
 * which). */
int asym_topology_load(const char* path, const char* key, unsigned flags,
                       asym_topology** out);

/* Build a topology from raw identity records without a GPU (host only).
 * records: n_records rows of 4 int32 {xcc_id register, hw_id register,
 * block index, unused}.  n_cus_expected / n_xccs_expected are the device's
 * counts the invariants are checked against.  mask_bit_cu (nullable): for each
 * mask bit b < n_cus_expected, the index into `records` of a record of the CU
 * that bit controls (-1 if unknown).  Errors: ASYM_EINVAL, ASYM_EINVARIANT. */
int asym_topology_from_records(const int32_t* records, int n_records,
                               int n_cus_expected, int n_xccs_expected,
                               const int32_t* mask_bit_record,
                               asym_topology** out);

void asym_topology_free(asym_topology* topo);

/* Counts of the map.  cus_per_xcd and group_of_xcd (nullable) must hold
 * ASYM_MAX_XCDS ints; group ids are -1 without a latency probe. */
int asym_topology_info(const asym_topology* topo, int* n_cus, int* n_xcds,
                       int* cus_per_xcd, int* group_of_xcd);

/* Record of dense CU `cu_index`: XCC, shader engine, shader array, CU id
 * within its array, and the CU-mask bit controlling it (-1 if no mask map). */
int asym_topology_cu(const asym_topology* topo, int cu_index, int* xcc,
                     int* se, int* sh, int* cu, int* mask_bit);

/* Dispatch consistency of the IDENTITY probe's full-grid launch: the share of
 * workgroups that ran on the XCC holding most of their residue class (block
 * index mod n_xccs); 1.0 = every class on one XCC (round-robin dealing, up to
 * which XCC the dealing starts on). */
int asym_topology_dispatch(const asym_topology* topo, double* rr_fraction);

/* Where launches land on a CU set: runs 4 x n_cus workgroups of the identity
 * kernel on a stream restricted to `mask` (CU-mask bits, ASYM_MASK_WORDS
 * words; NULL = every CU; the same rules as asym_stream_create) and reports
 * the share of workgroups on the XCC holding most of their residue class
 * (block index mod the XCD count), and (nullable, ASYM_MAX_XCDS ints) how
 * many workgroups each XCD ran.  The aware schedules assume each class stays
 * on one XCD, for locality only.  Synchronous.
 * Errors: ASYM_EINVAL, ASYM_EUNSUPPORTED, ASYM_EHIP. */
int asym_dispatch_check(const asym_topology* topo, const uint32_t* mask,
                        double* rr_fraction, int* blocks_per_xcd);

/* The same probe, run right after a launch of pre_blocks workgroups on the
 * same stream (0 = none), also reporting the rotation: the k for which
 * workgroup b ran on XCC (b + k) mod n_xccs most often.  Shows whether the
 * XCC that dealing starts on follows earlier launches.  Synchronous.
 * Errors: as asym_dispatch_check. */
int asym_dispatch_probe(const asym_topology* topo, const uint32_t* mask, int pre_blocks,
                        double* class_fraction, int* rotation, int* blocks_per_xcd);

/* Latency-probe results; ASYM_EUNSUPPORTED if the map was probed without LATENCY. */
int asym_topology_latency(const asym_topology* topo, asym_latency_summary* out);

/* JSON text of the map into buf (len bytes incl. NUL); *needed receives the
 * size required.  Returns ASYM_EINVAL if buf is too small (needed still set). */
int asym_topology_json(const asym_topology* topo, char* buf, size_t len,
                       size_t* needed);

/* ---- latency / affinity probe (Section 6.1, Appendices C and G) -------- */
/* Run the probe on `device` with params p (NULL = defaults).  lat (nullable)
 * receives the per-address minima, uint32 [3][n_xcds][n_samples] in regime
 * order L2, MALL, HBM (L2 rows hold l2_samples values, the rest 0).  The
 * summary is asym_latency_analyze of the HBM regime plus the per-regime
 * means.  Allocates alloc_bytes plus a 1 GiB flush buffer for the duration
 * of the call.  Synchronous; takes seconds at the defaults.
 * Errors: ASYM_EINVAL, ASYM_ENOMEM, ASYM_EHIP, ASYM_ETIMEOUT (no workgroup
 * reached an XCD). */
int asym_latency_probe(int device, const asym_latency_params* p, uint32_t* lat,
                       asym_latency_summary* out);

/* Affinity analysis of HBM-regime latencies (host only, no GPU):
 * hbm_lat is uint32 [n_xcds][n_samples].  corr[x][y] is the Pearson
 * correlation of rows x and y (0 when either row is constant; 1 on the
 * diagonal).  XCDs are joined into a group when their correlation exceeds
 * group_threshold, transitively (connected components).  An address's home is
 * the group with the lowest mean latency over its XCDs (ties to the lower
 * group); it is unclassified when the second-lowest group mean is less than
 * tie_cycles above it (never with a single group).  Fills n_xcds, n_samples,
 * hbm, group_of_xcd, n_groups, home_share, unclassified_share, corr and
 * hbm_by_home of *out; other fields are set to -1.
 * Errors: ASYM_EINVAL. */
int asym_latency_analyze(const uint32_t* hbm_lat, int n_xcds, int n_samples,
                         double group_threshold, double tie_cycles,
                         asym_latency_summary* out);

/* ---- partition-hash discovery (Section 6.1, NUMA partition identification) */
/* Which address bits decide an address's memory partition.  The partition of
 * an address is its home affinity group, classified from HBM-regime latencies
 * as in asym_latency_analyze.  On the GPUs the paper dissects the partition is
 * one parity (XOR) over some physical address bits; flipping one bit of an
 * address and seeing whether the partition changes tells whether the bit takes
 * part, and the lowest bit that takes part sets the granularity.
 *
 * The probe allocates max(2^hi_bit, 2 MiB) bytes starting on a 2 MiB boundary
 * and times, from every XCD (HBM regime, minimum over passes), n_bases blocks
 * of lines.  Block b is, in order: a base line (uniform among the 128-byte
 * lines below 2^hi_bit), the base with offset bit k flipped for each k in
 * [lo_bit, hi_bit), then n_pairs variants with two distinct such bits flipped.
 * Bases and pairs come from splitmix64 seeded with `seed`.  The translation
 * warm-up load before each timed load goes to offset ^ 0x1F0000 (bits 16-20,
 * same 2 MiB page), which is never another line of the same block.  Offsets
 * below the base alignment equal virtual-address bits; bits below the
 * translation page (2 MiB assumed) equal physical bits; flips above it land on
 * other physical pages, whose contribution shows as undetermined bits unless
 * the allocation is physically contiguous there. */
typedef struct asym_interleave_params {
  int n_bases;            /* blocks, 1..4096 */
  int lo_bit;             /* lowest flipped bit, 7..hi_bit-1 (7: 128-byte lines) */
  int hi_bit;             /* one past the highest flipped bit, lo_bit+1..36 */
  int n_pairs;            /* two-bit variants per block, 0..64 (0 if one bit is flipped) */
  int passes;             /* 1..64 */
  uint64_t seed;
  double group_threshold; /* as asym_latency_params */
  double tie_cycles;      /* as asym_latency_params */
  double decide;          /* verdict margin, in (0, 0.5) */
} asym_interleave_params;

/* Defaults: 128 bases, bits 7..31, 4 pairs, 8 passes, seed 1, threshold 0.5,
 * tie 20 cycles, margin 0.1. */
void asym_interleave_params_default(asym_interleave_params* p);

enum { ASYM_BIT_UNDETERMINED = -1, ASYM_BIT_NOT_TESTED = -2 };

typedef struct asym_interleave_result {
  int n_xcds;
  int n_groups;
  int group_of_xcd[ASYM_MAX_XCDS];
  int n_addresses;
  int block;                 /* addresses per block */
  double flip_fraction[64];  /* per bit: share of usable blocks whose base and one-bit
                                variant have different homes; -1 if none usable */
  int usable[64];            /* blocks where both homes were classified */
  int verdict[64];           /* 1 takes part (fraction >= 1 - decide), 0 does not
                                (<= decide), ASYM_BIT_UNDETERMINED (between, or no
                                usable block), ASYM_BIT_NOT_TESTED (never flipped) */
  uint64_t hash_mask;        /* bits with verdict 1 */
  int lowest_bit;            /* lowest bit with verdict 1, -1 if none */
  int determined_below;      /* lowest tested bit that is undetermined (one past the
                                highest tested bit if none): every tested bit below
                                it has a verdict */
  int64_t granularity;       /* 2^lowest_bit bytes when lowest_bit < determined_below,
                                else -1 */
  int pair_checks;           /* two-bit variants whose bits both have verdicts and whose
                                homes (and the base's) are classified */
  int pair_agree;            /* of those, variants whose home differs from the base's
                                exactly when one of the two bits takes part */
  double linear_consistency; /* pair_agree / pair_checks, -1 without checks */
  double unclassified_share; /* addresses with no home (tie) */
  double local_cycles;       /* mean HBM latency from an XCD to lines homed in its own
                                group, over (XCD, line) pairs; -1 if none */
  double remote_cycles;      /* same, lines homed in another group */
  uint64_t base_align;       /* probe only (0 from the analysis): the largest power of
                                two dividing the walked range's start address */
} asym_interleave_result;

/* Run the probe on `device` with params p (NULL = defaults).  With
 * n = n_bases * (1 + hi_bit - lo_bit + n_pairs) addresses: offs (nullable)
 * receives their byte offsets [n], lat (nullable) the HBM latencies
 * uint32 [n_xcds][n] (n_xcds <= ASYM_MAX_XCDS), home (nullable) each address's
 * home group or -1 [n].  The result is asym_interleave_analyze of the
 * measurement plus base_align.  Allocates max(2^hi_bit, 2 MiB) + 2 MiB and a
 * 1 GiB flush buffer for the duration of the call.  Synchronous.
 * Errors: ASYM_EINVAL, ASYM_ENOMEM, ASYM_EHIP, ASYM_ETIMEOUT. */
int asym_interleave_probe(int device, const asym_interleave_params* p, uint64_t* offs,
                          uint32_t* lat, int8_t* home, asym_interleave_result* out);

/* Analysis alone (host only, no GPU).  hbm_lat uint32 [n_xcds][n_addr],
 * offs [n_addr] in blocks of `block` (base first; a variant's flipped bits are
 * its offset XOR its base's: one bit = a flip test, two = a pair check, other
 * counts are ignored).  Homes as asym_latency_analyze with group_threshold and
 * tie_cycles; home (nullable) receives them.  Errors: ASYM_EINVAL (sizes, a
 * partial block, decide outside (0, 0.5)). */
int asym_interleave_analyze(const uint32_t* hbm_lat, int n_xcds, int n_addr,
                            const uint64_t* offs, int block, double group_threshold,
                            double tie_cycles, double decide, int8_t* home,
                            asym_interleave_result* out);

/* ---- home map of an allocation, local / remote reads (Section 6.1 local
 *      and remote bandwidth; Appendix on NUMA-aware address remapping) ---- */
/* Home group (0 or 1) of every 2^chunk_log2-byte chunk of the caller's device
 * range [ptr, ptr + bytes).  The first line of every 2 MiB page is timed from
 * every XCD (HBM regime, minimum over `passes`, translation touch 1 MiB away in
 * the same page), giving the page's home; a chunk's home is its page's home
 * XOR the parity of (chunk offset in the page & hash_mask), the partition
 * hash from asym_interleave_probe restricted to bits below 2 MiB.  Chunks of a
 * page whose first line has no home (tie) get -1.  group_of_xcd (nullable,
 * n_xcds ints) gives the XCD groups; NULL = found from the timed lines by
 * correlation as in asym_latency_analyze.  n_verify random lines (seeded) are
 * also timed and their measured homes compared with the map.  The range is
 * only read.
 * Requirements: ptr and bytes multiples of 2 MiB, 12 <= chunk_log2 <= 21,
 * hash_mask without bits below chunk_log2 inside the page (a chunk must have
 * one home), exactly two groups, at least 16 pages when the groups are found
 * here.  chunk_home receives bytes >> chunk_log2 entries.  Synchronous;
 * allocates a 1 GiB flush buffer for the call.
 * Errors: ASYM_EINVAL, ASYM_EUNSUPPORTED (not two groups), ASYM_EHIP,
 * ASYM_ETIMEOUT. */
typedef struct asym_home_map_info {
  int n_pages;
  int n_chunks;
  int n_groups;
  int group_of_xcd[ASYM_MAX_XCDS];
  int unclassified_pages;
  double chunk_share[2];     /* chunks homed on group 0 / group 1 */
  int n_verify;
  int verify_classified;     /* verification lines with a measured home */
  int verify_agree;          /* of those, lines whose measured home equals the map's */
  double local_cycles;       /* page lines: mean HBM latency from an XCD to lines of
                                its own group / of the other group */
  double remote_cycles;
} asym_home_map_info;

int asym_home_map(int device, const void* ptr, size_t bytes, uint64_t hash_mask, int chunk_log2,
                  const int* group_of_xcd, int passes, int n_verify, uint64_t seed,
                  double tie_cycles, int8_t* chunk_home, asym_home_map_info* info);

/* The map's host analysis alone (no GPU): lat uint32 [n_xcds][n_pages +
 * n_verify] holds the HBM latencies of each page's first line, then of the
 * verification lines at byte offsets verify_offs[n_verify] (below n_pages *
 * 2 MiB); group_of_xcd (required) the two groups.  Same outputs and rules as
 * asym_home_map.  Errors: ASYM_EINVAL, ASYM_EUNSUPPORTED. */
int asym_home_map_analyze(const uint32_t* lat, int n_xcds, int n_pages, const uint64_t* verify_offs,
                          int n_verify, const int* group_of_xcd, uint64_t hash_mask, int chunk_log2,
                          double tie_cycles, int8_t* chunk_home, asym_home_map_info* info);

/* Which chunks each XCD reads, for the read-bandwidth kernel (host only).
 * Active XCDs: bits of xcd_mask (0 = all n_xcds).  Modes:
 *   ALL:    every chunk, dealt round-robin over the active XCDs in chunk order;
 *   LOCAL:  the chunks homed on group g, dealt round-robin over g's active XCDs;
 *   REMOTE: the chunks homed on g, dealt over the other group's active XCDs.
 * LOCAL and REMOTE skip chunks with no home and chunks whose readers have no
 * active XCD.  chunks_out receives the chunk indices XCD by XCD (at most
 * n_chunks), off_out[n_xcds + 1] the start of each XCD's list, *n_listed the
 * total.  Errors: ASYM_EINVAL (sizes, a group id outside 0..1, no active XCD). */
enum asym_chunk_mode { ASYM_CHUNKS_ALL = 0, ASYM_CHUNKS_LOCAL = 1, ASYM_CHUNKS_REMOTE = 2 };
int asym_chunk_lists(const int8_t* chunk_home, int n_chunks, int n_xcds, const int* group_of_xcd,
                     uint32_t xcd_mask, int mode, uint32_t* chunks_out, int* off_out, int* n_listed);

/* Read-bandwidth kernel: every XCD x reads the 2^chunk_log2-byte chunks
 * chunks[off[x] .. off[x+1]) of the device range [base, base + bytes) (chunk
 * c at base + c << chunk_log2; every index must lie below bytes >> chunk_log2,
 * checked on the host), 16 bytes per lane, with 256 workgroups of 256 threads per
 * XCD (a workgroup reads the list of the XCD it runs on, XCC_ID, as one of the
 * workers of its residue class of block indices mod n_xcds, which the hardware
 * deals to one XCD).  Runs `iters` times on `stream` (NULL = null stream) between
 * two events and reports ms per iteration; checksum_out (nullable, 4 words)
 * receives the XOR of every 16-byte word read by one iteration.  chunks and
 * off are host arrays, copied to the device for the call; n_xcds must be the
 * device's XCD count; 12 <= chunk_log2 <= 21; base 16-byte aligned.  Synchronous.
 * Errors: ASYM_EINVAL, ASYM_EHIP. */
int asym_chunk_read_bw(const void* base, size_t bytes, int chunk_log2, const uint32_t* chunks,
                       const int* off,
                       int n_xcds, int iters, void* stream, uint32_t* checksum_out,
                       double* ms_per_iter);

/* The same reader with workers_per_xcd workgroups per XCD (1 .. 4096): few
 * workers keep few loads in flight, so the time per chunk follows the
 * latency of the memory the chunks live in (local or remote to the reading
 * XCD's I/O die) rather than the bandwidth (Section 6.1 measures both).
 * Errors: as asym_chunk_read_bw. */
int asym_chunk_read(const void* base, size_t bytes, int chunk_log2, const uint32_t* chunks,
                    const int* off, int n_xcds, int workers_per_xcd, int iters, void* stream,
                    uint32_t* checksum_out, double* ms_per_iter);

/* ---- CU sets and masked streams ----------------------------------------- */
/* Choose n_cus compute units by `policy` among the CUs not in `exclude`
 * (nullable), and write their CU-mask bits to mask_out[ASYM_MASK_WORDS].
 * Needs a topology probed with MASKMAP.  XCD-aligned policies need n_cus to be
 * a whole number of XCDs.  Errors: ASYM_EINVAL, ASYM_EUNSUPPORTED. */
int asym_cuset_make(const asym_topology* topo, int n_cus, int policy,
                    uint64_t seed, const uint32_t* exclude, uint32_t* mask_out);

/* Two CU sets on disjoint whole-XCD sides: A works on the XCDs in
 * xcd_mask_a, B on the others.  Each side gives the other its lowest CU on
 * each of its XCDs, so that neither mask leaves an XCD empty and workgroups a
 * kernel deals to the other side's XCDs find a free CU there and leave at once
 * (run A with xcd_mask = xcd_mask_a and B with the complement).  Needs a
 * topology with a mask map.  Errors: ASYM_EINVAL, ASYM_EUNSUPPORTED. */
int asym_cuset_split_xcds(const asym_topology* topo, uint32_t xcd_mask_a,
                          uint32_t* mask_a, uint32_t* mask_b);

/* Per-XCD CU counts of a mask (mask bits, ASYM_MASK_WORDS words). */
int asym_cuset_counts(const asym_topology* topo, const uint32_t* mask,
                      int* per_xcd /* ASYM_MAX_XCDS */);

/* Create a stream whose queue may only use the CUs in `mask`
 * (hipExtStreamCreateWithCUMask).  The mask must leave every XCD at least one
 * CU (a queue with an empty XCD is refused: ASYM_EUNSUPPORTED), which needs a
 * topology with a mask map; mask == NULL gives an unmasked stream.  *out
 * receives a hipStream_t.  Errors: ASYM_EINVAL, ASYM_EUNSUPPORTED, ASYM_EHIP. */
int asym_stream_create(const asym_topology* topo, const uint32_t* mask,
                       void** out);
int asym_stream_destroy(void* stream);

/* ---- tile schedule (host only) ------------------------------------------ */
/* Tile order for a tiles_m x tiles_n grid under `mapping`, for n_xcds XCDs
 * with slots[x] persistent workgroups each (0 = XCD excluded).
 * order[tiles_m*tiles_n] receives tile ids (row*tiles_n + col); for AWARE the
 * tiles of XCD x are order[off[x] .. off[x+1]), off has n_xcds+1 entries:
 * every band of `band` tile rows is walked column by column and cut into one
 * contiguous run per XCD, of length proportional to slots[x] (largest
 * remainder, ties to the lower XCD), and XCD x's list is its run of band 0,
 * then of band 1, and so on; quota[x] = off[x+1]-off[x].  For the oblivious
 * mappings off/quota describe which XCD round-robin dispatch sends each order
 * position to.  band = tile rows per band (0 = the height h minimising
 * h + ceil(max slots / h), ties to a divisor of tiles_m, then the taller).
 * Errors: ASYM_EINVAL. */
int asym_schedule_build(int tiles_m, int tiles_n, int n_xcds,
                        const int* slots, int mapping, int band, int* order,
                        int* off, int* quota);

/* Grouped form of the tile schedule (the expert layer of mixture-of-experts
 * models, to which Section 7.1 applies the same recipe): group g has
 * tiles_m[g] >= 0 tile rows of tiles_n columns; tile ids number the tiles in
 * group order, row-major inside a group (base_g + r * tiles_n + c).  Each group
 * is one band, walked column by column, top to bottom.  AWARE shares every
 * group out among the XCDs in contiguous runs of its walk, largest-remainder
 * lengths by slots[x], ties to the lower XCD; XCD x's list is its runs, group
 * after group.  OBLIVIOUS_GROUPED: the walk; OBLIVIOUS_ROWMAJOR: ids in order;
 * both with off/quota as in asym_schedule_build.  order receives
 * sum(tiles_m) * tiles_n ids.  Errors: ASYM_EINVAL. */
int asym_grouped_schedule_build(int G, const int* tiles_m, int tiles_n, int n_xcds,
                                const int* slots, int mapping, int* order, int* off,
                                int* quota);

/* ---- persistent bf16 GEMM (Section 7.1) --------------------------------- */
/* C = A . B, bf16 inputs, fp32 accumulation, bf16 round-to-nearest-even
 * output.  A: [M][lda] row-major.  B: ASYM_B_NK, [N][ldb] row-major (the
 * logical B is its transpose; ldb >= K), or ASYM_B_KN, [K][ldb] row-major
 * (ldb >= N): then B is first transposed, an exact copy on `stream` into a
 * per-stream library buffer of N x K bf16 (grown after a stream
 * synchronisation when a call needs more), and the product runs as for
 * ASYM_B_NK, so both layouts of one logical B give bitwise the same C.
 * C: [M][ldc] row-major.  Requires M, N, K >= 1,
 * lda >= K, ldc >= N; 16-byte aligned pointers with lda, ldb, K
 * multiples of 8 and ldc a multiple of 4 take the vector path, anything else a
 * slower fully predicated path.  The CU set scheduled for is the stream's CU
 * mask (hipExtStreamGetCUMask) restricted to the XCDs in xcd_mask (bit x =
 * XCD x; 0 = all); workgroups landing on other XCDs exit at once.  topo may be
 * NULL (a per-device identity probe made on first use is taken); a stream
 * with a partial CU mask needs a topology with a mask map.  Accumulation order
 * differs from a sequential sum but not between mappings: results are bitwise
 * identical across mappings, CU masks and runs.  (One exception: a product of
 * at most 64 rows whose K the small-M kernel splits on the whole set runs on
 * the persistent kernel under a whole-XCD restriction, and the two fp32 sums
 * may differ in their last bits; see asym_gemm_set_small_m.)  Asynchronous on
 * `stream`.
 * Errors: ASYM_EINVAL, ASYM_EUNSUPPORTED, ASYM_EHIP. */
int asym_gemm_bf16(const asym_topology* topo, int M, int N, int K,
                   const void* A, int lda, const void* B, int ldb,
                   int b_layout, void* C, int ldc, int mapping,
                   uint32_t xcd_mask, void* stream);

/* Grouped GEMM, one launch (Section 7.1 applies the persistent, partition-
 * aware recipe to grouped GEMM, the mixture-of-experts expert layer): for each
 * group g = 0 .. G-1, C_g = A_g . B_g with the numerics of asym_gemm_bf16.
 * M: host array of G row counts (>= 0; zero-row groups are skipped).  A:
 * the groups' rows packed in group order, [sum M][lda]; group g's rows start
 * at row M_0 + ... + M_(g-1).  B: the groups' weights, each stored [N][K] as
 * in ASYM_B_NK, one after the other: [G * N][ldb], group g's at row g * N.
 * C: packed like A, [sum M][ldc].  Tiles never cross a group boundary; rows
 * of other groups are neither read nor written by a group's tiles.  The tile
 * schedule is asym_grouped_schedule_build's, over the stream's CU set as in
 * asym_gemm_bf16; the tile table and schedule are rebuilt on the host and
 * copied to the device on `stream` at every call (the library keeps the
 * device buffers per stream).  Bitwise identical across mappings and CU sets.
 * Asynchronous on `stream`.  Errors: ASYM_EINVAL, ASYM_EUNSUPPORTED,
 * ASYM_EHIP. */
int asym_gemm_grouped_bf16(const asym_topology* topo, int G, const int* M, int N, int K,
                           const void* A, int lda, const void* B, int ldb,
                           void* C, int ldc, int mapping, uint32_t xcd_mask,
                           void* stream);

/* ---- GEMM without allocation ------------------------------------------- */
/* For callers that cannot allocate device memory (code under stream capture,
 * tight serving loops, harnesses that forbid the allocator): asym_gemm_bf16
 * with the same arguments, numerics and kernels (bitwise the same C), but
 * every device buffer that call keeps in its per-stream workspace (the tile
 * schedule, the claim counters of the aware kernel's claiming form, the fp32
 * partial tiles of a split K) sits in one fixed library array per GPU
 * (asym_gemm_noalloc_limits: 17 MiB), held until the process ends.  It calls
 * no allocator, device or pinned: a schedule the array does not hold yet is
 * written into it by small kernels that carry it in their arguments.
 * Limits: topo must be a probed topology (NULL is refused: the first-use
 * probe would allocate); ASYM_B_KN is refused (it needs a transposed copy of
 * B); at most asym_gemm_noalloc_limits' max_tiles output tiles (262016:
 * e.g. M = N = 128000 at 256 x 256 tiles); split-K partials within
 * max_partial_bytes (16 MiB, all a 256-CU device needs).
 * Every call on one GPU shares the array and it keeps the last call's
 * contents (the schedule is tracked on the host, the counters are cleared
 * before each claiming launch): calls that overlap in time on one GPU, on any
 * streams, race and must be serialised by the caller.  Asynchronous.
 * Errors: those of asym_gemm_bf16, plus ASYM_EINVAL beyond the limits. */
int asym_gemm_bf16_noalloc(const asym_topology* topo, int M, int N, int K,
                           const void* A, int lda, const void* B, int ldb,
                           int b_layout, void* C, int ldc, int mapping,
                           uint32_t xcd_mask, void* stream);

/* Size of the per-GPU array, the most output tiles a call may have, and the
 * most bytes of split-K partials (all nullable).  Host only; always ASYM_OK. */
int asym_gemm_noalloc_limits(size_t* scratch_bytes, int* max_tiles, size_t* max_partial_bytes);

/* ---- per-workgroup trace of the persistent GEMM ---------------------------- */
/* One record per workgroup of a traced launch.  Times are the constant-rate
 * clock read by s_memrealtime (asym_device_info.wall_clock_khz ticks per ms),
 * comparable across XCDs. */
typedef struct asym_wg_record {
  uint64_t start;       /* the workgroup began */
  uint64_t first_tile;  /* its first tile began (0: it computed none) */
  uint64_t end;         /* it left */
  uint32_t xcc;         /* XCC_ID it ran on */
  uint32_t hw_id;       /* HW_ID register (SE, shader array, CU, SIMD, wave slot) */
  uint32_t tiles;       /* tiles it computed */
  uint32_t worked;      /* 1 if it computed a tile */
  uint64_t cycles;      /* shader-clock cycles (s_memtime) from start to end: with
                           end - start, the mean clock of the CU it ran on */
} asym_wg_record;

/* asym_gemm_bf16 on the persistent kernel, with every workgroup writing its
 * record to records[block index] (caller-owned device memory, capacity
 * entries): shows how a launch's workgroups are placed and when they start,
 * work and leave (Section 7.1's persistent blocks; the per-CU timing the
 * co-location studies of Sections 7.2 and 7.3 compare).  The traced kernels
 * are separate instantiations of the same code; the bits of C are those of
 * asym_gemm_bf16.  *n_records (host) receives the grid.  Every shape runs
 * the persistent kernel (the small-M kernel has no traced form, so a product
 * asym_gemm_bf16 would give to it gets the persistent kernel's bits);
 * ASYM_B_KN is refused (ASYM_EUNSUPPORTED); capacity below the grid
 * (asym_gemm_plan's grid) is refused (ASYM_EINVAL).  Asynchronous.
 * Errors: those of asym_gemm_bf16. */
int asym_gemm_bf16_trace(const asym_topology* topo, int M, int N, int K,
                         const void* A, int lda, const void* B, int ldb,
                         int b_layout, void* C, int ldc, int mapping,
                         uint32_t xcd_mask, void* stream,
                         asym_wg_record* records, int capacity, int* n_records);

/* What asym_gemm_bf16 with the same arguments would launch, without
 * launching it or touching the matrices: the same checks and errors, the
 * output tile (tile_m x tile_n; the width is taken from 256, 224 and 192 to
 * minimise the rounds of tiles the persistent workers run, Section 7.1's wave
 * quantization), the tile grid, the workgroups launched and the workers that
 * take tiles, per XCD and in all.  claims = 1 when the aware mapping hands
 * tiles out through per-XCD counters (CU sets with unequal XCD counts),
 * 0 when every worker walks a fixed list.  vector_path = 1 for 16-byte loads
 * into LDS, 0 for the predicated path.  Synchronous, host only.
 * Errors: as asym_gemm_bf16. */
typedef struct asym_gemm_plan_info {
  int tile_m, tile_n;
  int tiles_m, tiles_n;
  int grid;
  int workers;
  int claims;
  int vector_path;
  int n_xcds;
  int workers_per_xcd[ASYM_MAX_XCDS]; /* persistent kernel only (0 on the small-M path) */
  int small_m;     /* 1: the small-M kernel (a plain launch of column tiles of
                      tile_n = 64 columns, or 8 to 56 for one unsplit row tile with
                      fewer 64-column tiles than CUs; tile_m = 16, 32 or 64 rows,
                      each wave 16 columns over all of K; grid = workgroups in the
                      mapping's order) */
  int k_splits;    /* small-M kernel with one row tile and fewer 64-column tiles
                      than the device has CUs: K is cut into this many ranges, one
                      workgroup each, and a second launch adds the fp32 partial
                      tiles in range order (1 = no split) */
  int b_transposed; /* 1: B is stored [K][N] and is transposed into the
                       library's per-stream buffer before the product */
} asym_gemm_plan_info;

int asym_gemm_plan(const asym_topology* topo, int M, int N, int K,
                   const void* A, int lda, const void* B, int ldb,
                   int b_layout, const void* C, int ldc, int mapping,
                   uint32_t xcd_mask, void* stream, asym_gemm_plan_info* out);

/* Small-M path.  A GEMM with M <= 64 (a grouped GEMM whose groups all have at
 * most 64 rows), or with at most 256 rows when its 64-row tiles number no more
 * than two per CU of the set, on the vector path and on every XCD of its CU
 * set (xcd_mask 0 or all XCDs) runs a different kernel, built for reading B
 * at HBM rate.  With one row tile no B byte is reused and every mapping gives
 * the same launch; with several, the mapping orders the workgroups: aware runs
 * the row tiles that read one B panel one after another on one XCD (the panel
 * crosses into its L2 once), the oblivious orders put them on neighbouring
 * workgroups (column-major, different XCDs) or a row of tiles apart
 * (row-major).  Every order gives bitwise the same result.  Each workgroup
 * computes 64 columns of C for all rows (a single unsplit row tile with fewer
 * 64-column tiles than the device has CUs takes narrower tiles, a multiple of
 * 8 columns giving about one per CU; the same bits); each of its four waves
 * streams its 16 rows of B over all of K straight into MFMA operands, with A
 * shared through LDS.  This call
 * switches the path on or off for the whole process (default on; off sends
 * such products to the persistent kernel, for comparison) and returns the
 * previous setting.  Not synchronised with launches in flight. */
int asym_gemm_set_small_m(int enable);

/* ---- decode attention (Section 7.1 attention workloads, decode; Appendix F) */
/* One query token per request against cached keys and values, with grouped
 * key/value heads: for request b and query head h, with g = h / (H_q / H_kv),
 *   O[b][h] = softmax_t(scale * q[b][h] . K[b][g][t]) . V[b][g][t]
 *   lse[b][h] = log sum_t exp(scale * q[b][h] . K[b][g][t])   (nullable output)
 * Layout (contiguous, caller-owned device memory): q [B][H_q][D], K and V
 * [B][H_kv][S_k][D], O [B][H_q][D], all bf16; lse fp32 [B][H_q].  D must be
 * 128 and H_q / H_kv one of 1, 2, 4, 8, 16.  q, K, V 16-byte aligned; O and
 * lse 4-byte aligned.
 * The sequence is cut into splits of split_tokens tokens (0 = automatic: the
 * longest of 1024, 512, ... 64 giving at least 2048 tasks); a task is one
 * (request, key/value head, split) and serves that head's query heads, so K
 * and V are read once.  A second launch merges the splits of each (request,
 * head) in an order fixed by the split count.  Mapping: AWARE gives each XCD a share of the tasks
 * proportional to its CU count in the stream's CU set (and honours a
 * whole-XCD restriction); its workgroups read the XCD they run on and claim
 * groups of 4 tasks from that XCD's share, then from the others; the
 * oblivious mappings (both) hand out tasks round-robin by workgroup, an equal
 * share per XCD.  On a CU set with equal CUs per XCD over every XCD, when each
 * claiming workgroup would hold one group at most and splits are at most 128
 * tokens, a dense AWARE call deals its groups round-robin as the oblivious
 * mappings do (there the shares are equal and claims only cost their round
 * trips); asym_attn_decode_plan reports it.  Every mapping gives the same bits.  fp32 partials live in a per-stream library workspace, grown
 * (after a stream synchronisation) when a call needs more.  Asynchronous.
 * Errors: ASYM_EINVAL, ASYM_EUNSUPPORTED, ASYM_EHIP. */
int asym_attn_decode_bf16(const asym_topology* topo, int B, int H_q, int H_kv, int S_k, int D,
                          const void* q, const void* k, const void* v, void* o, float* lse,
                          float scale, int split_tokens, int mapping, uint32_t xcd_mask,
                          void* stream);

typedef struct asym_attn_plan_info {
  int split_tokens;
  int n_splits;
  int tasks;               /* B * H_kv * n_splits */
  int grid;                /* workgroups of the split launch */
  int tasks_per_workgroup; /* one per wave */
  int n_xcds;
  int tasks_per_xcd[ASYM_MAX_XCDS];
  size_t workspace_bytes;  /* fp32 partials: B * H_q * n_splits * 130 * 4 */
  int dense_static;        /* AWARE: 1 if a dense call deals its groups statically
                              (grid = ceil(tasks / tasks_per_workgroup), no claims;
                              grid and tasks_per_xcd above are the claiming launch's,
                              which paged calls always take) */
} asym_attn_plan_info;

/* What asym_attn_decode_bf16 would launch (no pointers needed; launches
 * nothing).  Errors as asym_attn_decode_bf16. */
int asym_attn_decode_plan(const asym_topology* topo, int B, int H_q, int H_kv, int S_k, int D,
                          int split_tokens, int mapping, uint32_t xcd_mask, void* stream,
                          asym_attn_plan_info* out);

/* Paged form of asym_attn_decode_bf16 (Appendix E: memory remapping, here of
 * the key/value cache).  K and V live in caller-owned pools of pool_pages
 * pages of 8 KiB each, a page holding 32 consecutive tokens of one head
 * ([pool_pages][32][128] bf16; pool_pages * 8 KiB at most 2 GiB); k_pages and
 * v_pages (device int32 [B][H_kv][ceil(S_k / 32)]) give the pool page of each
 * (request, head, 32-token page), the tokens past S_k in a head's last page
 * being ignored.  Two table entries may name the same page; an entry outside
 * [0, pool_pages) reads zeros or other bytes of the pool, never memory outside
 * it (the pools are read through buffer descriptors sized to them).  Splits are
 * at most 2048 tokens (0 = automatic).  Everything else, and the bits of O
 * and lse, as asym_attn_decode_bf16 on the dense K and V the tables describe:
 * the tables only change where each page's bytes are.
 * Errors: those of asym_attn_decode_bf16. */
int asym_attn_decode_paged_bf16(const asym_topology* topo, int B, int H_q, int H_kv, int S_k,
                                const void* q, const void* k_pool, const void* v_pool,
                                size_t pool_pages, const int32_t* k_pages, const int32_t* v_pages,
                                void* o, float* lse, float scale, int split_tokens, int mapping,
                                uint32_t xcd_mask, void* stream);

/* Page placement for asym_attn_decode_paged_bf16 (Appendix E's placement by
 * home: each task's pages in memory homed on the die of the XCD that reads
 * them).  From a plan of the AWARE mapping (asym_attn_decode_plan: task t
 * belongs to the XCD whose share, in XCD order, holds it), pool_home
 * (pool_pages entries, the home group 0 / 1 of each pool page as
 * asym_home_map gives it, -1 unknown; nullable for IN_ORDER) and
 * group_of_xcd (n_xcds entries), fills pages (host int32
 * [B][H_kv][ceil(S_k / 32)]):
 *   ASYM_PAGES_IN_ORDER: page i of the table is pool page i (the dense layout);
 *   ASYM_PAGES_LOCAL: the next unused pool page homed on the group of the XCD
 *     that owns the task reading the page (its first token's task);
 *   ASYM_PAGES_REMOTE: the same on the other group (the worst placement).
 * Every table entry is a distinct pool page.  Host only.
 * Errors: ASYM_EINVAL (inconsistent plan, too few pool pages of a group). */
enum asym_page_policy { ASYM_PAGES_IN_ORDER = 0, ASYM_PAGES_LOCAL = 1, ASYM_PAGES_REMOTE = 2 };
int asym_attn_pages_place(const asym_attn_plan_info* plan, int B, int H_kv, int S_k,
                          const int8_t* pool_home, size_t pool_pages, const int* group_of_xcd,
                          int policy, int32_t* pages);

/* ---- multi-head latent attention, decode (Section 7.1; Appendix F) ---- */
/* One query token per request against a compressed latent cache shared by
 * all query heads (the decode form of multi-head latent attention, with the
 * projections absorbed into the query; Appendix F counts one row of 512 + 64
 * values per token).  For request b and query head h:
 *   s_t = scale * <q[b][h], kv[b][t]>                  (576 values)
 *   O[b][h] = sum_t softmax_t(s)_t * kv[b][t][0 .. 511]
 *   lse[b][h] = log sum_t exp(s_t)                     (nullable output)
 * Layout (contiguous, caller-owned device memory): q [B][H_q][576],
 * kv [B][S_k][576] (per token: 512 latent values, which are also the value,
 * then 64 rotary key values), O [B][H_q][512], all bf16; lse fp32 [B][H_q].
 * H_q a multiple of 16 (at most 1024); q, kv and O 16-byte aligned; a
 * request's cache below 2 GiB.
 * The sequence is cut into splits of split_tokens tokens (0 = automatic: the
 * longest of 1024, 512, ... 32 giving at least 1024 blocks of 16 heads times
 * splits, lengthened until there are at most 256 splits, and in the
 * workgroup forms further, up to 8192, while at least two tasks per CU of the
 * set remain; a split of 1024 tokens or more is halved when that gives the
 * 128-head form more tasks than half the set's CUs; else a multiple of 32); a task is one (request, split, block of 16 query heads) on one wave
 * of the matrix cores (wave form, 16-token blocks), or, when H_q is a
 * multiple of 64, one (request, split, four blocks of 16 heads) on one
 * workgroup whose four waves share each 32-token block of rows through LDS
 * (64-head form), or, when H_q is a multiple of 128 and those tasks number
 * more than half the CUs of the set, one (request, split, eight blocks of 16
 * heads) on one workgroup, two head blocks per wave (128-head form).  The two workgroup forms give the same bits (the same
 * operations per head); the wave form, with a softmax step every 16 tokens,
 * rounds differently (asym_mla_set_workgroup_form).  A second launch merges
 * the splits of each (request, head) in an order fixed by the split count.  Mapping: AWARE numbers the tasks request-split
 * major, so the head blocks that read the same cache rows are consecutive,
 * gives each XCD a share of that list in proportion to its CUs in the
 * stream's CU set (honouring a whole-XCD restriction), and lets workgroups
 * claim groups of 4 tasks (one task in the workgroup form) from their XCD's
 * share, then from the others: the
 * rows cross into one XCD's L2 once.  The oblivious mappings (both) number
 * them head-block major and hand out 4 per workgroup in order, so the head
 * blocks of one split land on different XCDs and every XCD gets an equal
 * share.  On a CU set with equal CUs per XCD over every XCD, when each
 * claiming workgroup would hold one group of tasks at most (every task runs
 * at once and claims could move no work), an AWARE call deals its tasks as
 * the oblivious mappings do; asym_mla_decode_plan reports it.
 * Every mapping gives the same bits.  fp32 partials live in a
 * per-stream library workspace, grown (after a stream synchronisation) when a
 * call needs more.  Asynchronous.
 * Errors: ASYM_EINVAL, ASYM_EUNSUPPORTED, ASYM_EHIP. */
int asym_mla_decode_bf16(const asym_topology* topo, int B, int H_q, int S_k,
                         const void* q, const void* kv, void* o, float* lse,
                         float scale, int split_tokens, int mapping, uint32_t xcd_mask,
                         void* stream);

typedef struct asym_mla_plan_info {
  int split_tokens;
  int n_splits;
  int head_blocks;         /* H_q / 16 */
  int tasks;               /* B * n_splits * head_blocks (wave form),
                              B * n_splits * head_blocks / 4 or / 8 (64- and 128-head forms) */
  int grid;                /* workgroups of the split launch */
  int tasks_per_workgroup; /* 4, one per wave (wave form); 1 (workgroup forms) */
  int n_xcds;
  int tasks_per_xcd[ASYM_MAX_XCDS];
  int workgroup_form;      /* 0: wave form; 1: 64-head form; 2: 128-head form */
  size_t workspace_bytes;  /* fp32 partials: B * H_q * n_splits * 514 * 4 */
  int static_deal;         /* AWARE: 1 if the call deals its tasks statically
                              (grid = ceil(tasks / tasks_per_workgroup), no claims;
                              grid and tasks_per_xcd above are the claiming launch's) */
} asym_mla_plan_info;

/* Which kernel forms asym_mla_decode_bf16 may take, for the process: 0 runs
 * every head count in the wave form, 1 allows the 64-head form, 2 (the
 * default) also the 128-head form where it has enough tasks, 3 the 128-head
 * form wherever H_q is a multiple of 128; for comparisons.  Returns the
 * previous level.  Not synchronised with launches in flight.
 * Errors: ASYM_EINVAL (a level other than 0 to 3). */
int asym_mla_set_workgroup_form(int level);

/* What asym_mla_decode_bf16 would launch (no pointers needed; launches
 * nothing).  Errors as asym_mla_decode_bf16. */
int asym_mla_decode_plan(const asym_topology* topo, int B, int H_q, int S_k, int split_tokens,
                         int mapping, uint32_t xcd_mask, void* stream, asym_mla_plan_info* out);

/* ---- streaming copy and co-run (Sections 7.2, 7.3) ---------------------- */
/* The bandwidth-bound tenant of the co-location study (Section 7.3 runs a
 * second tenant on the complementary units): dst[i] = src[i] for n_bytes
 * bytes, `passes` times over the buffer, with 16-byte accesses from every lane
 * (non-temporal).  dst and src: caller-owned device buffers, 16-byte aligned,
 * not overlapping; n_bytes a nonzero multiple of 16, below 2^40; passes >= 1.
 * The CU set is the stream's CU mask restricted to the XCDs in xcd_mask
 * (0 = all), as for asym_gemm_bf16 (topo NULL: the per-device identity probe;
 * a partial mask needs a topology with a mask map; a mask that leaves an XCD
 * without a CU is refused).  The buffer is cut into one slice per XCD of the
 * set, in proportion to its CUs there, copied by the workgroups the hardware
 * deals to that XCD; workgroups on XCDs outside xcd_mask exit at once.  No
 * atomics, no barriers: the copy always ends after `passes` passes.  If
 * stop_flag (a device int, nullable) is nonzero when a wave starts a pass
 * after its first, that wave ends there (it never extends the copy).
 * Asynchronous on `stream`.
 * Errors: ASYM_EINVAL, ASYM_EUNSUPPORTED, ASYM_EHIP. */
int asym_copy_bf16(const asym_topology* topo, void* dst, const void* src, size_t n_bytes,
                   int passes, const int* stop_flag, uint32_t xcd_mask, void* stream);

/* One task of a co-run: a GEMM or a streaming copy on its own CU set. */
typedef struct asym_task {
  int kind;        /* 0 = GEMM, 1 = streaming copy, 2 = read (whole-buffer reader) */
  uint32_t mask[ASYM_MASK_WORDS]; /* CU-mask bits; all-zero = all CUs */
  uint32_t xcd_mask;              /* whole-XCD restriction, 0 = none */
  int iters;       /* GEMM launches, or copy / read passes (>= 1) */
  int mapping;     /* GEMM mapping */
  int M, N, K;     /* GEMM shape, dense row-major A, B ([N][K]), C */
  const void* A; const void* B; void* C;
  const void* src; void* dst; size_t n_bytes; /* copy: both (16-byte aligned,
                                                 not overlapping); read: src; n_bytes
                                                 a multiple of 16, < 2^40 */
  int grid;        /* copy / read: workgroups; 0 = 8 per CU of the XCD of its set
                      with the most CUs, times the XCD count */
  int warm_iters;  /* untimed launches / passes queued right before the timed
                      ones (>= 0), so the shader clock has settled under the
                      co-run's own load when timing starts */
} asym_task;

typedef struct asym_task_result {
  double ms_total;    /* first launch start to last launch end */
  double ms_per_iter;
  double tflops;      /* GEMM */
  double gbps;        /* copy: bytes read + written per second / 1e9; read: bytes read */
  int iters_done;
  uint32_t checksum[4]; /* read: XOR of every 16-byte word read, over all passes
                           (for an odd pass count, the XOR of the buffer's words
                           when each was read once per pass) */
} asym_task_result;

/* Run tasks concurrently, each on its own stream (masked streams for partial
 * masks, unmasked streams with XCD filtering for whole-XCD sets; Sections
 * 7.2 and 7.3).  All tasks are released together.  A copy task makes `iters`
 * passes of asym_copy_bf16 over its buffers and a read task `iters` passes of
 * a whole-buffer reader (16-byte loads, no atomics); both cut their buffer
 * into one slice per XCD of their set, in proportion to their CUs there, and
 * an xcd_mask keeps their work on those XCDs (workgroups elsewhere, e.g. on
 * CUs a split mask lends them there, leave at once).  No task is open-ended:
 * a tenant that ran until the GEMMs ended could deadlock with a persistent
 * GEMM whose workgroups dealt to the tenant's XCDs wait for its CUs, so a
 * copy task with iters < 1 is refused; size the passes to outlast the GEMMs.
 * Every GEMM task is launched once, untimed, before the release, so that its
 * one-time setup (workspace, schedule upload) does not wait for tasks already
 * running.  With warm_iters > 0 on any task, every task first runs its
 * warm_iters untimed (the caller sizes them to end together) and each
 * stream's timed part waits for every task's warm-up to end: the shader clock
 * rises over tens to hundreds of milliseconds of sustained load, so a short
 * timed co-run straight after an idle host sync runs at a lower clock than
 * the same co-run in steady state.  Synchronous.
 * Errors: ASYM_EINVAL, ASYM_EUNSUPPORTED, ASYM_EHIP. */
int asym_corun(const asym_topology* topo, const asym_task* tasks, int n_tasks,
               asym_task_result* out);

/* ---- misc ---------------------------------------------------------------- */
const char* asym_last_error(void);
int asym_version(void);

#ifdef __cplusplus
}
#endif
#endif /* ASYM_H */
