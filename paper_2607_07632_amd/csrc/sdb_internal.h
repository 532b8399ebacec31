// Internal structures shared by the host runtime (sdb_api.cpp) and the
// device kernels (sdb_kernels.hip). Nothing here is part of the public ABI.
#pragma once

#include <stdint.h>

#include <hip/hip_runtime_api.h>

#include "sdb.h"

namespace sdb {

constexpr int kMaxStages = SDB_MAX_STAGES;
constexpr int kMaxEager = SDB_MAX_EAGER;
constexpr int kBlock = 256;              // default threads per block of the fused kernel
constexpr int kMaxBlock = 512;           // launch bound of the fused kernel
constexpr int kBigBlock = 1024;          // launch bound of its big-block instances (4-row items, IPT 1 or 2)
constexpr int kUnrollStages = 4;         // stage copies of the fused kernel's unrolled instances
// partitioned terminal: at most this many record regions per fused-kernel
// block (sdb_plan.part_subs; wave w writes region w mod part_subs of its
// block), so that the partition scatter pass, one block per region, runs
// several blocks per CU
constexpr int kPartSubRegions = 4;
constexpr int kLdsGroupLimit = 2048;     // LDS terminal: sums + counts of G <= 2048 groups (32 KB)
constexpr int kLdsStageBudget = 32768;   // LDS bytes per block for staged dimension tables
constexpr int kXcdCopies = 8;            // XCDs of an MI355X: private group-table copies
constexpr int kFinBlock = 256;           // finalize: threads per block
constexpr int kFinPerThread = 4;         // finalize: groups per thread
constexpr int kFinGroupsPerBlock = kFinBlock * kFinPerThread;
constexpr int kDenseSlack = 1024;        // dense limit: key range <= max(2 * n_rows, 1024)

enum StageKind : int32_t { ST_PRED = 0, ST_DENSE = 1, ST_HASH = 2 };

// What the fused kernel does for a stage, fixed by the host so the kernel
// branches once per stage and tile instead of once per row.
enum StageOp : int32_t {
    OP_PRED = 0,      // literal range test
    OP_NEVER = 1,     // lookup in an empty table: every row misses
    OP_LDS_BITS = 2,  // pass bitmap in LDS
    OP_LDS_MAP1 = 3,  // whole map in LDS, 1/2/4-byte codes
    OP_LDS_MAP2 = 4,
    OP_LDS_MAP4 = 5,
    OP_MAP1 = 6,      // map in device memory, 1/2/4-byte codes
    OP_MAP2 = 7,
    OP_MAP4 = 8,
    OP_HASH = 9,      // open-addressing table in device memory
    OP_LDS_RANK1 = 10,  // pass bitmap, ranks and passing codes in LDS, 1/2/4-byte codes
    OP_LDS_RANK2 = 11,
    OP_LDS_RANK4 = 12,
    OP_COARSE1 = 13,    // coarse pass bitmap in LDS, then the device map, 1/2/4-byte codes
    OP_COARSE2 = 14,
    OP_COARSE4 = 15,
    OP_HASH_PAIR = 16,  // OP_HASH reading the home slot and the next with one 16-byte load
    OP_WINDOW1 = 17,    // pass bitmap of a key window in LDS, the device map outside it, 1/2/4-byte codes
    OP_WINDOW2 = 18,
    OP_WINDOW4 = 19
};
// How a table's code becomes part of the group id.
enum GroupMode : int32_t { GK_NONE = 0, GK_ONE = 1, GK_GENERAL = 2 };
enum LdsMode : int32_t {
    LDS_GLOBAL = SDB_LDS_GLOBAL,
    LDS_MAP = SDB_LDS_MAP,
    LDS_BITS = SDB_LDS_BITS,
    LDS_RANK = SDB_LDS_RANK,
    LDS_COARSE = SDB_LDS_COARSE,
    LDS_WINDOW = SDB_LDS_WINDOW
};
enum Terminal : int32_t { TERM_SCALAR = 1, TERM_LDS = 2, TERM_GLOBAL = 3, TERM_PART = 4 };

// Partitioned aggregation (TERM_PART): partition of group g is g >> part_shift.
constexpr int kPartMaxParts = 4096;       // LDS histogram bins in the fused and scatter kernels
constexpr int kPartMaxShift = 12;         // at most 4096 groups per partition (64 KB LDS table)
constexpr int kPartChunk = 65536;         // records per aggregation work item
constexpr int kScatterChunk = 4096;       // records one scatter block sorts in LDS at a time
constexpr uint32_t kRingEntries = 128;     // fused kernel: per-wave record ring (group id + value)
constexpr uint32_t kLdsRankBudget = 98304;  // LDS for a stage's rank tables (bitmap, counts, codes)
constexpr uint32_t kRankGroups = 4096;      // at most this many 64-slot groups (one scan block)

// Sliced hash probe: fact rows partitioned by the top bits of the key's hash.
constexpr int kSliceBlock = 1024;          // threads per block of the count and scatter passes
constexpr int kSliceRowsPerThread = 16;    // rows a thread holds per scatter chunk
constexpr int kSliceChunk = kSliceBlock * kSliceRowsPerThread;   // rows one block sorts in LDS at a time
constexpr int kSliceMaxGrid = 256;         // one block per compute unit of an MI355X
static_assert(SDB_MAX_SLICE_BITS <= 10, "scatter LDS holds 3 x 2^10 partition counters");

// A literal comparison lowered to one unsigned range test over int32:
// pass  <=>  ((uint32_t)(x - lo) <= span) != negate.
struct RangeTest {
    int32_t lo;
    uint32_t span;
    int32_t negate;
};

// One stage of the fused pass, as the kernel reads it (kernel argument).
struct StageDev {
    int32_t kind;          // StageKind
    int32_t op;            // StageOp
    int32_t gk_mode;       // GroupMode: GK_ONE adds code * gk_stride[0]
    int32_t col;           // fact column index
    RangeTest test;        // ST_PRED
    int32_t width;         // ST_DENSE: bytes per map entry (1, 2, 4)
    int32_t kmin;          // ST_DENSE: key of slot 0
    uint32_t nslots;       // ST_DENSE: slots; ST_HASH: capacity (power of two)
    uint32_t hmask;        // ST_HASH: capacity - 1
    int32_t hshift;        // ST_HASH: 32 - log2(capacity)
    uint32_t sentinel;     // code meaning "no passing dimension row"
    const void* map;       // ST_DENSE / ST_HASH table
    const void* bits;      // ST_DENSE: pass bitmap (32-bit words)
    int32_t lds_mode;      // LdsMode: where the probe looks the key up
    uint32_t lds_off;      // byte offset of the staged table in dynamic LDS
    uint32_t lds_bytes;    // staged bytes (a multiple of 16)
    int32_t defer;         // LDS_BITS with group keys: 0 = gather the code after all stages
    int32_t n_gk;          // group keys decoded from this table's code
    uint32_t gk_div[SDB_MAX_PAYLOADS];     // key code = (code / div) % radix (div 1: skip)
    uint32_t gk_radix[SDB_MAX_PAYLOADS];   // 0: no modulo needed
    uint32_t gk_stride[SDB_MAX_PAYLOADS];  // group-id stride of that key
    int32_t eg_slot;       // eager slot holding this stage's column, or -1
    // LDS_RANK: running counts (uint32 per 64 slots) and the passing slots'
    // codes, staged from device memory (run scratch) behind the bitmap
    const void* rank;
    const void* codes;
    uint32_t lds_rank_off;
    uint32_t lds_rank_bytes;
    uint32_t lds_codes_off;
    uint32_t lds_codes_bytes;
    // LDS_COARSE: bit j of the staged bitmap (at lds_off, staged from `bits`,
    // which then points at the coarse bitmap in the run scratch) covers
    // slots [j << coarse_shift, (j + 1) << coarse_shift)
    int32_t coarse_shift;
    // LDS_WINDOW: the staged bitmap (at lds_off, staged from `bits`, which then
    // points at the window's first word) covers slots [win_lo, win_lo + win_slots)
    uint32_t win_lo;
    uint32_t win_slots;
    int32_t sample_hist;   // planner sampling: 1 = histogram this dense stage's keys
};
// sampling: key histogram buckets per dense stage; pass-pattern bins a block
// counts in LDS (plans of up to 12 stages)
constexpr int kKeyBuckets = 256;
constexpr int kSamplePatternsLds = 4096;
// sampled row ranges for segmented plans (plans of up to kSampleRangeStages stages)
constexpr int kSampleRanges = 16;
constexpr int kSampleRangeStages = 10;

// Derives a coarse pass bitmap (LDS_COARSE) from a dense table's pass bitmap.
struct CoarseParams {
    const uint32_t* bits;      // pass bitmap, nslots bits
    uint32_t nslots;
    uint32_t shift;            // 1 .. SDB_MAX_COARSE_SHIFT
    uint32_t* out;             // n_words words
    uint32_t n_words;          // ceil(ceil(nslots / 2^shift) / 32), padded to whole 16-byte groups
};
hipError_t launch_coarse_build(const CoarseParams& cp, hipStream_t s);

// Derives a dense table's rank tables (LDS_RANK) in device memory.
struct RankParams {
    const uint32_t* bits;      // pass bitmap, nslots bits
    const void* map;           // packed codes, width bytes per slot
    int32_t width;
    uint32_t nslots;
    uint32_t* prefix;          // (nslots + 63) / 64 entries: passing slots before each 64-slot group
    void* codes;               // codes of the passing slots in slot order
};

struct FusedParams {
    const int32_t* cols[SDB_MAX_FACT_COLS];
    int64_t n;
    const uint32_t* n_dev;     // non-null: rows are min(n, *n_dev) (a count another kernel wrote)
    const int32_t* tile_map;   // non-null: loop index t runs tile tile_map[t] (< 0: none), t < n_vtiles
    int64_t n_vtiles;
    int32_t nstages;
    int32_t agg_kind;
    int32_t agg_a;
    int32_t agg_b;
    uint32_t n_groups;
    uint32_t term_lds_bytes;   // LDS group table at the start of dynamic LDS (LDS terminal)
    int32_t defer_stage;       // stage whose code is gathered after all stages, or -1
    int32_t xcd_copies;        // > 0: global terminal adds into xtab copy (XCC id mod copies)
    unsigned long long* sums;
    unsigned long long* counts;
    unsigned long long* xtab;  // interleaved {sum, count} x n_groups x xcd_copies
    // TERM_PART: region r = (region_base + block) * part_subs + (wave mod
    // part_subs) appends survivors to records [r * part_cap, (r + 1) * part_cap)
    uint32_t* region_count;    // records each block wrote
    uint32_t* rec_gid;
    void* rec_val;             // int64 values if rec_wide, else int32
    uint32_t* part_hist;       // records per (partition, region): [q * n_regions + region]
    uint32_t region_base;      // region of block 0 (a segmented plan launches once per segment)
    uint32_t n_regions;        // regions of all launches
    uint32_t part_cap;
    int32_t part_shift;
    uint32_t n_parts;
    uint32_t part_subs;        // record regions per block (1 .. kPartSubRegions)
    uint32_t ring_off;         // byte offset of the per-wave record rings in dynamic LDS
    int32_t rec_wide;          // 1: record values need 64 bits (aggregate of two columns)
    // eager columns (4-row items): slot k holds cols[eg_col[k]] for the current items
    int32_t eg_n;
    int32_t eg_col[kMaxEager];
    int32_t agg_a_slot;        // eager slot of agg_a / agg_b, or -1
    int32_t agg_b_slot;
    StageDev st[kMaxStages];
};

// Statistics block at the start of a dimension workspace.
struct DimStats {
    int32_t kmin;
    int32_t kmax;
    unsigned long long npass;
    int32_t pmin[SDB_MAX_PAYLOADS];
    int32_t pmax[SDB_MAX_PAYLOADS];
    uint32_t dup;          // 1: duplicate key seen; 2: hash table full (cannot happen when sized)
    uint32_t pad_;
    unsigned long long occupied;   // dense: slots that some row holds
    int32_t pkmin;                 // key range over passing rows
    int32_t pkmax;
};
static_assert(sizeof(DimStats) <= 256, "stats must fit the reserved 256 bytes");
static_assert(sizeof(FusedParams) <= 4096, "kernel arguments must fit the 4 KB kernarg segment");

// most statistics blocks per table: each writes its partial statistics (one
// DimStats) to the table region, which the build fills only afterwards, and a
// second kernel combines them, so no statistic is updated with atomics
constexpr int kStatsMaxBlocks = 1024;
constexpr int kBuildRows = 16;            // rows per thread and step of a 256-thread statistics or dense-scatter block

struct BuildParams {
    const int32_t* key;
    int64_t n;
    const int32_t* cols[SDB_MAX_DIM_COLS];
    int32_t n_preds;
    int32_t pred_col[SDB_MAX_DIM_PREDS];
    RangeTest pred[SDB_MAX_DIM_PREDS];
    int32_t n_payloads;
    int32_t payload_col[SDB_MAX_PAYLOADS];
    int32_t pmin[SDB_MAX_PAYLOADS];
    uint32_t pdiv[SDB_MAX_PAYLOADS];
    DimStats* stats;
    DimStats* stats_part;      // stats_blocks partial statistics (in the table region)
    int32_t stats_blocks;
    int32_t pad3_;
    void* map;                 // dense map or hash table
    uint32_t* pass_bits;       // dense pass bitmap
    int32_t width;
    int32_t kmin;
    uint64_t nslots;
    uint32_t sentinel;         // dense: code of a filtered row; codes >= sentinel mean "no passing row"
    uint32_t missing;          // dense: code of a key no row holds (all ones)
    uint32_t hmask;
    int32_t hshift;
    int32_t dense;             // 1: dense map (scatter + bitmap), 0: hash table (inserts)
    uint32_t fill_value;       // the table's initial word value (all ones dense, 0 hash)
    uint64_t fill_words;       // 32-bit words of the table to fill before the scatter / inserts
                               // (a hash table's pass filter follows its slots and is filled too)
    uint32_t* filt;            // hash: pass filter words (SDB_FILTER_*), or null
    uint64_t filt_bits;
    int32_t filt_kind;
    int32_t filt_via_bytes;    // 1: a bitmap filter built through a byte per key in the slot
                               // region before the slots are filled (no atomics); 0: the
                               // inserts set its bits with atomics
};

// Every table of one sdb_build_dims call; kernels take table blockIdx.y.
struct BuildBatch {
    int32_t n;
    int32_t pad_;
    DimStats* host_stats;      // n statistics blocks in pinned host memory (device address), or null
    BuildParams bp[SDB_MAX_JOINS];
};

struct FinalizeParams {
    const long long* sums;
    const long long* counts;
    uint64_t n_groups;
    int32_t n_keys;
    int32_t scalar;
    int32_t key_min[SDB_MAX_GROUP_KEYS];
    uint32_t radix[SDB_MAX_GROUP_KEYS];
    uint32_t stride[SDB_MAX_GROUP_KEYS];
    int32_t* out_keys;
    long long* out_sums;
    long long* out_counts;
    long long* out_n;
    long long* block_off;      // scratch: one entry per finalize block
    int64_t n_blocks;
};

// Scan, scatter and aggregation passes of TERM_PART (scratch layout in sdb_api.cpp).
struct PartParams {
    uint64_t n_groups;
    int32_t part_shift;
    uint32_t n_parts;
    uint32_t n_regions;        // blocks of the fused kernel
    uint32_t part_cap;
    const uint32_t* region_count;
    const uint32_t* rec_gid;
    const void* rec_val;
    int32_t rec_wide;
    uint32_t pad_;
    uint32_t* part_hist;       // [q * n_regions + b]: counts, then exclusive offsets within partition q
    uint32_t* part_count;      // records per partition
    uint32_t* part_start;      // n_parts + 1 entries
    uint32_t* chunk_start;     // n_parts + 1 entries; [n_parts] = total work items
    uint32_t* sorted_gid;
    void* sorted_val;
    unsigned long long* item_sum;   // per work item partial tables: [item * groups per partition + k]
    uint32_t* item_cnt;
    unsigned long long* sums;
    unsigned long long* counts;
};

// Count and scatter passes of the sliced hash probe. Block b of the grid
// reads fact rows [b * rows_per_block, (b + 1) * rows_per_block) in both.
struct SliceParams {
    const int32_t* cols[SDB_MAX_FACT_COLS];
    int64_t n;                 // fact rows
    int64_t rows_per_block;    // a multiple of kSliceChunk; columns are 16-byte aligned
    int32_t key_col;           // the probe's fact key column
    int32_t val_col;           // the aggregate's (first) column
    int32_t val2_col;          // its second column (MUL, SUB, ADD), or -1
    int32_t n_preds;
    int32_t bits;              // 2^bits partitions, 1 .. SDB_MAX_SLICE_BITS
    int32_t pred_col[kMaxStages];
    RangeTest pred[kMaxStages];
    uint32_t* hist;            // [q * grid + b]: passing rows, then their offset within partition q
    uint32_t* part_count;      // rows per partition
    uint32_t* part_start;      // n_parts + 1 entries; [n_parts] = all passing rows
    uint32_t* chunk_start;     // n_parts + 1 entries (written by the shared scan, unused)
    int32_t* out_key;          // partitioned keys and values, all passing rows
    int32_t* out_val;
    int32_t* out_val2;         // val2_col >= 0: the second operands
    // tile order of the fused launch over them: its tiles of tile_rows rows;
    // XCD x (x = q mod 8) walks the tiles whose first row lies in partition q
    int64_t tile_rows;
    uint32_t* tile_base;       // n_parts entries: rank of partition q's first tile among its XCD's tiles
    int32_t* tile_map;         // n_vtiles entries: [8 * rank + x] = tile, -1 where XCD x has fewer tiles
    int64_t n_vtiles;
    // pre-filter: rows whose key the table's pass filter rejects are dropped
    // by the count pass, which writes one byte per 4-row group (bit j: row
    // 4 g + j kept) for the scatter pass; filt null: no pre-filter
    const uint32_t* filt;
    uint64_t filt_bits;
    int32_t filt_kind;
    int32_t filt_key_min;
    uint8_t* keep;             // ceil(n / 4) bytes
};

// ---- launchers (sdb_kernels.hip) -----------------------------------------
hipError_t launch_fill_u32(uint32_t* p, uint64_t n_words, uint32_t value, hipStream_t s);
hipError_t launch_fill_u64(unsigned long long* p, uint64_t n, hipStream_t s);
hipError_t launch_zero_pair(unsigned long long* a, unsigned long long* b, uint64_t n, hipStream_t s);
// statistics pass of every table: per-block partials, then the combined
// statistics block of each table (also copied to bb.host_stats when set)
hipError_t launch_build_stats(const BuildBatch& bb, hipStream_t s);
// table fill, then dense scatter + pass bitmap or hash inserts, of every table
hipError_t launch_build_tables(const BuildBatch& bb, hipStream_t s);
// copies every table's statistics block to bb.host_stats (one launch)
hipError_t launch_export_stats(const BuildBatch& bb, hipStream_t s);
// copies words0 words from src0, then words1 from src1, to dst (pinned host
// memory, device address) in one launch
hipError_t launch_copy_out(const uint32_t* src0, uint32_t words0, const uint32_t* src1, uint32_t words1,
                           uint32_t* dst, hipStream_t s);
// Planner sampling: pass-pattern histograms (n_ranges x 2^nstages uint32: the
// sampled rows split into n_ranges equal runs) and per-stage key histograms
// (kMaxStages x kKeyBuckets uint32), both zeroed first (by one fill where the
// key histograms follow the pattern histograms' 2^kMaxStages words).
hipError_t launch_sample(const FusedParams& p, int64_t step, int64_t n_sample, int32_t n_ranges,
                         uint32_t* pattern_hist, uint32_t* key_hist, hipStream_t s);
// Returns the kernel's occupancy (blocks per CU) for the given instance, or <= 0 if
// the instance does not exist.
// `unroll`: the instance whose stage loop is written out kUnrollStages times
// (plans of at most that many stages, 4-row items, 2 per lane, blocks of
// kMaxBlock or kBigBlock, no eager loads).
int fused_blocks_per_cu(int vector, int ipt, int terminal, int eager, int block, int unroll, size_t lds_bytes);
hipError_t launch_fused(const FusedParams& p, int vector, int ipt, int terminal, int eager, int unroll, int grid,
                        int block, size_t lds_bytes, hipStream_t s);
hipError_t launch_rank_build(const RankParams& rp, hipStream_t s);
// kernel-at-a-time run of the stages and aggregate of p (device tables only)
hipError_t launch_unfused(const FusedParams& p, uint8_t* flags, uint32_t* gid, hipStream_t s);
hipError_t launch_handoff(const FusedParams& p, uint8_t* flags, uint32_t* gid, hipStream_t s);

struct ReadParams {
    const int32_t* cols[SDB_MAX_FACT_COLS];
    int32_t n_cols;
    int32_t pad_;
    int64_t n;
    unsigned long long* out;
};
hipError_t launch_read_columns(const ReadParams& p, int grid, hipStream_t s);
hipError_t launch_xcd_merge(const unsigned long long* xtab, int copies, uint64_t n_groups,
                            unsigned long long* sums, unsigned long long* counts, hipStream_t s);
hipError_t launch_finalize(const FinalizeParams& fp, hipStream_t s);
hipError_t launch_part_passes(const PartParams& pp, hipStream_t s);
// count pass, per-partition offsets, scatter pass over `grid` blocks
hipError_t launch_slice_partition(const SliceParams& sp, int grid, hipStream_t s);

// the fixed run scratch of sdb_run_star_query_noalloc: its device address on
// the calling thread's current device
constexpr int kNoallocMaxDevices = 64;
constexpr uint64_t kNoallocScratchBytes = (uint64_t)SDB_NOALLOC_SCRATCH_BYTES;
hipError_t noalloc_scratch(void** out);

}  // namespace sdb
