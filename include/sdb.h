/*
 * sdb.h -- C ABI of libsdb, a fused star-schema query engine for one AMD
 * Instinct MI355X (gfx950).
 *
 * The library evaluates the query shape the paper studies (Sections 3.3, 4.2
 * and 4.3): one pass over int32 fact columns that applies literal predicates
 * on fact columns, probes lookup tables built from filtered dimension tables,
 * gathers dimension attributes as group keys, and ends in a scalar SUM or a
 * GROUP BY ... SUM over 64-bit integers.
 *
 * Conventions for every entry point
 *  - Plain C structs and pointers only. "device" pointers point to GPU memory
 *    (hipMalloc / torch CUDA tensors); "host" pointers to CPU memory.
 *  - The caller owns every buffer: fact and dimension columns, the dimension
 *    workspace, the planner and finalize scratch, and all outputs. They must
 *    stay valid until the work queued on the stream has finished. The library
 *    allocates no device memory and keeps no global mutable state besides a
 *    per-thread error string, the per-thread measurement events of
 *    sdb_set_fused_events, a per-device properties cache and a 96 KB pinned,
 *    coherent host buffer per calling thread (allocated on the first build or
 *    sampled plan, kept while the thread lives) for the small reads those
 *    calls synchronize on, which kernels write directly; calls on different
 *    streams may run concurrently.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *  - Every call returns an sdb_status; nothing throws across the ABI.
 *    sdb_last_error() returns a message for the last failing call on the
 *    calling thread. Arguments are validated on the host before any launch.
 *  - All arithmetic is integer. Sums wrap modulo 2^64 and are reported as
 *    signed int64; the result does not depend on execution order.
 */
#ifndef SDB_H
#define SDB_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SDB_API __attribute__((visibility("default")))

#define SDB_ABI_VERSION 10

typedef enum sdb_status {
    SDB_OK = 0,
    SDB_INVALID_ARG = 1,          /* null pointer, negative size, index out of range, bad op code */
    SDB_UNSUPPORTED = 2,          /* a limit below is exceeded (columns, stages, payload domain) */
    SDB_CAPACITY = 3,             /* group count exceeds the caller's capacity or 2^31 - 1 */
    SDB_WORKSPACE_TOO_SMALL = 4,  /* workspace / scratch smaller than the required size */
    SDB_DUP_KEY = 5,              /* a dimension key occurs in more than one row */
    SDB_KEY_RANGE = 6,            /* DENSE forced but the key range exceeds the dense limit */
    SDB_HIP_ERROR = 7             /* a HIP runtime call or kernel launch failed */
} sdb_status;

/* Comparison operators of a predicate `column OP literal`. Literals are int64,
 * so a bound outside the int32 range is legal and simply always/never holds.
 * BETWEEN is inclusive on both ends: lo <= x <= hi (the paper lowers a BETWEEN
 * to the conjunction of its two bounds, Section 4.2). */
enum { SDB_OP_EQ = 0, SDB_OP_NE = 1, SDB_OP_LT = 2, SDB_OP_LE = 3,
       SDB_OP_GT = 4, SDB_OP_GE = 5, SDB_OP_BETWEEN = 6 };

/* Dimension lookup-table layouts (Section 3.3: a direct-mapped table indexed
 * by a dense primary key, or a double-sized open-addressing hash table). */
enum { SDB_TABLE_AUTO = 0, SDB_TABLE_DENSE = 1, SDB_TABLE_HASH = 2 };
/* pass filter of a hash table's keys (sdb_dim.filter_kind) */
enum { SDB_FILTER_NONE = 0, SDB_FILTER_BITMAP = 1, SDB_FILTER_BLOOM = 2 };
/* most bytes a hash table's pass filter takes in its workspace */
#define SDB_MAX_FILTER_BYTES (4ll << 20)

/* Aggregate expressions over fact columns a and b, computed in int64. */
enum { SDB_AGG_COL = 0, SDB_AGG_MUL = 1, SDB_AGG_SUB = 2, SDB_AGG_ADD = 3 };

/* Terminals (Sections 3.2, 3.3 and 4.3): one register accumulator per lane
 * reduced to one atomic per block; a block-private group table in LDS flushed
 * once per block; one global atomic per surviving row; or partitioned
 * aggregation for large group tables with many survivors (the fused kernel
 * appends (group id, value) records, later passes sort them by group-id range
 * and sum each range in LDS). */
enum { SDB_TERMINAL_AUTO = 0, SDB_TERMINAL_SCALAR = 1, SDB_TERMINAL_LDS = 2,
       SDB_TERMINAL_GLOBAL = 3, SDB_TERMINAL_PART = 4 };

#define SDB_MAX_DIM_COLS 8
#define SDB_MAX_DIM_PREDS 4
#define SDB_MAX_PAYLOADS 3
#define SDB_MAX_FACT_COLS 16
#define SDB_MAX_FACT_PREDS 8
#define SDB_MAX_JOINS 6
#define SDB_MAX_GROUP_KEYS 4
#define SDB_MAX_STAGES (SDB_MAX_FACT_PREDS + SDB_MAX_JOINS)
/* row ranges of a plan whose stage order changes along the fact table */
#define SDB_MAX_SEGMENTS 8
#define SDB_PLAN_SCRATCH_BYTES 81920
/* fact columns the fused kernel can load eagerly (sdb_plan.eager) */
#define SDB_MAX_EAGER 4

/* One predicate. `col` indexes the owning descriptor's `cols[]`. `hi` is
 * used by SDB_OP_BETWEEN only. */
typedef struct sdb_pred {
    int32_t col;
    int32_t op;
    int64_t lo;
    int64_t hi;
} sdb_pred;

/* A dimension table to turn into a lookup table.
 *  key          device, n_rows int32 primary keys (must be distinct)
 *  cols[]       device, n_rows int32 each: attribute columns referenced by
 *               preds[].col and payload_cols[]
 *  preds[]      conjunctive filter on the dimension rows (Section 3.3)
 *  payload_cols attributes to gather for passing rows (group keys), 0..3
 *  kind         SDB_TABLE_*; AUTO picks DENSE when the key range is at most
 *               max(2 * n_rows, 1024) slots, or when the dense table fits
 *               dense_budget_bytes, else HASH (the paper checks the key range
 *               at run time and falls back to a hash table, 4.3)
 *  load_factor  HASH only; 0 means 0.5 (the paper's double-sized table)
 *  dense_budget_bytes  the memory budget of that runtime choice: a dense
 *               table (packed map plus pass bitmap) of at most this many
 *               bytes is built whatever its key range (one load per probe
 *               instead of a hash chain, paid for in memory); 0: the key-range
 *               rule alone. sdb_dim_required_bytes grows to hold it. */
typedef struct sdb_dim_desc {
    const int32_t* key;
    int64_t n_rows;
    int32_t n_cols;
    const int32_t* cols[SDB_MAX_DIM_COLS];
    int32_t n_preds;
    sdb_pred preds[SDB_MAX_DIM_PREDS];
    int32_t n_payloads;
    int32_t payload_cols[SDB_MAX_PAYLOADS];
    int32_t kind;
    double load_factor;
    int64_t dense_budget_bytes;
} sdb_dim_desc;

/* A built lookup table: a plain handle into the caller's workspace.
 * A passing row's code is sum_p (payload_p - payload_min[p]) * payload_div[p]
 * with payload_div of the last payload 1; `domain` codes exist.
 *  DENSE: map[key - key_min] is the code (width bytes) of a passing row,
 *         `sentinel` (all ones of the width minus one) for a filtered row, or
 *         all ones for a key no row holds, so a code >= sentinel means "no
 *         passing row"; bit (key - key_min) of the bitmap `bits` (32-bit
 *         words) is set iff a passing row holds that key.
 *  HASH:  n_slots = 2^hash_bits 8-byte slots {low 32 bits: key, high 32
 *         bits: code + 1, or 0xFFFFFFFF for a filtered row}; a slot with high
 *         half 0 is empty. Slot of key k starts at (k * 0x9E3779B1 mod 2^32)
 *         >> (32 - hash_bits) (Fibonacci hashing) and probes linearly.
 *         Beside the slots, a pass filter of filter_bits bits (32-bit words at
 *         `filter`) that holds every passing row's key, so a fact key it
 *         rejects cannot pass the join (Section 3.3's filtered build, turned
 *         into a test that needs no probe):
 *           SDB_FILTER_BITMAP: bit (key - key_min) is set iff a passing row
 *             holds that key (filter_bits = key range), exact;
 *           SDB_FILTER_BLOOM: a blocked Bloom filter for key ranges too wide
 *             for a bitmap: m = (k ^ k >> 16) * 0x85EBCA6B, m ^= m >> 13,
 *             m *= 0xC2B2AE35, m ^= m >> 16 (mod 2^32: the 32-bit finalizer
 *             of MurmurHash3); word
 *             m mod (filter_bits / 32) holds bits t >> 27, (t >> 22) & 31 and
 *             (t >> 17) & 31 of t = rotl(m, 16) * 0x9E3779B1, all set for a
 *             passing key (false positives, no false negatives).
 *         The filter takes at most SDB_MAX_FILTER_BYTES (8 bits per row up to
 *         that); SDB_FILTER_NONE on handles that carry none. */
typedef struct sdb_dim {
    int32_t kind;                 /* SDB_TABLE_DENSE or SDB_TABLE_HASH */
    int32_t width;                /* DENSE: 1, 2 or 4 bytes per entry; HASH: 8 */
    int64_t n_rows;
    int64_t n_pass;               /* rows that pass the dimension predicates */
    int32_t key_min;              /* over all rows (0 when n_rows == 0) */
    int32_t key_max;
    int32_t pass_key_min;         /* over passing rows (0 and -1 when none pass) */
    int32_t pass_key_max;
    uint64_t n_slots;
    int32_t hash_bits;
    uint32_t sentinel;
    uint64_t domain;
    int32_t n_payloads;
    int32_t payload_min[SDB_MAX_PAYLOADS];     /* over passing rows */
    uint32_t payload_radix[SDB_MAX_PAYLOADS];  /* max - min + 1 over passing rows; 1 if none pass */
    uint64_t payload_div[SDB_MAX_PAYLOADS];
    void* map;                    /* device, inside the workspace */
    void* stats;                  /* device, inside the workspace */
    void* bits;                   /* DENSE: device pass bitmap inside the workspace; HASH: NULL */
    void* filter;                 /* HASH: device pass filter inside the workspace; DENSE: NULL */
    uint64_t filter_bits;         /* bits of the filter (a multiple of 32 for BLOOM) */
    int32_t filter_kind;          /* SDB_FILTER_* */
    int32_t reserved_;            /* 0 */
} sdb_dim;

/* What a built lookup table holds, as sdb_dim_info reports it: the layout the
 * build chose (Section 4.3: the key-range check picks a direct-mapped map or
 * falls back to a hash table) and the ranges the plan derives group radices
 * from (Section 4.3: the group table is sized from the payload domains). */
typedef struct sdb_dim_summary {
    int32_t kind;                 /* SDB_TABLE_DENSE or SDB_TABLE_HASH */
    int32_t width;                /* bytes per map entry (1, 2, 4) or per hash slot (8) */
    int64_t n_rows;
    int64_t n_pass;               /* rows that pass the dimension predicates */
    int32_t key_min;              /* over all rows (0 and -1 when there are none) */
    int32_t key_max;
    int32_t pass_key_min;         /* over passing rows (0 and -1 when none pass) */
    int32_t pass_key_max;
    int32_t pass_keys_contiguous; /* 1: the passing keys are exactly pass_key_min..pass_key_max
                                     (the table can be probed as a key range) */
    int32_t n_payloads;
    uint64_t n_slots;             /* map entries (key range) or hash slots */
    uint64_t table_bytes;         /* device bytes the lookup table occupies in the workspace:
                                     map plus pass bitmap, or hash slots */
    double occupancy;             /* n_rows / n_slots (a hash table's load factor); 0 without slots */
    int32_t payload_min[SDB_MAX_PAYLOADS];     /* over passing rows */
    int32_t payload_max[SDB_MAX_PAYLOADS];     /* payload_min + radix - 1 */
    uint32_t payload_radix[SDB_MAX_PAYLOADS];
    int32_t filter_kind;          /* HASH: SDB_FILTER_* of its pass filter; DENSE: SDB_FILTER_NONE */
    uint64_t domain;              /* product of the payload radices: distinct codes */
    uint64_t filter_bytes;        /* device bytes of that filter (not part of table_bytes) */
} sdb_dim_summary;

typedef struct sdb_join {
    int32_t fact_key_col;         /* index into sdb_query.cols[] */
    const sdb_dim* dim;           /* host pointer to a built handle */
} sdb_join;

typedef struct sdb_group_key {
    int32_t join;                 /* index into sdb_query.joins[] */
    int32_t payload;              /* index into that dimension's payloads */
} sdb_group_key;

typedef struct sdb_agg {
    int32_t kind;                 /* SDB_AGG_* */
    int32_t a;                    /* index into sdb_query.cols[] */
    int32_t b;                    /* index into sdb_query.cols[] (ignored for COL) */
} sdb_agg;

/* A star query over n_fact rows (the fact table is the spine: predicates
 * narrow the live rows, probes drop misses and filtered rows, gathers pull
 * group keys, the terminal consumes the survivors; Section 4.2).
 * The force_* fields override the planner (0 = automatic):
 *  force_terminal  SDB_TERMINAL_*
 *  force_ipt       items per lane per loop iteration (1, 2 or 4)
 *  force_vector    1: 4-row items with 128-bit loads (columns must be 16-byte
 *                  aligned); -1: 1-row items
 *  force_order     1: keep query order (predicates, then joins), no sampling
 *  grid_blocks     blocks of the fused kernel
 *  force_lds       -1: every probe uses the device table (no LDS staging);
 *                  2: LDS maps and bitmaps, but no rank tables; 3: rank tables
 *                  for every deferred bitmap stage whose tables fit
 *  force_xcd       -1: no per-XCD group-table copies; 1: use them
 *  force_block     threads per block of the fused kernel: 64, 128, 256, 512
 *                  or 1024 (1024 needs 4-row items, ipt 1 or 2, no eager loads)
 *  force_eager     -1: every column is loaded when its stage is reached, for
 *                  the items that still hold a live row; k in 1..SDB_MAX_EAGER:
 *                  the first k columns in order of use are loaded together
 *                  when the items start (needs 4-row items and ipt 1 or 2)
 *  force_range     which probes run as a key range (sdb_plan.stage_range):
 *                  0: those that would otherwise look up a table in device
 *                  memory; 1: every one that can; -1: none
 *  force_coarse    coarse LDS pre-filters for dense tables left in device
 *                  memory (SDB_LDS_COARSE): 0: chosen by the planner; -1:
 *                  none; k in 1..SDB_MAX_COARSE_SHIFT: every such table whose
 *                  coarse bitmap of 2^k slots per bit fits in LDS
 *  force_slice     the hash probe over table slices (sdb_plan.slice_bits):
 *                  0: chosen by the planner; -1: never; 1: wherever the
 *                  query allows it
 *  force_unroll    the fused kernel with its stage loop written out
 *                  (sdb_plan.unroll): 0: wherever the plan allows it; -1:
 *                  never
 *  force_segments  stage orders per row range (sdb_plan.n_segments): 0: the
 *                  planner's choice; -1: one order for the whole table; 1:
 *                  a range gets an order of its own wherever its sampled
 *                  rows favour one, however small the modelled gain
 *  force_window    LDS windows (SDB_LDS_WINDOW): 0: the planner's choice
 *                  (none: measured on MI355X, a window does not pay); -1:
 *                  none; 1: the largest window that fits without lowering
 *                  the blocks per CU, for the dense device-memory stage it
 *                  serves most; k >= 2: the same with at most 128 * k slots
 *  force_prefilter the sliced hash probe's pre-filter (sdb_plan.slice_prefilter):
 *                  0: the planner's choice; -1: never; 1: whenever the plan
 *                  slices a hash probe into a table with a pass filter */
typedef struct sdb_query {
    int64_t n_fact;
    int32_t n_cols;
    const int32_t* cols[SDB_MAX_FACT_COLS];
    int32_t n_preds;
    sdb_pred preds[SDB_MAX_FACT_PREDS];
    int32_t n_joins;
    sdb_join joins[SDB_MAX_JOINS];
    int32_t n_group_keys;
    sdb_group_key group_keys[SDB_MAX_GROUP_KEYS];
    sdb_agg agg;
    int32_t force_terminal;
    int32_t force_ipt;
    int32_t force_vector;
    int32_t force_order;
    int32_t grid_blocks;
    int32_t force_lds;
    int32_t force_xcd;
    int32_t force_eager;
    int32_t force_block;
    int32_t force_range;
    int32_t force_coarse;
    int32_t force_slice;
    int32_t force_unroll;
    int32_t force_window;
    int32_t force_segments;
    int32_t force_prefilter;
} sdb_query;

/* Where a probe looks its table up (sdb_plan.stage_lds):
 *  GLOBAL  the map or hash table in device memory, one gather per live row;
 *  MAP     the whole dense map copied into each block's LDS;
 *  BITS    the dense table's pass bitmap copied into LDS; the group-key code,
 *          if any, is gathered from the device map for the rows that survive
 *          every stage (stage_defer >= 0) or right after the bit test;
 *  RANK    the pass bitmap, the number of passing slots before every 64-slot
 *          group, and the codes of the passing slots alone in slot order, all
 *          copied into LDS (sdb_run_star_query derives the last two in its
 *          run scratch): a passing key's code is the code at its rank, so the
 *          group key needs no device-memory gather. Its LDS footprint leaves room
 *          for one block per CU, so the planner pairs it with blocks of 1024;
 *  COARSE  the map stays in device memory, but a coarse pass bitmap sits in
 *          LDS: bit j is set iff any of the 2^stage_coarse[s] slots
 *          j * 2^stage_coarse[s] ... holds a passing key (sdb_run_star_query
 *          derives it from the pass bitmap in its run scratch). A row whose
 *          bit is clear dies without touching device memory; the others
 *          gather their code from the map as with GLOBAL;
 *  WINDOW  the pass bitmap of slots stage_window_lo[s] ...
 *          stage_window_lo[s] + stage_window_slots[s] - 1 sits in LDS (a
 *          window of the key range, placed where the sampled keys are
 *          densest): a row whose key falls in it and whose bit is clear
 *          dies without touching device memory; every other row gathers its
 *          code from the device map as with GLOBAL (a passing row in the
 *          window only for its group key). */
enum { SDB_LDS_GLOBAL = 0, SDB_LDS_MAP = 1, SDB_LDS_BITS = 2, SDB_LDS_RANK = 3, SDB_LDS_COARSE = 4,
       SDB_LDS_WINDOW = 5 };
/* log2 of the slots one coarse bit covers: 1 ... SDB_MAX_COARSE_SHIFT */
#define SDB_MAX_COARSE_SHIFT 5

/* The one-pass plan. Stages run in the listed order; each is a fact
 * predicate (kind 0, index into preds[]) or a join probe (kind 1, index into
 * joins[]). Group id = sum_k (key_k - key_min[k]) * stride[k] with the last
 * key's stride 1, so ascending group ids are ascending key tuples.
 * With xcd_copies > 0 the global terminal accumulates into that many private
 * copies of the group table (one per XCD, in the run scratch) that a second
 * kernel adds into the outputs.
 * With slice_bits > 0 the hash probe of stage slice_stage runs over table
 * slices (the L2-resident lookup tables of Section 3.3, extended to a hash
 * table larger than the caches): a count pass and a scatter pass, slice_grid
 * blocks each, evaluate the fact predicates and write every passing row's
 * probe key and aggregate value into 2^slice_bits partitions by the top
 * slice_bits bits of the key's 32-bit hash, which also selects the table
 * slice its home slot lies in; the fused kernel then runs the probe alone
 * over the partitioned records, each XCD taking the partitions q with
 * q mod 8 equal to its index in turn (a tile map built after the count pass
 * orders the kernel's tiles so; results do not depend on that order), so
 * the slots one XCD reads at any time fit in its L2. The run scratch then
 * holds 8 bytes per fact row for the partitioned keys and values (12 for a
 * two-column aggregate, whose both operands travel with the key). With
 * slice_prefilter the count pass also drops rows whose key the table's pass
 * filter rejects and records which rows it keeps (one byte per 4 rows in the
 * run scratch), so the scatter pass writes and the fused kernel probes only
 * rows that can pass the join; the planner takes it when the join's sampled
 * pass fraction, with the filter's false positives added, is at most 0.7
 * (each dropped row saves a scatter write and a probe, each row costs one
 * L2-resident filter read). It needs
 * one hash probe, all other stages fact predicates, and the columns those
 * passes read 16-byte aligned. ipt, vector, eager (0), block, grid,
 * lds_bytes and the terminal fields describe that fused launch. */
typedef struct sdb_plan {
    int32_t n_stages;
    int32_t stage_kind[SDB_MAX_STAGES];
    int32_t stage_index[SDB_MAX_STAGES];
    double stage_pass[SDB_MAX_STAGES];    /* pass fraction on the sample among the sampled rows that
                                             pass every earlier stage (conditional), or the estimate
                                             used (the dimension's pass fraction) without a sample */
    double stage_pass_alone[SDB_MAX_STAGES];  /* the stage's pass fraction on the sample by itself */
    int32_t stage_lds[SDB_MAX_STAGES];    /* SDB_LDS_* */
    int32_t stage_defer[SDB_MAX_STAGES];  /* 0: an LDS_BITS stage whose code is gathered after all
                                             stages; -1 otherwise */
    int32_t stage_range[SDB_MAX_STAGES];  /* 1: a probe run as `fact key BETWEEN pass_key_min AND
                                             pass_key_max` (its dimension's passing keys are exactly
                                             that range and it feeds no group key; Section 3.2's
                                             date-range scan, generalized); 0 otherwise */
    int32_t stage_coarse[SDB_MAX_STAGES]; /* SDB_LDS_COARSE: log2 of the slots per coarse bit; else 0 */
    int32_t stage_window_lo[SDB_MAX_STAGES];    /* SDB_LDS_WINDOW: first slot (a multiple of 128); else 0 */
    int32_t stage_window_slots[SDB_MAX_STAGES]; /* SDB_LDS_WINDOW: slots (a multiple of 128); else 0 */
    double stage_window_cover[SDB_MAX_STAGES];  /* SDB_LDS_WINDOW: sampled fraction of the stage's fact
                                                   keys that fall in the window; else 0 */
    int64_t sampled_rows;                 /* 0 when no sample was taken */
    double est_cost;                      /* cost model value of the chosen order */
    int32_t terminal;
    int32_t ipt;
    int32_t vector;                       /* 1: 4-row items with 128-bit loads */
    int32_t eager;                        /* columns loaded together when items start (first in order of use) */
    int32_t block;
    int32_t grid;                         /* 0: chosen at launch */
    int32_t xcd_copies;
    int32_t lds_bytes;                    /* dynamic LDS per block */
    int32_t part_shift;                   /* PART: partition of group g is g >> part_shift */
    int32_t n_parts;
    int32_t part_subs;                    /* PART: record regions per fused-kernel block (1 .. 4): wave
                                             w appends to region w mod part_subs of its block */
    int64_t part_cap;                     /* PART: records per region */
    int32_t n_group_keys;
    int32_t key_min[SDB_MAX_GROUP_KEYS];
    uint32_t radix[SDB_MAX_GROUP_KEYS];
    uint64_t stride[SDB_MAX_GROUP_KEYS];
    uint64_t n_groups;                    /* product of radices; 1 without GROUP BY */
    int64_t run_scratch_bytes;            /* device scratch sdb_run_star_query needs */
    int32_t slice_bits;                   /* 0: no sliced probe; else 1 .. SDB_MAX_SLICE_BITS */
    int32_t slice_stage;                  /* stage of the sliced hash probe (slice_bits > 0) */
    int32_t slice_grid;                   /* blocks of the count and scatter passes */
    int32_t slice_prefilter;              /* 1: the count pass also tests each row's key against the
                                             table's pass filter and keeps only rows it lets through
                                             (one bit per row for the scatter pass), so rows that
                                             cannot pass the join are neither partitioned nor
                                             probed; 0 otherwise */
    int32_t unroll;                       /* 1: the fused kernel's instance with its stage loop
                                             written out four times (stage parameters stay in
                                             scalar registers across tiles); allowed for plans of
                                             at most 4 stages, 4-row items, ipt 2, blocks of 512
                                             or 1024, no eager loads and no hash-table probe;
                                             0 otherwise */
    int32_t n_segments;                   /* 1, or 2 .. SDB_MAX_SEGMENTS row ranges that run the
                                             stages in orders of their own (mid-scan reordering:
                                             the sample is split by row range, each range's order
                                             is chosen on its own pass patterns, and neighbours
                                             with equal orders are merged); the fused kernel is
                                             launched once per segment over its rows, every
                                             launch adding into the same terminal */
    int32_t segment_order[SDB_MAX_SEGMENTS][SDB_MAX_STAGES];   /* segment g runs the plan's stages
                                             (positions 0 .. n_stages - 1) in this order */
    int64_t segment_start[SDB_MAX_SEGMENTS + 1];   /* first fact row of each segment (multiples of
                                             4096); segment_start[n_segments] = n_fact */
} sdb_plan;
/* most partitions of the sliced hash probe: 2^SDB_MAX_SLICE_BITS */
#define SDB_MAX_SLICE_BITS 10

/* ---- errors and ABI ---------------------------------------------------- */

/* Message for the last failing call on this thread ("" if none). The string
 * stays valid until the next call on the same thread. */
SDB_API const char* sdb_last_error(void);

/* Fixed name of a status code. */
SDB_API const char* sdb_status_string(int32_t status);

/* SDB_ABI_VERSION of the built library. */
SDB_API int32_t sdb_abi_version(void);

/* Writes sizeof of sdb_pred, sdb_dim_desc, sdb_dim, sdb_join, sdb_group_key,
 * sdb_agg, sdb_query, sdb_plan, sdb_dim_summary (in that order) to
 * sizes[0..n-1], n <= 9, so a binding can check its struct layout. Host
 * only. */
SDB_API sdb_status sdb_struct_sizes(int64_t* sizes, int32_t n);

/* ---- dimension build (separate from the fused pass, Section 4.2) ------- */

/* Host only. Workspace bytes sdb_build_dim needs for `desc`: 256 bytes of
 * statistics, then the lookup table sized by an upper bound (a DENSE map of
 * max(2 * n_rows, 1024) 4-byte slots plus its pass bitmap, or
 * dense_budget_bytes plus 512 bytes of alignment when that is larger, and/or
 * a HASH table of next_pow2(n_rows / load_factor) 8-byte slots, padded to
 * 256 bytes, and its pass filter of min(max(next_pow2(n_rows), 256),
 * SDB_MAX_FILTER_BYTES) bytes). */
SDB_API sdb_status sdb_dim_required_bytes(const sdb_dim_desc* desc, int64_t* bytes);

/* Builds the lookup table for `desc` into `workspace` (device, 256-byte
 * aligned, workspace_bytes >= sdb_dim_required_bytes) on `stream`, and fills
 * `out` (host). Passes over the dimension rows: statistics (key range, pass
 * count, payload ranges), then the direct-mapped map (Section 3.3: one code
 * per key, the sentinel for a filtered row, all ones for an absent key; 1, 2
 * or 4 bytes by payload domain) and its pass bitmap, or the open-addressing
 * table (64-bit compare-and-swap inserts) and its pass filter (a bitmap over
 * the key range when that fits the filter's bytes, set through one byte per
 * key in the slot region before the slots are filled; else the Bloom filter,
 * set with atomics by the inserts).
 * Synchronizes the stream twice (to
 * read the statistics, then the duplicate-key check: a dense map must end
 * with one occupied slot per row).
 * Errors: INVALID_ARG, UNSUPPORTED (payload domain >= 2^32 - 2), KEY_RANGE,
 * WORKSPACE_TOO_SMALL, DUP_KEY, HIP_ERROR. */
SDB_API sdb_status sdb_build_dim(const sdb_dim_desc* desc, void* workspace,
                                 int64_t workspace_bytes, void* stream, sdb_dim* out);

/* sdb_build_dim for n_dims tables (0 <= n_dims <= SDB_MAX_JOINS) at once:
 * descs[d] is built into workspaces[d] (workspace_bytes[d] bytes) and
 * described in outs[d] (all arrays host). Every table's statistics pass runs
 * before the one synchronization that reads them, and every table's map
 * before the one that checks them, so a star query's tables cost two stream
 * synchronizations in all. Arguments of every table are checked before
 * anything launches. On error the message names the dimension index; the
 * outputs are then undefined. Errors: as sdb_build_dim. */
SDB_API sdb_status sdb_build_dims(int32_t n_dims, const sdb_dim_desc* descs, void* const* workspaces,
                                  const int64_t* workspace_bytes, void* stream, sdb_dim* outs);

/* Host only. Describes the table `dim` (a handle sdb_build_dim or
 * sdb_build_dims filled) in `out` (host): its layout, key ranges, pass count,
 * payload domains and pass filter, without touching the device (Sections 3.3
 * and 4.3: the direct-mapped or hash layout a build chose, and the domains
 * the group table is sized from). Errors: INVALID_ARG (null pointer, or a
 * handle whose fields contradict each other: unknown kind, a width or slot
 * count the kind does not allow, a pass count above the row count, a missing
 * map, a pass filter on a dense table, without its words, or of a size its
 * kind does not allow). */
SDB_API sdb_status sdb_dim_info(const sdb_dim* dim, sdb_dim_summary* out);

/* ---- planning ----------------------------------------------------------- */

/* Plans `q` (host) into `plan` (host): the runtime choices of Section 4.3
 * (key-range checks, the group table sized from the payload domains, the
 * terminal by group count) and the stage order of Section 4.2's fact-spine
 * lowering. Unless q->force_order is set, a sampling kernel evaluates every
 * stage over every ceil(n_fact / 65536)-th fact row and records, per sampled
 * row, which stages it passes (a histogram over the 2^stages pass patterns)
 * and, when a window is forced, per dense-table stage a 256-bucket histogram
 * of its fact keys over the table's key range; this needs `scratch` (device,
 * >= SDB_PLAN_SCRATCH_BYTES) and synchronizes `stream` once. With
 * force_order set, scratch and stream are unused, no GPU call is made and
 * the stages keep query order (predicates, then joins), with the
 * dimensions' pass fractions taken as independent estimates. The plan fixes:
 * which small dense tables are staged in LDS (whole maps, pass bitmaps or
 * rank tables) and which probes run as key ranges; the stage order with the
 * least modelled cost (fact columns streamed at 128-byte line granularity
 * plus each stage's lookups for the rows that reach it, the rows reaching a
 * stage counted exactly from the sampled pass patterns, so correlated
 * predicates are priced as measured; every order is tried up to 7 stages, a
 * greedy rank on conditional pass fractions beyond); when forced, an LDS
 * window for the dense device-memory stage whose sampled keys it serves
 * most (4-row items then run in blocks of 1024); group radices and strides
 * from the built
 * tables' payload ranges; the terminal (scalar without GROUP BY, LDS when
 * the group table fits a block's LDS, partitioned when at least a million
 * rows survive, 16 or more per group, else global, with per-XCD copies when
 * enough rows survive);
 * items per lane, block size, eager columns, and for the partitioned
 * terminal the grid and region sizes; whether the hash probe runs over
 * table slices (chosen for a table of at least 16 MiB and at least 2^24 fact
 * rows, when the query allows it). Errors: INVALID_ARG, UNSUPPORTED,
 * CAPACITY, WORKSPACE_TOO_SMALL, HIP_ERROR. */
SDB_API sdb_status sdb_plan_star_query(const sdb_query* q, void* scratch, int64_t scratch_bytes,
                                       void* stream, sdb_plan* plan);

/* ---- the fused pass ----------------------------------------------------- */

/* Runs `q` with `plan` (from sdb_plan_star_query for this query and these
 * tables) as one fused probe-filter-aggregate kernel (Sections 3.2 and 4.2),
 * all queued on `stream` (asynchronous): rank tables are derived first when
 * the plan stages any, a sliced hash probe's count and scatter passes come
 * before the fused kernel, and the partitioned terminal's sort and sum passes or
 * the per-XCD copies' merge follow the fused kernel. Only kernels are
 * enqueued (no memset, copy or synchronization), so the call can be captured
 * in a HIP graph. The outputs are zeroed first (or, with per-XCD copies, the
 * copies are zeroed and then added into them).
 * sums/counts: device int64[plan->n_groups], indexed by group id;
 * n_groups_capacity >= plan->n_groups. Without GROUP BY, sums[0] and
 * counts[0] hold the total and the live row count. scratch: device,
 * 256-byte aligned, >= plan->run_scratch_bytes (may be NULL when that is 0).
 * Errors: INVALID_ARG, CAPACITY, WORKSPACE_TOO_SMALL, HIP_ERROR (launch
 * failures only). */
SDB_API sdb_status sdb_run_star_query(const sdb_query* q, const sdb_plan* plan,
                                      int64_t* sums, int64_t* counts,
                                      int64_t n_groups_capacity, void* scratch,
                                      int64_t scratch_bytes, void* stream);

/* Size of the fixed run scratch of sdb_run_star_query_noalloc: 64 MiB per
 * device, held from the library's first use of that device until the
 * process ends. */
#define SDB_NOALLOC_SCRATCH_BYTES (64ll << 20)

/* For callers that cannot allocate device memory (code under HIP stream
 * capture, tight serving loops, harnesses that forbid hipMalloc): as
 * sdb_run_star_query, with the run scratch taken from a fixed array of
 * SDB_NOALLOC_SCRATCH_BYTES that the library holds on every device it runs
 * on, instead of a caller buffer. The caller still owns the outputs. The
 * call allocates nothing: no hipMalloc, hipFree or allocating library call
 * (its first call on a device looks the array's device address up once).
 * The array belongs to the device, not to the call: every call on a device
 * uses the same array, so calls whose work overlaps on one device (two
 * streams, or two host threads) race and give undefined results; calls one
 * after another on one stream are safe, each clearing what it needs.
 * Plans whose run_scratch_bytes exceed the array (the partitioned terminal
 * or the sliced hash probe at large row counts, per-XCD copies of more than
 * 4 Mi groups) are refused with SDB_WORKSPACE_TOO_SMALL before any launch;
 * plan such a query with force_terminal = SDB_TERMINAL_GLOBAL, force_xcd =
 * -1 and force_slice = -1, which leaves only the small rank and coarse
 * tables in the scratch. Errors: as sdb_run_star_query. */
SDB_API sdb_status sdb_run_star_query_noalloc(const sdb_query* q, const sdb_plan* plan, int64_t* sums,
                                              int64_t* counts, int64_t n_groups_capacity, void* stream);

/* Measurement hook, host only. With both events non-NULL (hipEvent_t
 * handles the caller created and owns), every later sdb_run_star_query on
 * this thread records `start` on its stream just before the fused kernel and
 * `stop` just after it (before any terminal pass), so the elapsed time
 * between them is that kernel's duration; with a sliced hash probe `start`
 * comes before its count pass, so the time covers both passes and the
 * kernel. NULL, NULL turns it off. */
SDB_API sdb_status sdb_set_fused_events(void* start, void* stop);

/* Measurement only: the plain streaming read the fused pass is compared
 * with (the practical bandwidth ceiling of reading fact columns). Adds every
 * int32 of the n_cols columns of n rows (host array of device pointers, each
 * 16-byte aligned) into *sum (device int64[1], zeroed first), mod 2^64,
 * asynchronously on `stream`, with the fused kernel's load shape: 128-bit
 * non-temporal loads, two 4-row items per lane, four columns at a time, in
 * blocks of 512 threads, blocks_per_cu (1 to 4; 0: 2) per compute unit.
 * Errors: INVALID_ARG, HIP_ERROR. */
SDB_API sdb_status sdb_read_columns(const int32_t* const* cols, int32_t n_cols, int64_t n,
                                    int32_t blocks_per_cu, int64_t* sum, void* stream);

/* ---- baselines for the fusion ablation ---------------------------------- */

/* How sdb_run_star_query_baseline executes a query (Sections 4.1 and 4.2):
 *  SDB_BASELINE_PER_OPERATOR  kernel at a time: one kernel sets every row's
 *                             live flag, one kernel per stage reads its fact
 *                             column, the flags and the group ids and writes
 *                             them back, one kernel adds the live rows into
 *                             the outputs with device-scope atomics;
 *  SDB_BASELINE_GLOBAL_HANDOFF one fused kernel, one row per thread, whose
 *                             operators still hand the live flag and the
 *                             group id to each other through the per-row
 *                             arrays in global memory (the fused engine
 *                             before its register table). */
typedef enum {
    SDB_BASELINE_PER_OPERATOR = 0,
    SDB_BASELINE_GLOBAL_HANDOFF = 1
} sdb_baseline_mode;

/* Host only. Scratch bytes sdb_run_star_query_baseline needs for n_fact
 * rows: a live flag (1 byte) and a group id (4 bytes) per fact row, in two
 * 256-byte aligned parts. Errors: INVALID_ARG (null `bytes`, n_fact < 0). */
SDB_API sdb_status sdb_baseline_scratch_bytes(int64_t n_fact, int64_t* bytes);

/* Runs `q` in the stage order of `plan` the way `mode` says, asynchronously
 * on `stream`. Every table is read in device memory; the plan's LDS
 * placements, terminal, items per lane and block size are ignored. Results
 * equal sdb_run_star_query's. For measurement only: these are the slow rungs
 * of the fusion ablation. Arguments as sdb_run_star_query, with scratch
 * (device, 256-byte aligned, caller-owned) >= sdb_baseline_scratch_bytes(
 * q->n_fact). Errors: as sdb_run_star_query, and INVALID_ARG for an unknown
 * mode. */
SDB_API sdb_status sdb_run_star_query_baseline(const sdb_query* q, const sdb_plan* plan,
                                               int32_t mode, int64_t* sums, int64_t* counts,
                                               int64_t n_groups_capacity, void* scratch,
                                               int64_t scratch_bytes, void* stream);

/* ---- finalize ----------------------------------------------------------- */

/* Host only. Scratch bytes sdb_finalize_groups needs for `plan`. */
SDB_API sdb_status sdb_finalize_scratch_bytes(const sdb_plan* plan, int64_t* bytes);

/* Compacts the group table on the device (asynchronous, on `stream`): every
 * group with counts[g] > 0 in ascending group id order, which is ascending
 * lexicographic key order. out_keys: device int32[out_capacity][n_group_keys]
 * (the key values, i.e. payload codes plus payload minima); out_sums,
 * out_counts: device int64[out_capacity]; out_n: device int64[1], the number
 * of groups written. Without GROUP BY one row is written even when its count
 * is 0. out_capacity must be >= plan->n_groups. scratch: device,
 * >= sdb_finalize_scratch_bytes. Errors: INVALID_ARG, CAPACITY,
 * WORKSPACE_TOO_SMALL, HIP_ERROR. */
SDB_API sdb_status sdb_finalize_groups(const sdb_plan* plan, const int64_t* sums,
                                       const int64_t* counts, int32_t* out_keys,
                                       int64_t* out_sums, int64_t* out_counts,
                                       int64_t out_capacity, int64_t* out_n,
                                       void* scratch, int64_t scratch_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SDB_H */
