// Host runtime of libsdb: argument validation, dimension-table sizing and
// bookkeeping, the one-pass planner, and the C ABI declared in include/sdb.h.
// All device work is queued on the caller's stream through the launchers in
// sdb_kernels.hip; this file allocates no device memory.

#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "sdb_internal.h"

using namespace sdb;

namespace {

thread_local std::string g_error;
thread_local hipEvent_t g_fused_start = nullptr;   // sdb_set_fused_events
thread_local hipEvent_t g_fused_stop = nullptr;

sdb_status fail(sdb_status s, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_error = std::string(sdb_status_string(s)) + ": " + buf;
    return s;
}

sdb_status ok() {
    g_error.clear();
    return SDB_OK;
}

sdb_status hip_fail(hipError_t e, const char* what) {
    return fail(SDB_HIP_ERROR, "%s: %s", what, hipGetErrorString(e));
}

#define SDB_HIP(call, what)                              \
    do {                                                 \
        hipError_t e_ = (call);                          \
        if (e_ != hipSuccess) return hip_fail(e_, what); \
    } while (0)

// Pinned host staging for the few small device-to-host reads that the builds
// and the planner synchronize on (statistics, duplicate-key flags, sample
// counts). A copy into pageable memory is staged by the runtime and waited
// for copy by copy (30-40 us each on MI355X, seen in a kernel trace as gaps
// between the copies); copies into pinned memory queue on the stream behind
// the kernels and all complete with its one synchronization. One buffer per
// host thread, allocated on first use and kept while the thread lives (calls
// on one thread never overlap: each synchronizes before it returns); if the
// allocation fails the reads go to the caller's stack as before.
constexpr size_t kStagingBytes = 96 * 1024;
// planner scratch: pass-pattern histogram, then the per-stage key histograms
constexpr size_t kPatternBytes = sizeof(uint32_t) << kMaxStages;
constexpr size_t kKeyHistBytes = sizeof(uint32_t) * kMaxStages * kKeyBuckets;
static_assert(sizeof(DimStats) * SDB_MAX_JOINS <= kStagingBytes, "statistics staging");
static_assert(kPatternBytes + kKeyHistBytes <= kStagingBytes, "sample staging");
static_assert(kPatternBytes + kKeyHistBytes <= SDB_PLAN_SCRATCH_BYTES, "planner scratch");
thread_local void* t_staging = nullptr;
thread_local void* t_staging_dev = nullptr;
thread_local bool t_staging_failed = false;

// Pinned, coherent host buffer for the small reads the builds and the planner
// wait for; kernels write it directly (through its device address), so a read
// costs one small kernel rather than one copy per block read.
void* host_staging() {
    if (!t_staging && !t_staging_failed) {
        if (hipHostMalloc(&t_staging, kStagingBytes, hipHostMallocCoherent | hipHostMallocPortable) != hipSuccess) {
            t_staging = nullptr;
            t_staging_failed = true;
            (void)hipGetLastError();
        } else if (hipHostGetDevicePointer(&t_staging_dev, t_staging, 0) != hipSuccess || !t_staging_dev) {
            t_staging_dev = nullptr;   // the buffer still serves copies
            (void)hipGetLastError();
        }
    }
    return t_staging;
}

// The staging buffer's device address, or null (then reads go through copies).
void* host_staging_device() {
    return host_staging() ? t_staging_dev : nullptr;
}

inline uint64_t align_up(uint64_t x, uint64_t a) { return (x + a - 1) / a * a; }

inline uint64_t next_pow2(uint64_t x) {
    uint64_t p = 1;
    while (p < x) p <<= 1;
    return p;
}

// ---- predicates -----------------------------------------------------------

bool valid_op(int32_t op) { return op >= SDB_OP_EQ && op <= SDB_OP_BETWEEN; }

// Lowers `x OP literal(s)` with int64 literals to one unsigned range test over
// int32 values: pass <=> ((uint32)(x - lo) <= span) != negate.
RangeTest lower_pred(const sdb_pred& p) {
    const int64_t kMin = INT32_MIN, kMax = INT32_MAX;
    auto clamp = [&](int64_t v) { return std::min(std::max(v, kMin - 1), kMax + 1); };
    int64_t a = kMin, b = kMax;   // inclusive range that passes (before negation)
    int negate = 0;
    const int64_t v = clamp(p.lo);
    switch (p.op) {
        case SDB_OP_EQ: a = v; b = v; break;
        case SDB_OP_NE: a = v; b = v; negate = 1; break;
        case SDB_OP_LT: b = v - 1; break;
        case SDB_OP_LE: b = v; break;
        case SDB_OP_GT: a = v + 1; break;
        case SDB_OP_GE: a = v; break;
        case SDB_OP_BETWEEN: a = v; b = clamp(p.hi); break;
    }
    a = std::max(a, kMin);
    b = std::min(b, kMax);
    RangeTest t;
    if (a > b) {   // nothing is inside: "in" never holds, "not in" always holds
        t.lo = INT32_MIN;
        t.span = 0xFFFFFFFFu;
        t.negate = negate ? 0 : 1;
        return t;
    }
    t.lo = (int32_t)a;
    t.span = (uint32_t)(b - a);
    t.negate = negate;
    return t;
}

// ---- device properties ----------------------------------------------------

struct DeviceInfo {
    int cus = 0;
};

std::mutex g_dev_mu;
std::vector<DeviceInfo> g_dev;

sdb_status device_info(DeviceInfo* out) {
    int dev = 0;
    SDB_HIP(hipGetDevice(&dev), "hipGetDevice");
    std::lock_guard<std::mutex> lk(g_dev_mu);
    if ((int)g_dev.size() <= dev) g_dev.resize(dev + 1);
    if (g_dev[dev].cus == 0) {
        int cus = 0;
        SDB_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev),
                "hipDeviceGetAttribute");
        g_dev[dev].cus = cus;
    }
    *out = g_dev[dev];
    return SDB_OK;
}

// ---- dimension sizing -----------------------------------------------------

constexpr uint64_t kStatsBytes = 256;
// the smallest table region (a dense map of 1024 one-byte codes and its bitmap)
// holds several blocks' partial statistics
static_assert(sizeof(DimStats) * 4 <= 512, "statistics partials");

// dense tables within a memory budget: key ranges up to 2^31 slots
constexpr int64_t kMaxDenseBudget = 1ll << 36;
constexpr uint64_t kMaxDenseSlots = 1ull << 31;

uint64_t dense_slot_limit(int64_t n_rows) {
    return std::max<uint64_t>(2 * (uint64_t)n_rows, (uint64_t)kDenseSlack);
}

// map and pass bitmap (each region 256-byte aligned)
uint64_t dense_bytes(uint64_t slots, int width) {
    return align_up(slots * (uint64_t)width, 256) + align_up((slots + 31) / 32 * 4, 256);
}

double effective_lf(const sdb_dim_desc* d) {
    return d->load_factor > 0.0 ? d->load_factor : 0.5;
}

uint64_t hash_capacity(int64_t n_rows, double lf) {
    uint64_t need = (uint64_t)std::ceil((double)n_rows / lf);
    need = std::max<uint64_t>(need, (uint64_t)n_rows + 1);   // at least one empty slot
    return std::max<uint64_t>(next_pow2(need), 2);
}

// Bytes of a hash table's pass filter: 8 bits per row, a power of two from
// 256 bytes to SDB_MAX_FILTER_BYTES (an L2 holds the largest with room to
// spare for the stream that probes it).
uint64_t filter_bytes(int64_t n_rows) {
    return std::min<uint64_t>((uint64_t)SDB_MAX_FILTER_BYTES, std::max<uint64_t>(256, next_pow2((uint64_t)n_rows)));
}

// Why a handle's pass filter fields contradict its kind or key range, or ""
// when they agree.
std::string filter_problem(const sdb_dim* d) {
    char buf[160];
    if (d->reserved_ != 0) return "sdb_dim.reserved_ must be 0";
    if (d->filter_kind == SDB_FILTER_NONE) return "";
    if (d->kind != SDB_TABLE_HASH) return "only a hash table carries a pass filter";
    if (d->filter_kind != SDB_FILTER_BITMAP && d->filter_kind != SDB_FILTER_BLOOM) {
        snprintf(buf, sizeof buf, "bad pass filter kind %d", d->filter_kind);
        return buf;
    }
    if (!d->filter) return "pass filter without its words";
    const uint64_t b = d->filter_bits, max_bits = (uint64_t)SDB_MAX_FILTER_BYTES * 8;
    if (d->filter_kind == SDB_FILTER_BITMAP) {
        const uint64_t range = d->n_rows > 0 ? (uint64_t)((int64_t)d->key_max - (int64_t)d->key_min + 1) : 0;
        if (b == 0 || b != range || b > max_bits) {
            snprintf(buf, sizeof buf, "pass filter bitmap of %llu bits for a key range of %llu",
                     (unsigned long long)b, (unsigned long long)range);
            return buf;
        }
    } else if (b < 32 || b % 32 != 0 || ((b / 32) & (b / 32 - 1)) != 0 || b > max_bits) {
        snprintf(buf, sizeof buf, "pass filter (Bloom) of %llu bits is not 32 x a power of two up to %llu",
                 (unsigned long long)b, (unsigned long long)max_bits);
        return buf;
    }
    return "";
}

// Fraction of keys outside the filter's set that a Bloom filter of `bits`
// bits holding `n_keys` keys lets through: each key sets 3 bits of one
// 32-bit word; a word holds Poisson(n_keys / words) keys.
double bloom_false_positive(uint64_t bits, int64_t n_keys) {
    const double words = (double)(bits / 32), lambda = (double)n_keys / std::max(words, 1.0);
    double fp = 0.0, pmf = std::exp(-lambda);
    const int jmax = (int)(lambda + 12.0 * std::sqrt(lambda + 1.0) + 24.0);
    for (int j = 0; j <= jmax; ++j) {
        const double set = 1.0 - std::pow(31.0 / 32.0, 3.0 * j);
        fp += pmf * set * set * set;
        pmf *= lambda / (double)(j + 1);
    }
    return std::min(1.0, fp);
}

sdb_status check_dim_desc(const sdb_dim_desc* d) {
    if (!d) return fail(SDB_INVALID_ARG, "null dimension descriptor");
    if (d->n_rows < 0) return fail(SDB_INVALID_ARG, "negative n_rows");
    if (d->n_rows > (int64_t)INT32_MAX) return fail(SDB_UNSUPPORTED, "n_rows above 2^31 - 1");
    if (d->n_rows > 0 && !d->key) return fail(SDB_INVALID_ARG, "null key column");
    if (d->n_cols < 0 || d->n_cols > SDB_MAX_DIM_COLS)
        return fail(SDB_UNSUPPORTED, "n_cols %d outside 0..%d", d->n_cols, SDB_MAX_DIM_COLS);
    for (int c = 0; c < d->n_cols; ++c)
        if (d->n_rows > 0 && !d->cols[c]) return fail(SDB_INVALID_ARG, "null dimension column %d", c);
    if (d->n_preds < 0 || d->n_preds > SDB_MAX_DIM_PREDS)
        return fail(SDB_UNSUPPORTED, "n_preds %d outside 0..%d", d->n_preds, SDB_MAX_DIM_PREDS);
    for (int q = 0; q < d->n_preds; ++q) {
        if (d->preds[q].col < 0 || d->preds[q].col >= d->n_cols)
            return fail(SDB_INVALID_ARG, "predicate %d names column %d of %d", q, d->preds[q].col, d->n_cols);
        if (!valid_op(d->preds[q].op)) return fail(SDB_INVALID_ARG, "predicate %d: bad op %d", q, d->preds[q].op);
    }
    if (d->n_payloads < 0 || d->n_payloads > SDB_MAX_PAYLOADS)
        return fail(SDB_UNSUPPORTED, "n_payloads %d outside 0..%d", d->n_payloads, SDB_MAX_PAYLOADS);
    for (int p = 0; p < d->n_payloads; ++p)
        if (d->payload_cols[p] < 0 || d->payload_cols[p] >= d->n_cols)
            return fail(SDB_INVALID_ARG, "payload %d names column %d of %d", p, d->payload_cols[p], d->n_cols);
    if (d->kind < SDB_TABLE_AUTO || d->kind > SDB_TABLE_HASH)
        return fail(SDB_INVALID_ARG, "bad table kind %d", d->kind);
    if (d->dense_budget_bytes < 0 || d->dense_budget_bytes > kMaxDenseBudget)
        return fail(SDB_INVALID_ARG, "dense_budget_bytes %lld outside 0..%lld", (long long)d->dense_budget_bytes,
                    (long long)kMaxDenseBudget);
    if (d->kind != SDB_TABLE_DENSE) {
        const double lf = effective_lf(d);
        if (!(lf > 0.0 && lf <= 0.9)) return fail(SDB_INVALID_ARG, "load factor %g outside (0, 0.9]", lf);
        if (hash_capacity(d->n_rows, lf) > (1ull << 31))
            return fail(SDB_UNSUPPORTED, "hash table above 2^31 slots");
    }
    return SDB_OK;
}

uint64_t required_bytes(const sdb_dim_desc* d) {
    uint64_t table = 0;
    if (d->kind != SDB_TABLE_HASH) {
        table = std::max(table, dense_bytes(dense_slot_limit(d->n_rows), 4));
        if (d->dense_budget_bytes > 0) table = std::max(table, (uint64_t)d->dense_budget_bytes + 512u);
    }
    if (d->kind != SDB_TABLE_DENSE)
        table = std::max(table, align_up(hash_capacity(d->n_rows, effective_lf(d)) * 8, 256) + filter_bytes(d->n_rows));
    return kStatsBytes + table;
}

BuildParams build_params(const sdb_dim_desc* d, DimStats* stats) {
    BuildParams bp;
    std::memset(&bp, 0, sizeof bp);
    bp.key = d->key;
    bp.n = d->n_rows;
    for (int c = 0; c < d->n_cols; ++c) bp.cols[c] = d->cols[c];
    bp.n_preds = d->n_preds;
    for (int q = 0; q < d->n_preds; ++q) {
        bp.pred_col[q] = d->preds[q].col;
        bp.pred[q] = lower_pred(d->preds[q]);
    }
    bp.n_payloads = d->n_payloads;
    for (int p = 0; p < d->n_payloads; ++p) bp.payload_col[p] = d->payload_cols[p];
    bp.stats = stats;
    // partial statistics go to the table region, which the build fills only after
    // they have been combined; one block per 256 * kBuildRows rows, as many as the region holds
    const uint64_t region = required_bytes(d) - kStatsBytes;
    const int64_t by_rows = (d->n_rows + 256 * kBuildRows - 1) / (256 * kBuildRows);
    const int64_t by_room = (int64_t)(region / sizeof(DimStats));
    bp.stats_part = reinterpret_cast<DimStats*>(reinterpret_cast<uint8_t*>(stats) + kStatsBytes);
    bp.stats_blocks = (int32_t)std::max<int64_t>(1, std::min<int64_t>({by_rows, by_room, (int64_t)kStatsMaxBlocks}));
    return bp;
}

// ---- query validation and stages -------------------------------------------

sdb_status check_query(const sdb_query* q) {
    if (!q) return fail(SDB_INVALID_ARG, "null query");
    if (q->n_fact < 0) return fail(SDB_INVALID_ARG, "negative n_fact");
    if (q->n_cols < 1 || q->n_cols > SDB_MAX_FACT_COLS)
        return fail(SDB_UNSUPPORTED, "n_cols %d outside 1..%d", q->n_cols, SDB_MAX_FACT_COLS);
    for (int c = 0; c < q->n_cols; ++c)
        if (q->n_fact > 0 && !q->cols[c]) return fail(SDB_INVALID_ARG, "null fact column %d", c);
    if (q->n_preds < 0 || q->n_preds > SDB_MAX_FACT_PREDS)
        return fail(SDB_UNSUPPORTED, "n_preds %d outside 0..%d", q->n_preds, SDB_MAX_FACT_PREDS);
    for (int i = 0; i < q->n_preds; ++i) {
        if (q->preds[i].col < 0 || q->preds[i].col >= q->n_cols)
            return fail(SDB_INVALID_ARG, "fact predicate %d names column %d of %d", i, q->preds[i].col, q->n_cols);
        if (!valid_op(q->preds[i].op)) return fail(SDB_INVALID_ARG, "fact predicate %d: bad op %d", i, q->preds[i].op);
    }
    if (q->n_joins < 0 || q->n_joins > SDB_MAX_JOINS)
        return fail(SDB_UNSUPPORTED, "n_joins %d outside 0..%d", q->n_joins, SDB_MAX_JOINS);
    for (int j = 0; j < q->n_joins; ++j) {
        const sdb_join& jn = q->joins[j];
        if (jn.fact_key_col < 0 || jn.fact_key_col >= q->n_cols)
            return fail(SDB_INVALID_ARG, "join %d names column %d of %d", j, jn.fact_key_col, q->n_cols);
        if (!jn.dim) return fail(SDB_INVALID_ARG, "join %d has no dimension table", j);
        if (jn.dim->kind != SDB_TABLE_DENSE && jn.dim->kind != SDB_TABLE_HASH)
            return fail(SDB_INVALID_ARG, "join %d: dimension table is not built", j);
        if (!jn.dim->map) return fail(SDB_INVALID_ARG, "join %d: dimension table has no map", j);
        if (jn.dim->kind == SDB_TABLE_DENSE && jn.dim->width != 1 && jn.dim->width != 2 && jn.dim->width != 4)
            return fail(SDB_INVALID_ARG, "join %d: bad dense width %d", j, jn.dim->width);
        if (jn.dim->kind == SDB_TABLE_HASH &&
            (jn.dim->hash_bits < 1 || jn.dim->hash_bits > 31 || jn.dim->n_slots != (1ull << jn.dim->hash_bits)))
            return fail(SDB_INVALID_ARG, "join %d: bad hash table geometry", j);
        const std::string fp = filter_problem(jn.dim);
        if (!fp.empty()) return fail(SDB_INVALID_ARG, "join %d: %s", j, fp.c_str());
    }
    if (q->n_group_keys < 0 || q->n_group_keys > SDB_MAX_GROUP_KEYS)
        return fail(SDB_UNSUPPORTED, "n_group_keys %d outside 0..%d", q->n_group_keys, SDB_MAX_GROUP_KEYS);
    for (int k = 0; k < q->n_group_keys; ++k) {
        const sdb_group_key& g = q->group_keys[k];
        if (g.join < 0 || g.join >= q->n_joins)
            return fail(SDB_INVALID_ARG, "group key %d names join %d of %d", k, g.join, q->n_joins);
        if (g.payload < 0 || g.payload >= q->joins[g.join].dim->n_payloads)
            return fail(SDB_INVALID_ARG, "group key %d names payload %d of %d", k, g.payload,
                        q->joins[g.join].dim->n_payloads);
    }
    if (q->agg.kind < SDB_AGG_COL || q->agg.kind > SDB_AGG_ADD)
        return fail(SDB_INVALID_ARG, "bad aggregate kind %d", q->agg.kind);
    if (q->agg.a < 0 || q->agg.a >= q->n_cols) return fail(SDB_INVALID_ARG, "aggregate operand a = %d", q->agg.a);
    if (q->agg.kind != SDB_AGG_COL && (q->agg.b < 0 || q->agg.b >= q->n_cols))
        return fail(SDB_INVALID_ARG, "aggregate operand b = %d", q->agg.b);
    if (q->force_terminal < SDB_TERMINAL_AUTO || q->force_terminal > SDB_TERMINAL_PART)
        return fail(SDB_INVALID_ARG, "bad force_terminal %d", q->force_terminal);
    if (q->force_ipt != 0 && q->force_ipt != 1 && q->force_ipt != 2 && q->force_ipt != 4)
        return fail(SDB_UNSUPPORTED, "force_ipt %d is not 0, 1, 2 or 4", q->force_ipt);
    if (q->force_vector < -1 || q->force_vector > 1) return fail(SDB_INVALID_ARG, "bad force_vector %d", q->force_vector);
    if (q->grid_blocks < 0) return fail(SDB_INVALID_ARG, "negative grid_blocks");
    if (q->force_lds < -1 || q->force_lds > 3 || q->force_lds == 1)
        return fail(SDB_INVALID_ARG, "force_lds %d is not -1, 0, 2 or 3", q->force_lds);
    if (q->force_block != 0 && q->force_block != 64 && q->force_block != 128 && q->force_block != 256 &&
        q->force_block != kMaxBlock && q->force_block != kBigBlock)
        return fail(SDB_INVALID_ARG, "force_block %d is not 0, 64, 128, 256, %d or %d", q->force_block, kMaxBlock,
                    kBigBlock);
    if (q->force_range < -1 || q->force_range > 1)
        return fail(SDB_INVALID_ARG, "force_range %d is not -1, 0 or 1", q->force_range);
    if (q->force_coarse < -1 || q->force_coarse > SDB_MAX_COARSE_SHIFT)
        return fail(SDB_INVALID_ARG, "force_coarse %d is not in [-1, %d]", q->force_coarse, SDB_MAX_COARSE_SHIFT);
    if (q->force_block == kBigBlock && (q->force_vector == -1 || q->force_ipt == 4 || q->force_eager > 0))
        return fail(SDB_INVALID_ARG, "blocks of %d threads need 4-row items, ipt 1 or 2 and no eager loads", kBigBlock);
    if (q->force_eager < -1 || q->force_eager > kMaxEager)
        return fail(SDB_INVALID_ARG, "force_eager %d is not in -1..%d", q->force_eager, kMaxEager);
    if (q->force_unroll < -1 || q->force_unroll > 0)
        return fail(SDB_INVALID_ARG, "force_unroll %d is not -1 or 0", q->force_unroll);
    if (q->force_window < -1 || q->force_window > (1 << 24))
        return fail(SDB_INVALID_ARG, "force_window %d is not in -1..2^24", q->force_window);
    if (q->force_segments < -1 || q->force_segments > 1)
        return fail(SDB_INVALID_ARG, "force_segments %d is not -1, 0 or 1", q->force_segments);
    if (q->force_prefilter < -1 || q->force_prefilter > 1)
        return fail(SDB_INVALID_ARG, "force_prefilter %d is not -1, 0 or 1", q->force_prefilter);
    return SDB_OK;
}

// Whether the plan may run the fused kernel's instance with the stage loop
// written out kUnrollStages times. The instance exists for 4-row items, two
// items per lane, blocks of kMaxBlock or kBigBlock and no eager loads. Unrolled, each
// stage's parameters stay in scalar registers across tiles instead of being
// reloaded and dispatched per stage and tile; measured on MI355X this helps
// plans whose lookups are in LDS or one device map (c3 2.49 -> 2.40 ms, c2
// 0.173 -> 0.157 ms) but not a hash probe (c5 3% slower; c4, with one item
// per lane, 40%), so hash probes keep the loop.
bool unroll_allowed(const sdb_query* q, const sdb_plan* plan) {
    if (!plan->vector || plan->ipt != 2 || plan->eager != 0 || (plan->block != kMaxBlock && plan->block != kBigBlock))
        return false;
    if (plan->n_stages > kUnrollStages || plan->slice_bits != 0) return false;
    for (int s = 0; s < plan->n_stages; ++s)
        if (plan->stage_kind[s] == 1 && !plan->stage_range[s] &&
            q->joins[plan->stage_index[s]].dim->kind != SDB_TABLE_DENSE)
            return false;
    return true;
}

// Group radices and strides: key k's code ranges over its payload radix;
// the last key varies fastest.
sdb_status group_layout(const sdb_query* q, sdb_plan* plan) {
    plan->n_group_keys = q->n_group_keys;
    uint64_t g = 1;
    for (int k = q->n_group_keys - 1; k >= 0; --k) {
        const sdb_dim* d = q->joins[q->group_keys[k].join].dim;
        const int p = q->group_keys[k].payload;
        plan->key_min[k] = d->payload_min[p];
        plan->radix[k] = d->payload_radix[p];
        plan->stride[k] = g;
        if (d->payload_radix[p] == 0) return fail(SDB_INVALID_ARG, "group key %d has radix 0", k);
        g *= d->payload_radix[p];
        if (g > (uint64_t)INT32_MAX)
            return fail(SDB_CAPACITY, "group domain exceeds 2^31 - 1 (key %d)", k);
    }
    plan->n_groups = g;
    return SDB_OK;
}

// The stage of a fact predicate or join probe in FusedParams form, with the
// A probe that feeds no group key and whose dimension's passing keys are
// exactly one contiguous range passes a fact row iff the row's key lies in
// that range: the build rejects duplicate keys, so n_pass distinct keys in
// [pass_key_min, pass_key_max] fill it when the range holds n_pass values.
bool range_eligible(const sdb_query* q, int join) {
    for (int k = 0; k < q->n_group_keys; ++k)
        if (q->group_keys[k].join == join) return false;
    const sdb_dim* d = q->joins[join].dim;
    if (d->n_pass == 0) return true;
    if (d->pass_key_max < d->pass_key_min) return false;
    return (int64_t)d->pass_key_max - (int64_t)d->pass_key_min + 1 == d->n_pass;
}

// The probe of join `join` as a predicate on its fact key column.
StageDev range_stage(const sdb_query* q, int join) {
    const sdb_dim* d = q->joins[join].dim;
    StageDev S;
    std::memset(&S, 0, sizeof S);
    S.defer = -1;
    S.kind = ST_PRED;
    S.op = OP_PRED;
    S.col = q->joins[join].fact_key_col;
    sdb_pred pr;
    std::memset(&pr, 0, sizeof pr);
    pr.op = SDB_OP_BETWEEN;
    pr.lo = d->n_pass > 0 ? d->pass_key_min : 1;   // no passing key: an empty range
    pr.hi = d->n_pass > 0 ? d->pass_key_max : 0;
    S.test = lower_pred(pr);
    return S;
}

// LDS placement and deferred-gather slot the plan chose for position `pos`
// (pos < 0: no placement, used by the sampling kernel).
StageDev make_stage(const sdb_query* q, const sdb_plan* plan, int kind, int index, int pos) {
    StageDev S;
    std::memset(&S, 0, sizeof S);
    S.defer = -1;
    if (kind == 0) {
        S.kind = ST_PRED;
        S.op = OP_PRED;
        S.col = q->preds[index].col;
        S.test = lower_pred(q->preds[index]);
        return S;
    }
    const sdb_join& jn = q->joins[index];
    const sdb_dim* d = jn.dim;
    S.col = jn.fact_key_col;
    S.map = d->map;
    S.bits = d->bits;
    S.sentinel = d->sentinel;
    if (d->kind == SDB_TABLE_DENSE) {
        S.kind = ST_DENSE;
        S.width = d->width;
        S.kmin = d->key_min;
        S.nslots = (uint32_t)d->n_slots;
    } else {
        S.kind = ST_HASH;
        S.width = 8;
        S.nslots = (uint32_t)d->n_slots;
        S.hmask = (uint32_t)(d->n_slots - 1);
        S.hshift = 32 - d->hash_bits;
    }
    S.n_gk = 0;
    if (plan) {
        for (int k = 0; k < q->n_group_keys; ++k) {
            if (q->group_keys[k].join != index) continue;
            const int p = q->group_keys[k].payload;
            const int n = S.n_gk++;
            S.gk_div[n] = (uint32_t)d->payload_div[p];
            // modulo is only needed when higher payloads share the code
            const bool top = (p == 0);
            S.gk_radix[n] = top ? 0u : d->payload_radix[p];
            S.gk_stride[n] = (uint32_t)plan->stride[k];
        }
        if (pos >= 0) {
            S.lds_mode = plan->stage_lds[pos];
            S.defer = plan->stage_defer[pos];
            S.coarse_shift = plan->stage_coarse[pos];
            if (S.lds_mode == LDS_WINDOW) {
                S.win_lo = (uint32_t)plan->stage_window_lo[pos];
                S.win_slots = (uint32_t)plan->stage_window_slots[pos];
                S.bits = static_cast<const uint32_t*>(d->bits) + S.win_lo / 32u;   // the staged words
            }
        }
    }
    S.gk_mode = S.n_gk == 0 ? GK_NONE
              : (S.n_gk == 1 && S.gk_div[0] == 1u && S.gk_radix[0] == 0u ? GK_ONE : GK_GENERAL);
    const int wsel = S.width == 1 ? 0 : (S.width == 2 ? 1 : 2);
    if (S.kind == ST_HASH) S.op = OP_HASH;
    else if (S.nslots == 0) S.op = OP_NEVER;
    else if (S.lds_mode == LDS_BITS) S.op = OP_LDS_BITS;
    else if (S.lds_mode == LDS_RANK) S.op = OP_LDS_RANK1 + wsel;
    else if (S.lds_mode == LDS_COARSE) S.op = OP_COARSE1 + wsel;
    else if (S.lds_mode == LDS_WINDOW) S.op = OP_WINDOW1 + wsel;
    else if (S.lds_mode == LDS_MAP) S.op = OP_LDS_MAP1 + wsel;
    else S.op = OP_MAP1 + wsel;
    return S;
}

uint64_t stage_table_bytes(const sdb_query* q, int kind, int index) {
    if (kind == 0) return 0;
    const sdb_dim* d = q->joins[index].dim;
    return d->n_slots * (uint64_t)d->width;
}

// Bytes a dense table occupies in LDS as its whole map or as its pass bitmap.
uint64_t lds_map_bytes(const sdb_dim* d) { return align_up(d->n_slots * (uint64_t)d->width, 16); }
uint64_t lds_bits_bytes(const sdb_dim* d) { return align_up((d->n_slots + 31) / 32 * 4, 16); }
// Rank tables of LDS_RANK behind the bitmap: one uint32 count per 64 slots,
// then the passing slots' codes (at least 16 bytes each part).
uint64_t lds_rank_bytes(const sdb_dim* d) { return std::max<uint64_t>(16, align_up((d->n_slots + 63) / 64 * 4, 16)); }
uint64_t lds_codes_bytes(const sdb_dim* d) {
    return std::max<uint64_t>(16, align_up((uint64_t)d->n_pass * (uint64_t)d->width, 16));
}
bool rank_fits(const sdb_dim* d) {
    return d->kind == SDB_TABLE_DENSE && d->bits && d->n_slots > 0 && (d->n_slots + 63) / 64 <= kRankGroups &&
           lds_bits_bytes(d) + lds_rank_bytes(d) + lds_codes_bytes(d) <= kLdsRankBudget;
}
// Coarse pass bitmap of LDS_COARSE: one bit per 2^shift slots, whole 16-byte groups.
uint64_t coarse_bits_bytes(const sdb_dim* d, int shift) {
    const uint64_t bits = (d->n_slots + (1ull << shift) - 1) >> shift;
    return std::max<uint64_t>(16, align_up((bits + 31) / 32 * 4, 16));
}
bool coarse_fits_table(const sdb_dim* d) { return d->kind == SDB_TABLE_DENSE && d->bits && d->n_slots > 0; }
// A stage's part of the run scratch (rank tables, coarse bitmaps): 256-byte aligned.
uint64_t scratch_part(uint64_t bytes) { return align_up(bytes, 256); }

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// Per-row cost of a stage's lookup relative to streaming one int32 column
// (measured on MI355X: a device-memory gather costs about 3 column streams
// when the table stays in L2, about 6 when it is several MB, and a probe into
// a table larger than the MALL is latency bound).
double probe_cost(const sdb_query* q, int kind, int index, int lds_mode) {
    if (kind == 0) return 0.05;
    if (lds_mode != LDS_GLOBAL) return 0.3;
    const sdb_dim* d = q->joins[index].dim;
    const uint64_t bytes = d->n_slots * (uint64_t)d->width;
    if (d->kind == SDB_TABLE_HASH) return bytes > (64ull << 20) ? 60.0 : 10.0;
    return bytes > (2ull << 20) ? 6.0 : 3.0;
}

double stage_cost(const sdb_query* q, const sdb_plan* plan, int s) {
    if (plan->stage_range[s]) return probe_cost(q, 0, 0, LDS_GLOBAL);   // a predicate
    return probe_cost(q, plan->stage_kind[s], plan->stage_index[s], plan->stage_lds[s]);
}

// Fraction of 128-byte lines (32 int32 rows) holding at least one live row.
double line_fraction(double f) { return 1.0 - std::pow(1.0 - std::min(std::max(f, 0.0), 1.0), 32.0); }

// What the planner's sampling kernel measured: for every subset m of the
// stages (bit i = the stage at query position i), the fraction of sampled
// rows that pass every stage in m, and each dense stage's key histogram.
struct Sample {
    bool have = false;
    int n = 0;
    double rows = 0.0;
    std::vector<double> joint;      // 2^n entries
    std::vector<uint32_t> keys;     // kMaxStages x kKeyBuckets
    double frac(uint32_t m) const { return rows > 0.0 ? joint[m] / rows : 0.0; }
};

// Joint pass counts from the pass-pattern histogram: the rows passing every
// stage in m are those whose pattern contains m (a sum over supersets).
void joint_from_patterns(const uint32_t* hist, int n, double rows, Sample* smp) {
    smp->have = true;
    smp->n = n;
    smp->rows = rows;
    smp->joint.assign((size_t)1 << n, 0.0);
    for (size_t m = 0; m < smp->joint.size(); ++m) smp->joint[m] = (double)hist[m];
    for (int b = 0; b < n; ++b)
        for (size_t m = 0; m < smp->joint.size(); ++m)
            if (!(m & ((size_t)1 << b))) smp->joint[m] += smp->joint[m | ((size_t)1 << b)];
}

// Fraction of rows that pass the stages at positions order[0 .. k-1]: measured
// jointly when there is a sample, else the product of the per-stage estimates.
struct Reach {
    const sdb_plan* plan;
    const Sample* smp;
    const int* bit;     // query position of the stage at each plan position
    double of(const int* order, int k) const {
        if (smp && smp->have) {
            uint32_t m = 0;
            for (int i = 0; i < k; ++i) m |= 1u << bit[order[i]];
            return smp->frac(m);
        }
        double f = 1.0;
        for (int i = 0; i < k; ++i) f *= plan->stage_pass[order[i]];
        return f;
    }
};

// Modeled cost of running the stages in `order`: column streaming at line
// granularity plus lookups for the rows that reach each stage, then the
// aggregate columns and deferred gathers for the survivors.
double order_cost(const sdb_query* q, const sdb_plan* plan, const int* order, int n, const Reach& reach) {
    double cost = 0.0;
    for (int i = 0; i < n; ++i) {
        const double f = reach.of(order, i);
        cost += line_fraction(f) + f * stage_cost(q, plan, order[i]);
    }
    const double f = reach.of(order, n);
    const int agg_cols = q->agg.kind == SDB_AGG_COL ? 1 : 2;
    cost += agg_cols * line_fraction(f);
    for (int s = 0; s < n; ++s)
        if (plan->stage_lds[s] == LDS_BITS && plan->stage_kind[s] == 1) {
            const sdb_dim* d = q->joins[plan->stage_index[s]].dim;
            bool gathers = false;
            for (int k = 0; k < q->n_group_keys; ++k) gathers |= q->group_keys[k].join == plan->stage_index[s];
            if (gathers) cost += f * (d->n_slots * (uint64_t)d->width > (2ull << 20) ? 6.0 : 3.0);
        }
    return cost;
}

// Cheapest order under order_cost: exhaustive up to 7 stages, else greedy:
// next the stage with the best (1 - conditional pass) / cost among those
// left, given the stages already chosen. Permutes the plan's stage arrays
// and `bit` alike, and leaves in stage_pass each stage's pass fraction given
// the stages before it (measured jointly when there is a sample).
void choose_order(const sdb_query* q, sdb_plan* plan, int* bit, const Sample* smp) {
    const int n = plan->n_stages;
    const Reach reach{plan, smp, bit};
    std::vector<int> order(n), best;
    for (int i = 0; i < n; ++i) order[i] = i;
    double best_cost = 0.0;
    if (n <= 7) {
        best_cost = order_cost(q, plan, order.data(), n, reach);
        best = order;
        while (std::next_permutation(order.begin(), order.end())) {
            const double c = order_cost(q, plan, order.data(), n, reach);
            if (c < best_cost - 1e-12) {
                best_cost = c;
                best = order;
            }
        }
    } else {
        std::vector<bool> used(n, false);
        for (int i = 0; i < n; ++i) {
            const double before = reach.of(best.data(), i);
            int pick = -1;
            double pick_rank = -1.0;
            for (int s = 0; s < n; ++s) {
                if (used[s]) continue;
                best.push_back(s);
                const double after = reach.of(best.data(), i + 1);
                best.pop_back();
                const double pass = before > 0.0 ? after / before : plan->stage_pass[s];
                const double rank = (1.0 - pass) / (1.0 + stage_cost(q, plan, s));
                if (rank > pick_rank + 1e-12) {
                    pick_rank = rank;
                    pick = s;
                }
            }
            used[pick] = true;
            best.push_back(pick);
        }
        best_cost = order_cost(q, plan, best.data(), n, reach);
    }
    const sdb_plan tmp = *plan;
    int tmp_bit[SDB_MAX_STAGES];
    for (int i = 0; i < n; ++i) tmp_bit[i] = bit[i];
    std::vector<double> cond(n);
    for (int i = 0; i < n; ++i) {
        const double before = reach.of(best.data(), i), after = reach.of(best.data(), i + 1);
        cond[i] = before > 0.0 ? after / before : tmp.stage_pass[best[i]];
    }
    for (int i = 0; i < n; ++i) {
        plan->stage_kind[i] = tmp.stage_kind[best[i]];
        plan->stage_index[i] = tmp.stage_index[best[i]];
        plan->stage_pass[i] = smp && smp->have ? cond[i] : tmp.stage_pass[best[i]];
        plan->stage_pass_alone[i] = tmp.stage_pass_alone[best[i]];
        plan->stage_lds[i] = tmp.stage_lds[best[i]];
        plan->stage_range[i] = tmp.stage_range[best[i]];
        bit[i] = tmp_bit[best[i]];
    }
    plan->est_cost = best_cost;
}

// Mid-scan reordering: each run of sampled rows (range) gets the order with
// the least modelled cost on its own pass patterns; neighbouring ranges with
// equal orders merge into one segment. Kept when the modelled cost over all
// ranges drops by at least kSegmentMinGain against the table's single order
// (any drop when forced), on tables of at least kSegmentMinRows rows, in at
// most SDB_MAX_SEGMENTS segments. Segment starts are the first sampled row of
// each range, rounded down to a multiple of kSegmentAlign rows.
constexpr double kSegmentMinGain = 0.03;
constexpr int64_t kSegmentMinRows = 1ll << 24;
constexpr int64_t kSegmentAlign = 4096;

void choose_segments(const sdb_query* q, sdb_plan* plan, const int* bit, const std::vector<Sample>& ranges,
                     int64_t step, int64_t n_sample, std::vector<double>* seg_survivors) {
    const int n = plan->n_stages, R = (int)ranges.size();
    if (n > 7 || R < 2) return;
    std::vector<std::vector<int>> best(R);
    double base = 0.0, tuned = 0.0;
    std::vector<int> ident(n);
    for (int i = 0; i < n; ++i) ident[i] = i;
    for (int r = 0; r < R; ++r) {
        const Reach reach{plan, &ranges[r], bit};
        std::vector<int> order = ident;
        const double c0 = order_cost(q, plan, order.data(), n, reach);
        double bc = c0;
        best[r] = order;
        while (std::next_permutation(order.begin(), order.end())) {
            const double c = order_cost(q, plan, order.data(), n, reach);
            if (c < bc - 1e-12) {
                bc = c;
                best[r] = order;
            }
        }
        base += c0;
        tuned += bc;
    }
    // merge neighbours with equal orders
    std::vector<int> first;   // first range of each segment
    for (int r = 0; r < R; ++r)
        if (r == 0 || best[r] != best[r - 1]) first.push_back(r);
    const int segs = (int)first.size();
    const bool forced = q->force_segments == 1;
    if (segs < 2 || segs > SDB_MAX_SEGMENTS) return;
    if (!forced && (q->n_fact < kSegmentMinRows || base <= 0.0 || (base - tuned) / base < kSegmentMinGain)) return;
    int64_t start[SDB_MAX_SEGMENTS + 1];
    for (int g = 0; g < segs; ++g) {
        const int64_t k = ((int64_t)first[g] * n_sample + R - 1) / R;   // first sampled row of the range
        start[g] = g == 0 ? 0 : std::min<int64_t>(k * step, q->n_fact) / kSegmentAlign * kSegmentAlign;
    }
    start[segs] = q->n_fact;
    for (int g = 1; g <= segs; ++g)
        if (start[g] <= start[g - 1]) return;   // a range too short for its own segment
    plan->n_segments = segs;
    for (int g = 0; g < segs; ++g)
        for (int i = 0; i < n; ++i) plan->segment_order[g][i] = best[first[g]][i];
    for (int g = 0; g <= segs; ++g) plan->segment_start[g] = start[g];
    // survivors per segment: each range's sampled fraction passing every stage
    const uint32_t all = (uint32_t)((1ull << n) - 1);
    seg_survivors->assign(segs, 0.0);
    for (int r = 0, g = 0; r < R; ++r) {
        if (g + 1 < segs && r >= first[g + 1]) ++g;
        (*seg_survivors)[g] += ranges[r].frac(all) * (double)q->n_fact / R;
    }
}

// LDS placement: dense tables, smallest first, as the whole map when it fits
// the remaining budget, else as the pass bitmap, else left in device memory.
void place_lds(const sdb_query* q, sdb_plan* plan, uint64_t budget) {
    std::vector<int> cand;
    for (int s = 0; s < plan->n_stages; ++s) {
        plan->stage_lds[s] = LDS_GLOBAL;
        if (plan->stage_kind[s] == 1 && !plan->stage_range[s] &&
            q->joins[plan->stage_index[s]].dim->kind == SDB_TABLE_DENSE &&
            q->joins[plan->stage_index[s]].dim->n_slots > 0)
            cand.push_back(s);
    }
    std::stable_sort(cand.begin(), cand.end(), [&](int x, int y) {
        return lds_bits_bytes(q->joins[plan->stage_index[x]].dim) < lds_bits_bytes(q->joins[plan->stage_index[y]].dim);
    });
    uint64_t left = budget;
    for (int s : cand) {
        const sdb_dim* d = q->joins[plan->stage_index[s]].dim;
        if (lds_map_bytes(d) <= left) {
            plan->stage_lds[s] = LDS_MAP;
            left -= lds_map_bytes(d);
        } else if (d->bits && lds_bits_bytes(d) <= left) {
            plan->stage_lds[s] = LDS_BITS;
            left -= lds_bits_bytes(d);
        }
    }
}

// Dynamic LDS layout of the fused kernel: the LDS group table, then each
// staged table at a 16-byte aligned offset. Returns the total bytes.
uint32_t lds_layout(const sdb_query* q, const sdb_plan* plan, FusedParams* p) {
    uint64_t off = 0;
    if (plan->terminal == TERM_LDS) off = plan->n_groups * 16;
    // (room for the most record regions a block may have, whatever part_subs)
    if (plan->terminal == TERM_PART) off = align_up((uint64_t)kPartSubRegions * (1 + (uint64_t)plan->n_parts) * 4, 16);
    if (p) p->term_lds_bytes = (uint32_t)off;
    for (int s = 0; s < plan->n_stages; ++s) {
        if (plan->stage_lds[s] == LDS_GLOBAL) continue;
        const sdb_dim* d = q->joins[plan->stage_index[s]].dim;
        const uint64_t bytes = plan->stage_lds[s] == LDS_MAP      ? lds_map_bytes(d)
                               : plan->stage_lds[s] == LDS_COARSE ? coarse_bits_bytes(d, plan->stage_coarse[s])
                               : plan->stage_lds[s] == LDS_WINDOW ? (uint64_t)plan->stage_window_slots[s] / 8u
                                                                  : lds_bits_bytes(d);
        if (p) {
            p->st[s].lds_off = (uint32_t)off;
            p->st[s].lds_bytes = (uint32_t)bytes;
        }
        off += bytes;
        if (plan->stage_lds[s] == LDS_RANK) {
            if (p) {
                p->st[s].lds_rank_off = (uint32_t)off;
                p->st[s].lds_rank_bytes = (uint32_t)lds_rank_bytes(d);
                p->st[s].lds_codes_off = (uint32_t)(off + lds_rank_bytes(d));
                p->st[s].lds_codes_bytes = (uint32_t)lds_codes_bytes(d);
            }
            off += lds_rank_bytes(d) + lds_codes_bytes(d);
        }
    }
    return (uint32_t)off;
}

int stage_column(const sdb_query* q, const sdb_plan* plan, int s) {
    return plan->stage_kind[s] == 0 ? q->preds[plan->stage_index[s]].col : q->joins[plan->stage_index[s]].fact_key_col;
}

// Distinct fact columns in order of first use (stages in plan order, then the
// aggregate operands), each with the fraction of rows still live there.
int columns_in_use_order(const sdb_query* q, const sdb_plan* plan, int* cols, double* live) {
    int n = 0;
    double f = 1.0;
    auto add = [&](int c) {
        for (int i = 0; i < n; ++i)
            if (cols[i] == c) return;
        cols[n] = c;
        live[n] = f;
        ++n;
    };
    for (int s = 0; s < plan->n_stages; ++s) {
        add(stage_column(q, plan, s));
        f *= plan->stage_pass[s];
    }
    add(q->agg.a);
    if (q->agg.kind != SDB_AGG_COL) add(q->agg.b);
    return n;
}

FusedParams fused_params(const sdb_query* q, const sdb_plan* plan, bool placed) {
    FusedParams p;
    std::memset(&p, 0, sizeof p);
    for (int c = 0; c < q->n_cols; ++c) p.cols[c] = q->cols[c];
    p.n = q->n_fact;
    p.nstages = plan->n_stages;
    p.defer_stage = -1;
    for (int s = 0; s < plan->n_stages; ++s) {
        if (plan->stage_range[s]) {
            p.st[s] = range_stage(q, plan->stage_index[s]);
            continue;
        }
        p.st[s] = make_stage(q, plan, plan->stage_kind[s], plan->stage_index[s], placed ? s : -1);
        if (placed && p.st[s].defer == 0) p.defer_stage = s;
    }
    p.agg_kind = q->agg.kind;
    p.agg_a = q->agg.a;
    p.agg_b = q->agg.kind == SDB_AGG_COL ? q->agg.a : q->agg.b;
    p.n_groups = (uint32_t)plan->n_groups;
    // eager slots: the first plan->eager columns in order of use
    int order_cols[SDB_MAX_FACT_COLS];
    double live[SDB_MAX_FACT_COLS];
    const int n_used = columns_in_use_order(q, plan, order_cols, live);
    p.eg_n = std::max(0, std::min(std::min((int)plan->eager, kMaxEager), n_used));
    for (int k = 0; k < p.eg_n; ++k) p.eg_col[k] = order_cols[k];
    auto slot_of = [&](int col) {
        for (int k = 0; k < p.eg_n; ++k)
            if (p.eg_col[k] == col) return k;
        return -1;
    };
    for (int s = 0; s < plan->n_stages; ++s) p.st[s].eg_slot = slot_of(p.st[s].col);
    p.agg_a_slot = slot_of(p.agg_a);
    p.agg_b_slot = slot_of(p.agg_b);
    if (placed) lds_layout(q, plan, &p);
    return p;
}

// Every column the fused kernel reads: stage columns and aggregate operands.
bool columns_aligned(const sdb_query* q, const sdb_plan* plan) {
    for (int s = 0; s < plan->n_stages; ++s)
        if (!aligned16(q->cols[stage_column(q, plan, s)])) return false;
    if (!aligned16(q->cols[q->agg.a])) return false;
    if (q->agg.kind != SDB_AGG_COL && !aligned16(q->cols[q->agg.b])) return false;
    return true;
}

constexpr int kDefaultIpt = 2;
constexpr bool kAutoEager = false;
// a 128-byte line holds 32 rows: at 2% live rows about half its lines are still read
constexpr double kEagerMinLive = 0.02;
// the partitioned terminal: at least a million survivors, and this many per group
constexpr double kPartMinPerGroup = 16.0;
// ... and about this many record regions per launch (sdb_plan.part_subs),
// for blocks expecting fewer than kPartSplitMaxRecords records
constexpr int64_t kPartRegions = 1024;
constexpr double kPartSplitMaxRecords = 262144.0;

// Partitioned-terminal records carry 64-bit values only when the aggregate
// combines two columns; a single int32 column's values fit 32 bits.
bool records_wide(const sdb_query* q) { return q->agg.kind != SDB_AGG_COL; }

// Run-scratch layout of the partitioned terminal.
struct PartLayout {
    uint64_t region_count, part_count, part_start, chunk_start, part_hist, rec_gid, rec_val, sorted_gid,
        sorted_val, item_sum, item_cnt, total;
};

// Record regions of a partitioned plan: part_subs per block of every launch
// (a segmented plan launches once per segment).
uint64_t part_regions(const sdb_plan* plan) {
    return (uint64_t)plan->grid * (uint64_t)std::max(1, plan->n_segments) * (uint64_t)plan->part_subs;
}

PartLayout part_layout(const sdb_query* q, const sdb_plan* plan) {
    PartLayout L;
    const uint64_t grid = part_regions(plan), P = (uint64_t)plan->n_parts;
    const uint64_t recs = grid * (uint64_t)plan->part_cap;
    const uint64_t vbytes = records_wide(q) ? 8 : 4;
    // aggregation work items: at most one partial chunk per partition plus full chunks
    const uint64_t items = P + recs / (uint64_t)kPartChunk;
    const uint64_t gpp = 1ull << plan->part_shift;
    uint64_t off = 0;
    auto take = [&](uint64_t bytes) {
        const uint64_t at = off;
        off += align_up(bytes, 256);
        return at;
    };
    L.region_count = take(grid * 4);
    L.part_count = take(P * 4);
    L.part_start = take((P + 1) * 4);
    L.chunk_start = take((P + 1) * 4);
    L.part_hist = take(P * grid * 4);
    L.rec_gid = take(recs * 4);
    L.rec_val = take(recs * vbytes);
    L.sorted_gid = take(recs * 4);
    L.sorted_val = take(recs * vbytes);
    L.item_sum = take(items * gpp * 8);
    L.item_cnt = take(items * gpp * 4);
    L.total = off;
    return L;
}

// Sliced hash probe (sdb_plan.slice_bits): chosen for a hash table of at
// least 16 MiB (random probes into it miss L2; measured on MI355X, 8-byte
// probes run at about 54G/s into 32-256 MiB and 215G/s into 0.5-2 MiB) over
// at least 2^24 fact rows. Slices of 2 MiB: more partitions would shorten
// the scatter's runs of stores (measured: its time grows from 2.6 ms at 64
// partitions to 3.8 ms at 512 for 600M rows) for little gain in the probe.
constexpr uint64_t kSliceMinTableBytes = 16ull << 20;
constexpr int64_t kSliceMinRows = 1ll << 24;
constexpr int64_t kSliceMaxRows = 0xFFFFF000ll;   // record positions are 32-bit
constexpr int kSliceLog2Bytes = 21;
// The pre-filter pays when at most this fraction of the rows gets through it.
// Measured on c5 (600M rows, half of them dropped): the filter reads add 2.3
// ms to the count pass, and the dropped rows save 0.9 ms of the scatter pass
// and 3.1 ms of the probe, so a row costs about 0.28 of what a dropped row
// saves.
constexpr double kPrefilterMaxKept = 0.7;

// The join the query allows to run over table slices, or -1: the only join,
// into a hash table, with every other stage a fact predicate, a SUM of one
// column (the partitioned records carry one 32-bit value), and the columns
// the count and scatter passes read 16-byte aligned (128-bit loads).
int slice_join(const sdb_query* q) {
    if (q->n_joins != 1 || q->n_fact > kSliceMaxRows) return -1;
    const sdb_dim* d = q->joins[0].dim;
    if (d->kind != SDB_TABLE_HASH || d->hash_bits < 1) return -1;
    if (!aligned16(q->cols[q->joins[0].fact_key_col]) || !aligned16(q->cols[q->agg.a])) return -1;
    if (q->agg.kind != SDB_AGG_COL && !aligned16(q->cols[q->agg.b])) return -1;
    for (int i = 0; i < q->n_preds; ++i)
        if (!aligned16(q->cols[q->preds[i].col])) return -1;
    return 0;
}

int slice_bits_for(const sdb_dim* d) {
    const int want = d->hash_bits + 3 - kSliceLog2Bytes;
    return std::max(1, std::min(want, std::min((int)d->hash_bits, SDB_MAX_SLICE_BITS)));
}

// Run-scratch layout of the sliced probe's partition passes.
struct SliceLayout {
    uint64_t hist, part_count, part_start, chunk_start, out_key, out_val, out_val2, keep, tile_base, tile_map, total;
    int64_t tile_rows, n_vtiles;
};

// Rows per tile of the fused launch over the partitioned rows, and the length
// of its tile map: 8 slots per tile, enough for any split of the tiles among
// the XCDs.
int64_t slice_tile_rows(const sdb_plan* plan) {
    return (int64_t)plan->block * plan->ipt * (plan->vector ? 4 : 1);
}

SliceLayout slice_layout(const sdb_query* q, const sdb_plan* plan) {
    SliceLayout L;
    std::memset(&L, 0, sizeof L);
    if (plan->slice_bits <= 0) return L;
    const uint64_t P = 1ull << plan->slice_bits, grid = (uint64_t)plan->slice_grid;
    const uint64_t n = (uint64_t)std::max<int64_t>(q->n_fact, 1);
    uint64_t off = 0;
    auto take = [&](uint64_t bytes) {
        const uint64_t at = off;
        off += align_up(bytes, 256);
        return at;
    };
    L.hist = take(P * grid * 4);
    L.part_count = take(P * 4);
    L.part_start = take((P + 1) * 4);
    L.chunk_start = take((P + 1) * 4);
    L.out_key = take(n * 4);
    L.out_val = take(n * 4);
    L.out_val2 = q->agg.kind != SDB_AGG_COL ? take(n * 4) : 0;
    L.keep = plan->slice_prefilter ? take((n + 3) / 4) : 0;
    L.tile_rows = std::max<int64_t>(1, slice_tile_rows(plan));
    L.n_vtiles = 8 * ((int64_t)((n + (uint64_t)L.tile_rows - 1) / (uint64_t)L.tile_rows) + 1);
    L.tile_base = take(P * 4);
    L.tile_map = take((uint64_t)L.n_vtiles * 4);
    L.total = off;
    return L;
}

// Run scratch of the LDS_RANK stages' tables and the LDS_COARSE stages'
// coarse bitmaps, in stage order; the terminal's scratch follows it.
uint64_t stage_scratch_bytes(const sdb_query* q, const sdb_plan* plan) {
    uint64_t b = 0;
    for (int s = 0; s < plan->n_stages; ++s) {
        const sdb_dim* d = plan->stage_kind[s] == 1 ? q->joins[plan->stage_index[s]].dim : nullptr;
        if (plan->stage_lds[s] == LDS_RANK)
            b += scratch_part(lds_rank_bytes(d)) + scratch_part(lds_codes_bytes(d));
        else if (plan->stage_lds[s] == LDS_COARSE)
            b += scratch_part(coarse_bits_bytes(d, plan->stage_coarse[s]));
    }
    return b;
}

// Dynamic LDS of a fused-kernel launch: the plan's layout, then (partitioned
// terminal) one record ring per wave.
uint32_t ring_lds_bytes(const sdb_query* q, const sdb_plan* plan) {
    if (plan->terminal != TERM_PART) return 0u;
    return (uint32_t)(plan->block / 64) * kRingEntries * (records_wide(q) ? 12u : 8u);
}

uint32_t launch_lds_bytes(const sdb_query* q, const sdb_plan* plan) {
    return (uint32_t)plan->lds_bytes + ring_lds_bytes(q, plan);
}

// LDS a block may use so that the blocks the grid counts on all fit (see choose_grid).
constexpr uint32_t kLdsUsable = 152u * 1024u;

sdb_status choose_grid(const sdb_query* q, const sdb_plan* plan, int* grid_out) {
    const int64_t rows_per_item = plan->vector ? 4 : 1;
    const int64_t n_items = q->n_fact / rows_per_item;
    const int64_t tile = (int64_t)plan->block * plan->ipt;
    int64_t tiles = (n_items + tile - 1) / tile;
    if (tiles < 1) tiles = 1;
    if (q->grid_blocks > 0) {
        *grid_out = (int)std::min<int64_t>(q->grid_blocks, INT32_MAX);
        return SDB_OK;
    }
    DeviceInfo di;
    sdb_status st = device_info(&di);
    if (st != SDB_OK) return st;
    int per_cu = fused_blocks_per_cu(plan->vector, plan->ipt, plan->terminal, plan->eager, plan->block, plan->unroll,
                                     (size_t)launch_lds_bytes(q, plan));
    if (per_cu <= 0) return fail(SDB_HIP_ERROR, "occupancy query failed for the fused kernel");
    // The occupancy query counts LDS as if all 160 KB were available in fine
    // granules; measured on MI355X, five blocks of 32,048 bytes do not run
    // together (a grid of five blocks per CU then runs a fifth of its blocks
    // late) while five of 27,568 do. Count LDS in 2 KB granules out of 152 KB.
    const uint32_t lds = launch_lds_bytes(q, plan);
    if (lds > 0) {
        const uint32_t granule = 2048, usable = kLdsUsable;
        const int by_lds = (int)(usable / (uint32_t)align_up(lds, granule));
        per_cu = std::max(1, std::min(per_cu, by_lds));
    }
    const int64_t full = (int64_t)di.cus * per_cu;
    *grid_out = (int)std::min<int64_t>(tiles, full);
    return SDB_OK;
}

// Checks shared by both run entry points: the query, the plan's stage list
// and deferred gathers, the group layout and the output capacity.
// LDS windows are a forced placement only: measured on MI355X they do not
// pay. On c3 a window over 29% of the customer keys spares 28M of the fused
// kernel's 211M L2 requests but leaves the kernel within 1% (2.219 against
// 2.229 ms) and the run and step slower; on c4 a window over 96% of the Zipf
// part keys, sized to keep 32 waves per CU, spares 30M of 90M requests and
// runs 5% slower (1.720 against 1.640 ms): c4 is bound by each wave's chain of
// dependent loads, not by the number of requests. The automatic rule below
// (a window that spares the gathers of at least 2% of all fact rows, on at
// least 2^24 rows) is kept for hardware where that trade differs.
constexpr bool kWindowAuto = false;
constexpr double kWindowMinGain = 0.02;
constexpr int64_t kWindowMinRows = 1ll << 24;

// Sampled fraction of a dense stage's fact keys inside slots [lo, lo + len):
// whole buckets count fully, a partly covered bucket by its covered share.
double window_cover(const uint32_t* hist, uint64_t nslots, uint64_t lo, uint64_t len) {
    double in = 0.0, all = 0.0;
    for (int b = 0; b < kKeyBuckets; ++b) {
        const uint64_t b0 = (uint64_t)b * nslots / kKeyBuckets, b1 = (uint64_t)(b + 1) * nslots / kKeyBuckets;
        all += hist[b];
        if (b1 <= b0) continue;
        const uint64_t o0 = std::max(b0, lo), o1 = std::min(b1, lo + len);
        if (o1 > o0) in += hist[b] * (double)(o1 - o0) / (double)(b1 - b0);
    }
    return all > 0.0 ? in / all : 0.0;
}

// LDS window (SDB_LDS_WINDOW) for the dense device-memory stage whose rows it
// serves most: window length from the LDS a block can take without lowering
// the blocks per CU its registers allow (measured on c4: a window that halves
// the waves per CU makes the kernel 60% slower although it spares 96% of the
// part-map gathers), start where the sampled keys are densest. Returns the
// stage or -1.
int place_window(const sdb_query* q, sdb_plan* plan, const Sample& smp, const int* bit, int64_t n_fact) {
    if (q->force_window == -1 || q->force_lds == -1) return -1;
    // (not forced and not placed automatically: skip the search, about 50 us
    // of host time per plan on c3, on the path from one fused kernel to the next)
    if (q->force_window == 0 && !kWindowAuto) return -1;
    const Reach reach{plan, &smp, bit};
    int order[SDB_MAX_STAGES];
    for (int i = 0; i < plan->n_stages; ++i) order[i] = i;
    const uint64_t used = lds_layout(q, plan, nullptr) + ring_lds_bytes(q, plan);
    int per_cu = fused_blocks_per_cu(plan->vector, plan->ipt, plan->terminal, plan->eager, plan->block,
                                     unroll_allowed(q, plan) && q->force_unroll != -1 ? 1 : 0, (size_t)used);
    if (per_cu < 1) per_cu = 1;
    const uint64_t per_block = (uint64_t)kLdsUsable / (uint64_t)per_cu / 2048u * 2048u;
    if (used + 2048u >= per_block) return -1;
    const uint64_t lds_left = per_block - used - 2048u;   // a granule of slack
    int best = -1;
    double best_gain = 0.0, best_cover = 0.0;
    uint64_t best_lo = 0, best_len = 0;
    for (int s = 0; s < plan->n_stages; ++s) {
        if (plan->stage_kind[s] != 1 || plan->stage_lds[s] != LDS_GLOBAL || plan->stage_range[s]) continue;
        const sdb_dim* d = q->joins[plan->stage_index[s]].dim;
        if (d->kind != SDB_TABLE_DENSE || !d->bits || d->n_slots == 0 || d->n_slots > 0xFFFFFFFFull) continue;
        const uint64_t padded = align_up(d->n_slots, 128);
        uint64_t len = std::min<uint64_t>(padded, lds_left * 8u / 128u * 128u);
        if (q->force_window >= 2) len = std::min<uint64_t>(len, 128ull * (uint64_t)q->force_window);
        if (len < 128) continue;
        uint64_t lo = 0;
        double cover = (double)std::min<uint64_t>(len, d->n_slots) / (double)d->n_slots;
        if (smp.have) {
            const uint32_t* hist = &smp.keys[(size_t)bit[s] * kKeyBuckets];
            cover = -1.0;
            for (int b = 0; b <= kKeyBuckets; ++b) {
                // windows starting at a bucket edge, and the one ending at the last slot
                uint64_t cand = b < kKeyBuckets ? (uint64_t)b * d->n_slots / kKeyBuckets / 128 * 128
                                                : padded - len;
                cand = std::min(cand, padded - len);
                const double c = window_cover(hist, d->n_slots, cand, len);
                if (c > cover + 1e-12) {
                    cover = c;
                    lo = cand;
                }
            }
        }
        const double gain = reach.of(order, s) * cover;   // rows whose gather the window saves
        if (gain > best_gain) {
            best_gain = gain;
            best = s;
            best_cover = cover;
            best_lo = lo;
            best_len = len;
        }
    }
    if (best < 0) return -1;
    if (q->force_window == 0 && (!kWindowAuto || best_gain < kWindowMinGain || n_fact < kWindowMinRows)) return -1;
    plan->stage_lds[best] = LDS_WINDOW;
    plan->stage_window_lo[best] = (int32_t)best_lo;
    plan->stage_window_slots[best] = (int32_t)best_len;
    plan->stage_window_cover[best] = best_cover;
    return best;
}

sdb_status check_run(const sdb_query* q, const sdb_plan* plan, int64_t* sums, int64_t* counts,
                     int64_t n_groups_capacity) {
    sdb_status st = check_query(q);
    if (st != SDB_OK) return st;
    if (!plan) return fail(SDB_INVALID_ARG, "null plan");
    if (!sums || !counts) return fail(SDB_INVALID_ARG, "null output");
    if (plan->n_stages != q->n_preds + q->n_joins) return fail(SDB_INVALID_ARG, "plan does not match the query");
    int n_defer = 0;
    {
        bool seen[SDB_MAX_STAGES] = {false};
        for (int s = 0; s < plan->n_stages; ++s) {
            const int k = plan->stage_kind[s], i = plan->stage_index[s];
            if ((k != 0 && k != 1) || i < 0 || (k == 0 && i >= q->n_preds) || (k == 1 && i >= q->n_joins))
                return fail(SDB_INVALID_ARG, "plan stage %d is invalid", s);
            const int slot = k == 0 ? i : q->n_preds + i;
            if (seen[slot]) return fail(SDB_INVALID_ARG, "plan stage %d repeats a stage", s);
            seen[slot] = true;
            const int lm = plan->stage_lds[s];
            if (lm != LDS_GLOBAL) {
                if (k != 1 || q->joins[i].dim->kind != SDB_TABLE_DENSE)
                    return fail(SDB_INVALID_ARG, "plan stage %d: LDS placement needs a dense table", s);
                if (lm != LDS_MAP && lm != LDS_BITS && lm != LDS_RANK && lm != LDS_COARSE && lm != LDS_WINDOW)
                    return fail(SDB_INVALID_ARG, "plan stage %d: bad LDS mode", s);
                if ((lm == LDS_BITS || lm == LDS_RANK || lm == LDS_COARSE || lm == LDS_WINDOW) &&
                    !q->joins[i].dim->bits)
                    return fail(SDB_INVALID_ARG, "plan stage %d: table has no bitmap", s);
                if (lm == LDS_RANK && !rank_fits(q->joins[i].dim))
                    return fail(SDB_INVALID_ARG, "plan stage %d: rank tables do not fit LDS", s);
            }
            if (plan->stage_defer[s] != -1) {
                if (plan->stage_defer[s] != 0 || lm != LDS_BITS)
                    return fail(SDB_INVALID_ARG, "plan stage %d: bad deferred gather", s);
                ++n_defer;
            }
            if (lm == LDS_WINDOW) {
                const uint64_t lo = (uint64_t)(uint32_t)plan->stage_window_lo[s];
                const uint64_t len = (uint64_t)(uint32_t)plan->stage_window_slots[s];
                const uint64_t padded = align_up(q->joins[i].dim->n_slots, 128);
                if (plan->stage_window_lo[s] < 0 || plan->stage_window_slots[s] <= 0 || lo % 128 || len % 128 ||
                    lo + len > padded)
                    return fail(SDB_INVALID_ARG, "plan stage %d: window of %lld slots at %lld outside the table's "
                                "%llu slots (or not whole 128-slot groups)", s,
                                (long long)plan->stage_window_slots[s], (long long)plan->stage_window_lo[s],
                                (unsigned long long)q->joins[i].dim->n_slots);
            } else if (plan->stage_window_lo[s] != 0 || plan->stage_window_slots[s] != 0) {
                return fail(SDB_INVALID_ARG, "plan stage %d: window fields without a window", s);
            }
            if (plan->stage_range[s] != 0) {
                if (plan->stage_range[s] != 1 || k != 1 || lm != LDS_GLOBAL || plan->stage_defer[s] != -1 ||
                    !range_eligible(q, i))
                    return fail(SDB_INVALID_ARG, "plan stage %d: the probe is not a key range", s);
            }
            if ((lm == LDS_COARSE) != (plan->stage_coarse[s] != 0))
                return fail(SDB_INVALID_ARG, "plan stage %d: coarse shift without the coarse placement", s);
            if (lm == LDS_COARSE && (plan->stage_coarse[s] < 1 || plan->stage_coarse[s] > SDB_MAX_COARSE_SHIFT ||
                                     plan->stage_defer[s] != -1 || plan->stage_range[s] != 0))
                return fail(SDB_INVALID_ARG, "plan stage %d: bad coarse placement", s);
        }
    }
    if (n_defer > 1) return fail(SDB_INVALID_ARG, "plan defers more than one gather");
    sdb_plan layout;
    std::memset(&layout, 0, sizeof layout);
    st = group_layout(q, &layout);
    if (st != SDB_OK) return st;
    if (layout.n_groups != plan->n_groups) return fail(SDB_INVALID_ARG, "plan group count does not match the query");
    for (int k = 0; k < q->n_group_keys; ++k)
        if (layout.stride[k] != plan->stride[k] || layout.radix[k] != plan->radix[k])
            return fail(SDB_INVALID_ARG, "plan group layout does not match the query");
    if (n_groups_capacity < 0 || (uint64_t)n_groups_capacity < plan->n_groups)
        return fail(SDB_CAPACITY, "output holds %lld groups, plan needs %llu", (long long)n_groups_capacity,
                    (unsigned long long)plan->n_groups);
    return SDB_OK;
}

}  // namespace

// ============================================================================
// C ABI
// ============================================================================

extern "C" {

SDB_API const char* sdb_last_error(void) { return g_error.c_str(); }

SDB_API const char* sdb_status_string(int32_t s) {
    switch (s) {
        case SDB_OK: return "SDB_OK";
        case SDB_INVALID_ARG: return "SDB_INVALID_ARG";
        case SDB_UNSUPPORTED: return "SDB_UNSUPPORTED";
        case SDB_CAPACITY: return "SDB_CAPACITY";
        case SDB_WORKSPACE_TOO_SMALL: return "SDB_WORKSPACE_TOO_SMALL";
        case SDB_DUP_KEY: return "SDB_DUP_KEY";
        case SDB_KEY_RANGE: return "SDB_KEY_RANGE";
        case SDB_HIP_ERROR: return "SDB_HIP_ERROR";
        default: return "SDB_UNKNOWN_STATUS";
    }
}

SDB_API int32_t sdb_abi_version(void) { return SDB_ABI_VERSION; }

SDB_API sdb_status sdb_struct_sizes(int64_t* sizes, int32_t n) {
    if (!sizes || n < 0 || n > 9) return fail(SDB_INVALID_ARG, "sizes must hold 0..9 entries");
    const int64_t all[9] = {(int64_t)sizeof(sdb_pred),  (int64_t)sizeof(sdb_dim_desc),
                            (int64_t)sizeof(sdb_dim),   (int64_t)sizeof(sdb_join),
                            (int64_t)sizeof(sdb_group_key), (int64_t)sizeof(sdb_agg),
                            (int64_t)sizeof(sdb_query), (int64_t)sizeof(sdb_plan),
                            (int64_t)sizeof(sdb_dim_summary)};
    for (int i = 0; i < n; ++i) sizes[i] = all[i];
    return ok();
}

SDB_API sdb_status sdb_dim_required_bytes(const sdb_dim_desc* desc, int64_t* bytes) {
    sdb_status st = check_dim_desc(desc);
    if (st != SDB_OK) return st;
    if (!bytes) return fail(SDB_INVALID_ARG, "null output");
    *bytes = (int64_t)required_bytes(desc);
    return ok();
}

SDB_API sdb_status sdb_build_dims(int32_t n_dims, const sdb_dim_desc* descs, void* const* workspaces,
                                  const int64_t* workspace_bytes, void* stream, sdb_dim* outs) {
    if (n_dims < 0 || n_dims > SDB_MAX_JOINS) return fail(SDB_INVALID_ARG, "n_dims %d is not in 0..%d", n_dims, SDB_MAX_JOINS);
    if (n_dims > 0 && (!descs || !workspaces || !workspace_bytes || !outs)) return fail(SDB_INVALID_ARG, "null argument");
    hipStream_t s = (hipStream_t)stream;
    BuildBatch bb;
    std::memset(&bb, 0, sizeof bb);
    bb.n = n_dims;
    BuildParams* bp = bb.bp;
    DimStats hs_stack[SDB_MAX_JOINS];
    DimStats* hs = hs_stack;   // pinned staging once the arguments have been checked
    // every table's arguments first, so nothing launches for an invalid batch
    for (int d = 0; d < n_dims; ++d) {
        const sdb_dim_desc* desc = &descs[d];
        sdb_status st = check_dim_desc(desc);
        if (st != SDB_OK) return fail(st, "dimension %d: %s", d, g_error.c_str());
        void* workspace = workspaces[d];
        if (!workspace) return fail(SDB_INVALID_ARG, "dimension %d: null workspace", d);
        if (((uintptr_t)workspace & 255u) != 0)
            return fail(SDB_INVALID_ARG, "dimension %d: workspace is not 256-byte aligned", d);
        const uint64_t need = required_bytes(desc);
        if (workspace_bytes[d] < 0 || (uint64_t)workspace_bytes[d] < need)
            return fail(SDB_WORKSPACE_TOO_SMALL, "dimension %d: workspace holds %lld bytes, %llu needed", d,
                        (long long)workspace_bytes[d], (unsigned long long)need);
        std::memset(&outs[d], 0, sizeof outs[d]);
    }

    // pass 1 for every table: statistics, read back with one synchronization
    for (int d = 0; d < n_dims; ++d) bp[d] = build_params(&descs[d], (DimStats*)workspaces[d]);
    if (void* pinned = host_staging()) hs = static_cast<DimStats*>(pinned);
    // the statistics kernels write the staging buffer themselves where it has a device address
    bb.host_stats = static_cast<DimStats*>(host_staging_device());
    SDB_HIP(launch_build_stats(bb, s), "dimension statistics launch");
    if (!bb.host_stats)
        for (int d = 0; d < n_dims; ++d)
            SDB_HIP(hipMemcpyAsync(&hs[d], workspaces[d], sizeof(DimStats), hipMemcpyDeviceToHost, s), "statistics copy");
    if (n_dims > 0) SDB_HIP(hipStreamSynchronize(s), "statistics sync");

    // pass 2 for every table: layout from the statistics, then the map or hash table
    int kinds[SDB_MAX_JOINS];
    for (int d = 0; d < n_dims; ++d) {
        const sdb_dim_desc* desc = &descs[d];
        sdb_dim* out = &outs[d];
        uint8_t* table = (uint8_t*)workspaces[d] + kStatsBytes;
        const int64_t n = desc->n_rows;
        out->n_rows = n;
        out->n_pass = (int64_t)hs[d].npass;
        out->key_min = n > 0 ? hs[d].kmin : 0;
        out->key_max = n > 0 ? hs[d].kmax : -1;
        out->pass_key_min = hs[d].npass > 0 ? hs[d].pkmin : 0;
        out->pass_key_max = hs[d].npass > 0 ? hs[d].pkmax : -1;
        out->n_payloads = desc->n_payloads;
        // payload codes: mixed radix over the payload ranges of passing rows, last payload fastest
        uint64_t domain = 1;
        for (int p = desc->n_payloads - 1; p >= 0; --p) {
            const bool any = hs[d].npass > 0;
            const int32_t lo = any ? hs[d].pmin[p] : 0;
            const uint64_t radix = any ? (uint64_t)((int64_t)hs[d].pmax[p] - (int64_t)lo + 1) : 1;
            out->payload_min[p] = lo;
            out->payload_div[p] = domain;
            if (radix > 0xFFFFFFFFull)
                return fail(SDB_UNSUPPORTED, "dimension %d: payload %d spans more than 2^32 - 1 values", d, p);
            out->payload_radix[p] = (uint32_t)radix;
            domain *= radix;
            if (domain >= 0xFFFFFFFEull)
                return fail(SDB_UNSUPPORTED, "dimension %d: payload domain reaches 2^32 - 2 codes", d);
        }
        out->domain = domain;

        const uint64_t range = n > 0 ? (uint64_t)((int64_t)out->key_max - (int64_t)out->key_min + 1) : 0;
        // the runtime dense-or-hash choice: by key range, or by the memory budget
        const int code_width = domain <= 0xFEull ? 1 : (domain <= 0xFFFEull ? 2 : 4);
        const bool in_budget = desc->dense_budget_bytes > 0 && range <= kMaxDenseSlots &&
                               dense_bytes(range, code_width) <= (uint64_t)desc->dense_budget_bytes;
        const bool dense_ok = range <= dense_slot_limit(n) || in_budget;
        int kind = desc->kind;
        if (kind == SDB_TABLE_AUTO) kind = dense_ok ? SDB_TABLE_DENSE : SDB_TABLE_HASH;
        if (kind == SDB_TABLE_DENSE && !dense_ok)
            return fail(SDB_KEY_RANGE, "dimension %d: key range %llu exceeds the dense limit %llu and the dense "
                        "budget of %lld bytes", d, (unsigned long long)range,
                        (unsigned long long)dense_slot_limit(n), (long long)desc->dense_budget_bytes);
        kinds[d] = kind;
        out->kind = kind;
        out->stats = workspaces[d];
        out->map = table;
        bp[d].kmin = out->key_min;
        for (int p = 0; p < desc->n_payloads; ++p) {
            bp[d].pmin[p] = out->payload_min[p];
            bp[d].pdiv[p] = (uint32_t)out->payload_div[p];
        }

        if (kind == SDB_TABLE_DENSE) {
            // codes stay below the two reserved top values of the width
            const int width = domain <= 0xFEull ? 1 : (domain <= 0xFFFEull ? 2 : 4);
            const uint32_t missing = width == 1 ? 0xFFu : (width == 2 ? 0xFFFFu : 0xFFFFFFFFu);
            out->width = width;
            out->sentinel = missing - 1u;
            out->n_slots = range;
            const uint64_t map_bytes = align_up(range * width, 256);
            uint32_t* pass_bits = (uint32_t*)(table + map_bytes);
            out->bits = pass_bits;
            bp[d].map = table;
            bp[d].pass_bits = pass_bits;
            bp[d].width = width;
            bp[d].nslots = range;
            bp[d].sentinel = missing - 1u;
            bp[d].missing = missing;
            bp[d].dense = 1;
            bp[d].fill_value = 0xFFFFFFFFu;
            bp[d].fill_words = map_bytes / 4;
        } else {
            const uint64_t cap = hash_capacity(n, effective_lf(desc));
            int bits = 0;
            while ((1ull << bits) < cap) ++bits;
            out->width = 8;
            out->sentinel = 0xFFFFFFFEu;   // code + 1 == 0xFFFFFFFF marks a filtered row
            out->n_slots = cap;
            out->hash_bits = bits;
            bp[d].map = table;
            bp[d].nslots = cap;
            bp[d].hmask = (uint32_t)(cap - 1);
            bp[d].hshift = 32 - bits;
            bp[d].dense = 0;
            bp[d].fill_value = 0u;
            // the pass filter after the slots: a bitmap over the key range when
            // it fits the filter's bytes, else the Bloom filter over all of them
            const uint64_t slot_bytes = align_up(cap * 8, 256), fbytes = filter_bytes(n);
            uint32_t* filt = (uint32_t*)(table + slot_bytes);
            const bool bitmap = range > 0 && range <= fbytes * 8;
            out->filter = filt;
            out->filter_kind = bitmap ? SDB_FILTER_BITMAP : SDB_FILTER_BLOOM;
            out->filter_bits = bitmap ? range : fbytes * 8;
            bp[d].filt = filt;
            bp[d].filt_kind = out->filter_kind;
            bp[d].filt_bits = out->filter_bits;
            // a bitmap goes through a byte per key in the slot region (no
            // atomics) when the range's bytes, rounded to whole words, fit
            // there; the slots are filled afterwards, the filter by the packing
            bp[d].filt_via_bytes = bitmap && align_up(range, 32) <= slot_bytes ? 1 : 0;
            bp[d].fill_words = (slot_bytes + (bp[d].filt_via_bytes ? 0 : fbytes)) / 4;
        }
    }

    SDB_HIP(launch_build_tables(bb, s), "table build launch");

    // duplicate-key checks of every table, with one synchronization
    if (bb.host_stats)
        SDB_HIP(launch_export_stats(bb, s), "flag export launch");
    else
        for (int d = 0; d < n_dims; ++d)
            SDB_HIP(hipMemcpyAsync(&hs[d], workspaces[d], sizeof(DimStats), hipMemcpyDeviceToHost, s), "flag copy");
    if (n_dims > 0) SDB_HIP(hipStreamSynchronize(s), "build sync");
    for (int d = 0; d < n_dims; ++d) {
        const DimStats& fin = hs[d];
        if (fin.dup & 1u) return fail(SDB_DUP_KEY, "dimension %d: key column holds a duplicate key", d);
        if (kinds[d] == SDB_TABLE_DENSE && fin.occupied != (unsigned long long)descs[d].n_rows)
            return fail(SDB_DUP_KEY, "dimension %d: key column holds a duplicate key (%llu distinct keys in %lld rows)",
                        d, (unsigned long long)fin.occupied, (long long)descs[d].n_rows);
        if (fin.dup) return fail(SDB_HIP_ERROR, "dimension %d: build inconsistency (flag %u)", d, fin.dup);
    }
    return ok();
}

SDB_API sdb_status sdb_dim_info(const sdb_dim* dim, sdb_dim_summary* out) {
    if (!dim || !out) return fail(SDB_INVALID_ARG, "null argument");
    const sdb_dim& d = *dim;
    if (d.kind != SDB_TABLE_DENSE && d.kind != SDB_TABLE_HASH)
        return fail(SDB_INVALID_ARG, "handle kind %d is neither DENSE nor HASH", d.kind);
    if (d.n_rows < 0 || d.n_pass < 0 || d.n_pass > d.n_rows)
        return fail(SDB_INVALID_ARG, "handle counts %lld passing of %lld rows", (long long)d.n_pass,
                    (long long)d.n_rows);
    if (d.n_payloads < 0 || d.n_payloads > SDB_MAX_PAYLOADS)
        return fail(SDB_INVALID_ARG, "handle has %d payloads", d.n_payloads);
    uint64_t table_bytes = 0;
    if (d.kind == SDB_TABLE_DENSE) {
        if (d.width != 1 && d.width != 2 && d.width != 4)
            return fail(SDB_INVALID_ARG, "dense handle with entry width %d", d.width);
        const uint64_t range = d.n_rows > 0 ? (uint64_t)((int64_t)d.key_max - (int64_t)d.key_min + 1) : 0;
        if (d.n_slots != range) return fail(SDB_INVALID_ARG, "dense handle: %llu slots for a key range of %llu",
                                            (unsigned long long)d.n_slots, (unsigned long long)range);
        if (d.n_slots > 0 && (!d.map || !d.bits)) return fail(SDB_INVALID_ARG, "dense handle without its map");
        table_bytes = dense_bytes(d.n_slots, d.width);
    } else {
        if (d.width != 8 || d.hash_bits < 1 || d.hash_bits > 32 || d.n_slots != (1ull << d.hash_bits))
            return fail(SDB_INVALID_ARG, "hash handle: width %d, %llu slots, hash_bits %d", d.width,
                        (unsigned long long)d.n_slots, d.hash_bits);
        if (!d.map) return fail(SDB_INVALID_ARG, "hash handle without its slots");
        table_bytes = d.n_slots * 8ull;
    }
    const std::string fp = filter_problem(&d);
    if (!fp.empty()) return fail(SDB_INVALID_ARG, "%s", fp.c_str());
    sdb_dim_summary o;
    std::memset(&o, 0, sizeof o);
    o.kind = d.kind;
    o.width = d.width;
    o.n_rows = d.n_rows;
    o.n_pass = d.n_pass;
    o.key_min = d.key_min;
    o.key_max = d.key_max;
    o.pass_key_min = d.pass_key_min;
    o.pass_key_max = d.pass_key_max;
    o.pass_keys_contiguous =
        d.n_pass > 0 && (int64_t)d.pass_key_max - (int64_t)d.pass_key_min + 1 == d.n_pass ? 1 : 0;
    o.n_payloads = d.n_payloads;
    o.n_slots = d.n_slots;
    o.table_bytes = table_bytes;
    o.occupancy = d.n_slots > 0 ? (double)d.n_rows / (double)d.n_slots : 0.0;
    o.filter_kind = d.filter_kind;
    o.filter_bytes = d.filter_kind != SDB_FILTER_NONE ? (d.filter_bits + 31) / 32 * 4 : 0;
    uint64_t domain = 1;
    for (int p = 0; p < d.n_payloads; ++p) {
        o.payload_min[p] = d.payload_min[p];
        o.payload_radix[p] = d.payload_radix[p];
        o.payload_max[p] = (int32_t)((int64_t)d.payload_min[p] + (int64_t)d.payload_radix[p] - 1);
        domain *= d.payload_radix[p];
    }
    o.domain = domain;
    *out = o;
    return ok();
}

SDB_API sdb_status sdb_build_dim(const sdb_dim_desc* desc, void* workspace, int64_t workspace_bytes,
                                 void* stream, sdb_dim* out) {
    if (!desc || !out) return fail(SDB_INVALID_ARG, "null argument");
    void* ws[1] = {workspace};
    const int64_t wb[1] = {workspace_bytes};
    return sdb_build_dims(1, desc, ws, wb, stream, out);
}

SDB_API sdb_status sdb_plan_star_query(const sdb_query* q, void* scratch, int64_t scratch_bytes,
                                       void* stream, sdb_plan* plan) {
    sdb_status st = check_query(q);
    if (st != SDB_OK) return st;
    if (!plan) return fail(SDB_INVALID_ARG, "null plan");
    std::memset(plan, 0, sizeof *plan);

    // stages in query order: predicates, then joins
    int n = 0;
    for (int i = 0; i < q->n_preds; ++i) {
        plan->stage_kind[n] = 0;
        plan->stage_index[n] = i;
        plan->stage_pass[n] = 0.5;
        ++n;
    }
    for (int j = 0; j < q->n_joins; ++j) {
        const sdb_dim* d = q->joins[j].dim;
        plan->stage_kind[n] = 1;
        plan->stage_index[n] = j;
        plan->stage_pass[n] = d->n_rows > 0 ? (double)d->n_pass / (double)d->n_rows : 0.0;
        ++n;
    }
    plan->n_stages = n;
    for (int s = 0; s < n; ++s) plan->stage_pass_alone[s] = plan->stage_pass[s];
    int bit[SDB_MAX_STAGES];   // query position of the stage at each plan position
    for (int s = 0; s < n; ++s) bit[s] = s;
    Sample smp;
    std::vector<Sample> range_smp;   // per run of sampled rows (segmented plans)
    int n_ranges = 1;
    int64_t sample_step = 0, sample_n = 0;
    for (int s = 0; s < SDB_MAX_STAGES; ++s) plan->stage_defer[s] = -1;
    if (q->force_range == 1)
        for (int s = 0; s < n; ++s)
            plan->stage_range[s] = plan->stage_kind[s] == 1 && range_eligible(q, plan->stage_index[s]);

    st = group_layout(q, plan);
    if (st != SDB_OK) return st;

    // the hash probe over table slices, where the query allows it
    int slice_j = (q->force_slice == -1 || q->force_eager > 0 || q->n_fact == 0) ? -1 : slice_join(q);
    if (slice_j >= 0 && q->force_slice != 1) {
        const sdb_dim* d = q->joins[slice_j].dim;
        if ((uint64_t)d->n_slots * 8u < kSliceMinTableBytes || q->n_fact < kSliceMinRows) slice_j = -1;
    }

    // terminal
    int term;
    if (q->force_terminal != SDB_TERMINAL_AUTO) term = q->force_terminal;
    else if (q->n_group_keys == 0) term = TERM_SCALAR;
    else if (plan->n_groups <= (uint64_t)kLdsGroupLimit) term = TERM_LDS;
    else term = TERM_GLOBAL;
    if (term == TERM_SCALAR && q->n_group_keys > 0)
        return fail(SDB_INVALID_ARG, "scalar terminal forced on a grouped query");
    if (term == TERM_LDS && plan->n_groups > (uint64_t)kLdsGroupLimit)
        return fail(SDB_CAPACITY, "LDS terminal holds at most %d groups, plan has %llu", kLdsGroupLimit,
                    (unsigned long long)plan->n_groups);
    if (term == TERM_PART && q->n_fact == 0) term = TERM_GLOBAL;
    plan->terminal = term;

    // pass fraction of every stage on a strided sample of the fact rows
    if (!q->force_order && n > 1 && q->n_fact > 0) {
        if (!scratch) return fail(SDB_INVALID_ARG, "null planner scratch");
        if (scratch_bytes < SDB_PLAN_SCRATCH_BYTES)
            return fail(SDB_WORKSPACE_TOO_SMALL, "planner scratch holds %lld bytes, %d needed",
                        (long long)scratch_bytes, SDB_PLAN_SCRATCH_BYTES);
        hipStream_t s = (hipStream_t)stream;
        FusedParams fp = fused_params(q, plan, false);
        // key histograms only where a window may be placed (windows are forced, never automatic)
        for (int i = 0; i < n; ++i) fp.st[i].sample_hist = q->force_window > 0 && q->force_lds != -1;
        const int64_t step = (q->n_fact + 65535) / 65536;
        const int64_t n_sample = (q->n_fact + step - 1) / step;
        uint32_t* dpattern = (uint32_t*)scratch;
        uint32_t* dkeys = (uint32_t*)((uint8_t*)scratch + kPatternBytes);
        // the sampled rows split into runs of rows for per-range stage orders
        n_ranges = (q->force_segments != -1 && n <= kSampleRangeStages && n_sample >= 64 * kSampleRanges)
                       ? kSampleRanges : 1;
        SDB_HIP(launch_sample(fp, step, n_sample, n_ranges, dpattern, dkeys, s), "sample launch");
        std::vector<uint8_t> fallback;
        uint8_t* host = static_cast<uint8_t*>(host_staging());
        if (!host) {
            fallback.resize(kPatternBytes + kKeyHistBytes);
            host = fallback.data();
        }
        const size_t pattern_bytes = (sizeof(uint32_t) << n) * (size_t)n_ranges;
        const size_t key_bytes = sizeof(uint32_t) * kKeyBuckets * (size_t)n;
        if (void* hdev = fallback.empty() ? host_staging_device() : nullptr) {
            // one kernel writes both histograms where the copies would put them
            SDB_HIP(launch_copy_out(dpattern, (uint32_t)(kPatternBytes / 4), dkeys, (uint32_t)(key_bytes / 4),
                                    static_cast<uint32_t*>(hdev), s), "sample export launch");
        } else {
            SDB_HIP(hipMemcpyAsync(host, dpattern, pattern_bytes, hipMemcpyDeviceToHost, s), "sample copy");
            SDB_HIP(hipMemcpyAsync(host + kPatternBytes, dkeys, key_bytes, hipMemcpyDeviceToHost, s), "sample copy");
        }
        SDB_HIP(hipStreamSynchronize(s), "sample sync");
        const uint32_t* ph = reinterpret_cast<const uint32_t*>(host);
        std::vector<uint32_t> whole((size_t)1 << n, 0u);
        range_smp.resize(n_ranges);
        for (int r = 0; r < n_ranges; ++r) {
            const uint32_t* h = ph + ((size_t)r << n);
            double rows = 0.0;
            for (size_t m = 0; m < whole.size(); ++m) {
                whole[m] += h[m];
                rows += h[m];
            }
            if (n_ranges > 1) joint_from_patterns(h, n, rows, &range_smp[r]);
        }
        joint_from_patterns(whole.data(), n, (double)n_sample, &smp);
        sample_step = step;
        sample_n = n_sample;
        const uint32_t* keys = reinterpret_cast<const uint32_t*>(host + kPatternBytes);
        smp.keys.assign((size_t)kMaxStages * kKeyBuckets, 0u);
        std::copy(keys, keys + (size_t)kKeyBuckets * n, smp.keys.begin());
        for (int i = 0; i < n; ++i) plan->stage_pass[i] = plan->stage_pass_alone[i] = smp.frac(1u << i);
        plan->sampled_rows = n_sample;
    }

    // LDS placement of small dense tables, then the cheapest stage order
    if (q->force_lds != -1) place_lds(q, plan, (uint64_t)kLdsStageBudget);
    // Probes left to device-memory lookups become key-range predicates where
    // they can (an LDS lookup costs about as much as the compare: measured).
    if (q->force_range == 0)
        for (int s = 0; s < n; ++s)
            plan->stage_range[s] = plan->stage_kind[s] == 1 && plan->stage_lds[s] == LDS_GLOBAL &&
                                   range_eligible(q, plan->stage_index[s]);
    for (int s = 0; s < n; ++s)
        if (plan->stage_kind[s] == 1 && plan->stage_range[s]) slice_j = -1;   // the probe became a compare
    if (!q->force_order && n > 1) {
        choose_order(q, plan, bit, &smp);
    } else {
        int order[SDB_MAX_STAGES];
        for (int i = 0; i < n; ++i) order[i] = i;
        plan->est_cost = order_cost(q, plan, order, n, Reach{plan, &smp, bit});
    }
    // stage orders of their own for runs of rows that favour one
    plan->n_segments = 1;
    for (int i = 0; i < n; ++i) plan->segment_order[0][i] = i;
    plan->segment_start[0] = 0;
    plan->segment_start[1] = q->n_fact;
    std::vector<double> seg_survivors;
    if (n_ranges > 1 && slice_j < 0 && q->force_eager <= 0)
        choose_segments(q, plan, bit, range_smp, sample_step, sample_n, &seg_survivors);
    // the first LDS-bitmap stage that carries group keys gathers its code after all stages
    for (int s = 0; s < n; ++s) {
        if (plan->stage_kind[s] != 1 || plan->stage_lds[s] != LDS_BITS) continue;
        bool gathers = false;
        for (int k = 0; k < q->n_group_keys; ++k) gathers |= q->group_keys[k].join == plan->stage_index[s];
        if (gathers) {
            plan->stage_defer[s] = 0;
            break;
        }
    }
    plan->lds_bytes = (int32_t)lds_layout(q, plan, nullptr);

    // (a sliced probe's fused kernel reads the partitioned records, which are aligned)
    const bool aligned = columns_aligned(q, plan) || slice_j >= 0;
    if (q->force_vector == 1 && !aligned && q->n_fact > 0)
        return fail(SDB_INVALID_ARG, "vector loads forced but a column is not 16-byte aligned");
    plan->vector = q->force_vector == -1 ? 0 : (aligned ? 1 : 0);
    plan->grid = q->grid_blocks;

    // large group tables with many survivors: partitioned aggregation
    double f = 1.0;
    for (int s = 0; s < n; ++s) f *= plan->stage_pass[s];
    const double survivors = f * (double)q->n_fact;
    if (term == TERM_GLOBAL || term == TERM_PART) {
        // the largest partitions the LDS table holds: long runs in the scatter
        int shift = 0;
        while (shift < kPartMaxShift && (1ull << shift) < plan->n_groups) ++shift;
        const uint64_t parts = (plan->n_groups + (1ull << shift) - 1) >> shift;
        const bool fits = parts <= (uint64_t)kPartMaxParts;
        // chosen automatically for many survivors per group (measured: c3,
        // 55 per group, 2.47 against 2.76 ms with per-XCD atomics; c4, about
        // 6 per group, 2.52 against 1.63 ms the other way round)
        bool part = term == TERM_PART ||
                    (q->force_terminal == SDB_TERMINAL_AUTO && fits && q->n_fact > 0 && survivors >= 1.0e6 &&
                     survivors >= kPartMinPerGroup * (double)plan->n_groups);
        if (part && !fits)
            return fail(SDB_CAPACITY, "partitioned terminal needs at most %d partitions of %d groups",
                        kPartMaxParts, 1 << kPartMaxShift);
        if (part) {
            term = TERM_PART;
            plan->terminal = TERM_PART;
            plan->part_shift = shift;
            plan->n_parts = (int32_t)parts;
        }
    }

    // Items per lane and block size, measured on the five workloads: plans
    // with two or more lookups in device memory (dense maps outside LDS, hash
    // tables) run fastest with one 4-row item per lane in blocks of 1024
    // (more waves in flight per CU); the others with two items per lane in
    // blocks of 512. 1-row items keep blocks of 256.
    // (a sliced hash probe reads mostly L2-resident slots: one lookup; measured
    // on c5, two items per lane in blocks of 512 run its fused kernel in 12.0
    // against 12.4 ms for one item in blocks of 1024)
    int device_lookups = 0;
    for (int s = 0; s < n; ++s) {
        if (plan->stage_kind[s] != 1 || plan->stage_range[s]) continue;
        const sdb_dim* d = q->joins[plan->stage_index[s]].dim;
        if (d->kind == SDB_TABLE_HASH) device_lookups += slice_j >= 0 ? 1 : 2;
        else if (plan->stage_lds[s] == LDS_GLOBAL) device_lookups += 1;
    }
    const bool many_waves = plan->vector && device_lookups >= 2 && q->force_eager <= 0;
    plan->ipt = q->force_ipt ? q->force_ipt : (many_waves ? 1 : kDefaultIpt);
    if (q->force_block) plan->block = q->force_block;
    else if (!plan->vector) plan->block = kBlock;
    else plan->block = many_waves && plan->ipt <= 2 ? kBigBlock : kMaxBlock;
    if (plan->block == kBigBlock && (!plan->vector || plan->ipt > 2))
        return fail(SDB_INVALID_ARG, "blocks of %d threads need 4-row items and ipt 1 or 2", kBigBlock);

    // eager columns: those whose lines the kernel reads anyway (enough rows
    // still live where the column is first used)
    plan->eager = 0;
    if (q->force_eager > 0 && (!plan->vector || plan->ipt > 2 || plan->block == kBigBlock))
        return fail(SDB_INVALID_ARG, "eager loads need 4-row items, ipt 1 or 2 and blocks of at most %d", kMaxBlock);
    if (plan->vector && plan->ipt <= 2 && plan->block <= kMaxBlock && q->n_fact > 0 && q->force_eager >= 0 &&
        slice_j < 0) {
        int cols[SDB_MAX_FACT_COLS];
        double live[SDB_MAX_FACT_COLS];
        const int n_used = columns_in_use_order(q, plan, cols, live);
        int k = 0;
        if (q->force_eager > 0) {
            k = std::min(q->force_eager, n_used);
        } else if (kAutoEager) {
            while (k < n_used && k < kMaxEager && live[k] >= kEagerMinLive) ++k;
        }
        plan->eager = k;
    }

    // An LDS window for the dense device-memory stage it helps most; with it a
    // block's LDS leaves room for one block per CU, so 4-row items run in
    // blocks of 1024 (16 waves per CU).
    if (plan->vector && plan->ipt <= 2 && plan->eager == 0 && slice_j < 0 &&
        (q->force_block == 0 || q->force_block == kBigBlock)) {
        const int block_before = plan->block;
        plan->block = kBigBlock;
        plan->lds_bytes = (int32_t)lds_layout(q, plan, nullptr);
        if (place_window(q, plan, smp, bit, q->n_fact) < 0) plan->block = block_before;
    } else if (q->force_window > 0 && slice_j < 0) {
        plan->lds_bytes = (int32_t)lds_layout(q, plan, nullptr);
        place_window(q, plan, smp, bit, q->n_fact);
    }

    // LDS rank tables instead of the deferred gather of a bitmap stage's code.
    // Their LDS footprint leaves one block of 1024 per CU, which pays when no
    // other lookup goes to device memory (measured: c2 0.185 -> 0.173 ms) or
    // when the plan runs two items per lane, whose registers allow no more
    // than 16 waves per CU anyway (c3: fused kernel 2.234 -> 2.195 ms, 21M
    // deferred gathers spared), not when a lookup-heavy plan runs one item per
    // lane at 32 waves per CU (c4: 1.67 -> 2.67 ms).
    const bool want_rank = q->force_lds == 3 ||
                           (q->force_lds == 0 && (device_lookups == 0 || (plan->ipt == 2 && plan->vector)));
    if (want_rank && plan->vector && plan->ipt <= 2 && plan->eager == 0 &&
        (q->force_block == 0 || q->force_block == kBigBlock)) {
        for (int s = 0; s < n; ++s) {
            if (plan->stage_defer[s] != 0 || !rank_fits(q->joins[plan->stage_index[s]].dim)) continue;
            plan->stage_lds[s] = LDS_RANK;
            plan->stage_defer[s] = -1;
            const int block_before = plan->block;
            plan->block = kBigBlock;
            if (lds_layout(q, plan, nullptr) + ring_lds_bytes(q, plan) > kLdsUsable) {   // keep the bitmap
                plan->stage_lds[s] = LDS_BITS;
                plan->stage_defer[s] = 0;
                plan->block = block_before;
            }
        }
    }
    // coarse LDS pre-filters for dense tables left in device memory
    if (q->force_coarse > 0) {
        for (int s = 0; s < n; ++s) {
            if (plan->stage_kind[s] != 1 || plan->stage_lds[s] != LDS_GLOBAL || plan->stage_range[s]) continue;
            if (!coarse_fits_table(q->joins[plan->stage_index[s]].dim)) continue;
            plan->stage_lds[s] = LDS_COARSE;
            plan->stage_coarse[s] = q->force_coarse;
            if (lds_layout(q, plan, nullptr) + ring_lds_bytes(q, plan) > kLdsUsable) {
                plan->stage_lds[s] = LDS_GLOBAL;
                plan->stage_coarse[s] = 0;
            }
        }
    }
    plan->lds_bytes = (int32_t)lds_layout(q, plan, nullptr);
    const uint64_t stage_bytes = stage_scratch_bytes(q, plan);
    plan->unroll = (q->force_unroll != -1 && slice_j < 0 && unroll_allowed(q, plan)) ? 1 : 0;

    // per-XCD private group tables for the global terminal when enough rows survive
    const uint64_t copy_bytes = (uint64_t)kXcdCopies * plan->n_groups * 16;
    bool xcd = term == TERM_GLOBAL && survivors >= 2.0 * (double)plan->n_groups && copy_bytes <= (1ull << 30);
    if (q->force_xcd == 1) xcd = term == TERM_GLOBAL;
    if (q->force_xcd == -1) xcd = false;
    plan->xcd_copies = xcd ? kXcdCopies : 0;
    plan->run_scratch_bytes = (int64_t)stage_bytes + (xcd ? (int64_t)copy_bytes : 0);

    if (term == TERM_PART) {
        // records are written per block: the grid is fixed now
        if (plan->grid <= 0) {
            int grid = 0;
            st = choose_grid(q, plan, &grid);
            if (st != SDB_OK) return st;
            plan->grid = grid;
        }
        // record regions per block: about kPartRegions in all, so that the
        // scatter pass runs several blocks per CU, where its blocks have few
        // records each and wait on latency (measured on c3, grid 256, 80K
        // records per block: 92 against 167 us with 4 regions per block);
        // blocks with many records already keep it near bandwidth (c5, 586K
        // per block: 1.10 ms with one region, 1.16 ms with 2 or 4)
        plan->part_subs = survivors / std::max(1, plan->grid) >= kPartSplitMaxRecords
                              ? 1
                              : (int32_t)std::max<int64_t>(
                                    1, std::min<int64_t>(kPartSubRegions, kPartRegions / std::max(1, plan->grid)));
        // records per block: 1.5 x the survivors the busiest launch (segment) expects
        double seg_rows = (double)q->n_fact, seg_surv = survivors;
        if (plan->n_segments > 1) {
            seg_rows = 0.0;
            seg_surv = 0.0;
            for (int g = 0; g < plan->n_segments; ++g) {
                seg_rows = std::max(seg_rows, (double)(plan->segment_start[g + 1] - plan->segment_start[g]));
                seg_surv = std::max(seg_surv, seg_survivors[g]);
            }
        }
        // (records per region: each of a block's part_subs regions takes the
        // records of its share of the block's waves)
        const double launch_regions = (double)plan->grid * plan->part_subs;
        const double cap_total = std::min(seg_rows, 1.5 * seg_surv + 256.0 * launch_regions);
        plan->part_cap = (int64_t)std::ceil(cap_total / launch_regions);
        plan->part_cap = (int64_t)align_up((uint64_t)std::max<int64_t>(plan->part_cap, 64), 64);
        const uint64_t regions = part_regions(plan);
        if ((uint64_t)plan->part_cap * regions > 0xFFFFFFF0ull)
            plan->part_cap = (int64_t)(0xFFFFFFF0ull / regions) / 64 * 64;
        plan->run_scratch_bytes = (int64_t)stage_bytes + (int64_t)part_layout(q, plan).total;
    }
    if (slice_j >= 0) {
        plan->slice_bits = slice_bits_for(q->joins[slice_j].dim);
        for (int s = 0; s < n; ++s)
            if (plan->stage_kind[s] == 1) plan->slice_stage = s;
        plan->slice_grid = (int32_t)std::min<int64_t>(
            kSliceMaxGrid, std::max<int64_t>(1, (q->n_fact + kSliceChunk - 1) / kSliceChunk));
        // pre-filter by the table's pass filter when enough rows would drop:
        // each row costs one filter read in the count pass, each dropped row
        // saves its scatter write and its probe
        const sdb_dim* d = q->joins[slice_j].dim;
        if (d->filter_kind != SDB_FILTER_NONE && q->force_prefilter != -1) {
            const int ss = plan->slice_stage;
            const double p = plan->sampled_rows > 0 ? plan->stage_pass_alone[ss] : plan->stage_pass[ss];
            const double fp = d->filter_kind == SDB_FILTER_BLOOM ? bloom_false_positive(d->filter_bits, d->n_pass) : 0.0;
            plan->slice_prefilter = (q->force_prefilter == 1 || p + (1.0 - p) * fp <= kPrefilterMaxKept) ? 1 : 0;
        }
        plan->run_scratch_bytes += (int64_t)slice_layout(q, plan).total;
    }
    return ok();
}

SDB_API sdb_status sdb_run_star_query(const sdb_query* q, const sdb_plan* plan, int64_t* sums,
                                      int64_t* counts, int64_t n_groups_capacity, void* scratch,
                                      int64_t scratch_bytes, void* stream) {
    sdb_status st = check_run(q, plan, sums, counts, n_groups_capacity);
    if (st != SDB_OK) return st;
    if (plan->terminal < TERM_SCALAR || plan->terminal > TERM_PART)
        return fail(SDB_INVALID_ARG, "bad plan terminal %d", plan->terminal);
    if (plan->terminal == TERM_PART) {
        if (plan->grid <= 0 || plan->part_cap <= 0 || plan->part_shift < 0 || plan->part_shift > kPartMaxShift ||
            plan->n_parts <= 0 || plan->n_parts > kPartMaxParts ||
            (uint64_t)plan->n_parts != ((plan->n_groups + (1ull << plan->part_shift) - 1) >> plan->part_shift) ||
            plan->part_subs < 1 || plan->part_subs > kPartSubRegions ||
            (uint64_t)plan->part_cap * part_regions(plan) > 0xFFFFFFFFull)
            return fail(SDB_INVALID_ARG, "bad partitioned-terminal plan");
    }
    if (plan->n_segments < 0 || plan->n_segments > SDB_MAX_SEGMENTS)
        return fail(SDB_INVALID_ARG, "bad plan n_segments %d", plan->n_segments);
    if (plan->n_segments > 1) {
        if (plan->eager != 0 || plan->slice_bits != 0)
            return fail(SDB_INVALID_ARG, "a segmented plan needs no eager loads and no table slices");
        if (plan->segment_start[0] != 0 || plan->segment_start[plan->n_segments] != q->n_fact)
            return fail(SDB_INVALID_ARG, "plan segments do not cover the fact rows");
        for (int g = 0; g < plan->n_segments; ++g) {
            const int64_t a = plan->segment_start[g], b = plan->segment_start[g + 1];
            if (b <= a || a % kSegmentAlign != 0)
                return fail(SDB_INVALID_ARG, "plan segment %d: rows %lld .. %lld (starts are increasing "
                            "multiples of %lld)", g, (long long)a, (long long)b, (long long)kSegmentAlign);
            bool seen[SDB_MAX_STAGES] = {false};
            for (int i = 0; i < plan->n_stages; ++i) {
                const int o = plan->segment_order[g][i];
                if (o < 0 || o >= plan->n_stages || seen[o])
                    return fail(SDB_INVALID_ARG, "plan segment %d: the order is not a permutation of the stages", g);
                seen[o] = true;
            }
        }
    }
    if (plan->terminal == TERM_SCALAR && q->n_group_keys > 0)
        return fail(SDB_INVALID_ARG, "scalar terminal on a grouped query");
    if (plan->terminal == TERM_LDS && plan->n_groups > (uint64_t)kLdsGroupLimit)
        return fail(SDB_CAPACITY, "LDS terminal holds at most %d groups", kLdsGroupLimit);
    if (plan->ipt != 1 && plan->ipt != 2 && plan->ipt != 4)
        return fail(SDB_INVALID_ARG, "bad plan ipt %d", plan->ipt);
    if (plan->block != 64 && plan->block != 128 && plan->block != 256 && plan->block != kMaxBlock &&
        plan->block != kBigBlock)
        return fail(SDB_INVALID_ARG, "bad plan block %d", plan->block);
    if (plan->block == kBigBlock && (!plan->vector || plan->ipt > 2 || plan->eager > 0))
        return fail(SDB_INVALID_ARG, "blocks of %d threads need 4-row items, ipt 1 or 2 and no eager loads",
                    kBigBlock);
    const bool sliced = plan->slice_bits != 0;
    if (sliced) {
        const int sj = slice_join(q);
        const int ss = plan->slice_stage;
        if (plan->slice_bits < 1 || plan->slice_bits > SDB_MAX_SLICE_BITS || sj < 0 || ss < 0 ||
            ss >= plan->n_stages || plan->stage_kind[ss] != 1 || plan->stage_index[ss] != sj ||
            plan->stage_range[ss] != 0 || plan->slice_bits > q->joins[sj].dim->hash_bits || plan->slice_grid < 1 ||
            plan->slice_grid > kSliceMaxGrid || plan->eager != 0)
            return fail(SDB_INVALID_ARG, "bad sliced-probe plan");
    }
    if (plan->slice_prefilter != 0 &&
        (plan->slice_prefilter != 1 || !sliced ||
         q->joins[plan->stage_index[plan->slice_stage]].dim->filter_kind == SDB_FILTER_NONE))
        return fail(SDB_INVALID_ARG, "slice_prefilter %d needs a sliced probe into a table with a pass filter",
                    plan->slice_prefilter);
    if (plan->unroll != 0 && (plan->unroll != 1 || !unroll_allowed(q, plan)))
        return fail(SDB_INVALID_ARG, "bad plan unroll %d (needs at most %d stages, 4-row items, ipt 2, blocks of "
                    "%d or %d, no eager loads, no hash probe and no table slices)", plan->unroll, kUnrollStages,
                    kMaxBlock, kBigBlock);
    if (plan->vector && q->n_fact > 0 && !sliced && !columns_aligned(q, plan))
        return fail(SDB_INVALID_ARG, "vector plan but a column is not 16-byte aligned");
    if (plan->eager < 0 || plan->eager > kMaxEager || (plan->eager > 0 && (!plan->vector || plan->ipt > 2)))
        return fail(SDB_INVALID_ARG, "bad plan eager %d (needs 4-row items and ipt 1 or 2)", plan->eager);
    if (plan->xcd_copies != 0 && (plan->xcd_copies != kXcdCopies || plan->terminal != TERM_GLOBAL))
        return fail(SDB_INVALID_ARG, "bad plan xcd_copies %d", plan->xcd_copies);
    // run scratch: the rank tables, then the terminal's part
    const uint64_t stage_bytes = stage_scratch_bytes(q, plan);
    uint64_t term_scratch = plan->xcd_copies ? (uint64_t)plan->xcd_copies * plan->n_groups * 16 : 0;
    if (plan->terminal == TERM_PART) term_scratch = part_layout(q, plan).total;
    const SliceLayout SL = slice_layout(q, plan);
    const uint64_t need_scratch = stage_bytes + SL.total + term_scratch;
    if (need_scratch) {
        if (!scratch) return fail(SDB_INVALID_ARG, "null run scratch");
        if (((uintptr_t)scratch & 255u) != 0) return fail(SDB_INVALID_ARG, "run scratch is not 256-byte aligned");
        if (scratch_bytes < 0 || (uint64_t)scratch_bytes < need_scratch)
            return fail(SDB_WORKSPACE_TOO_SMALL, "run scratch holds %lld bytes, %llu needed",
                        (long long)scratch_bytes, (unsigned long long)need_scratch);
    }

    FusedParams p = fused_params(q, plan, true);
    if ((int64_t)lds_layout(q, plan, nullptr) != (int64_t)plan->lds_bytes)
        return fail(SDB_INVALID_ARG, "plan LDS size does not match the tables");
    const uint32_t lds_bytes = launch_lds_bytes(q, plan);
    if (lds_bytes > 160u * 1024u) return fail(SDB_UNSUPPORTED, "plan needs %u bytes of LDS", lds_bytes);
    p.ring_off = (uint32_t)plan->lds_bytes;

    hipStream_t s = (hipStream_t)stream;
    uint8_t* slice_base = (uint8_t*)scratch + stage_bytes;
    uint8_t* term_base = slice_base + SL.total;
    SliceParams sp;
    std::memset(&sp, 0, sizeof sp);
    if (sliced) {
        // the count and scatter passes evaluate the predicates and write the
        // probe keys and aggregate values partitioned by slice; the fused
        // kernel runs the probe alone over them, up to the count they wrote
        const int ss = plan->slice_stage;
        for (int c = 0; c < q->n_cols; ++c) sp.cols[c] = q->cols[c];
        sp.n = q->n_fact;
        const int64_t per = (q->n_fact + plan->slice_grid - 1) / plan->slice_grid;
        sp.rows_per_block = (per + kSliceChunk - 1) / kSliceChunk * kSliceChunk;
        sp.key_col = q->joins[plan->stage_index[ss]].fact_key_col;
        sp.val_col = q->agg.a;
        sp.val2_col = q->agg.kind != SDB_AGG_COL ? q->agg.b : -1;
        sp.bits = plan->slice_bits;
        for (int st_i = 0; st_i < plan->n_stages; ++st_i) {
            if (plan->stage_kind[st_i] != 0) continue;
            const sdb_pred& pr = q->preds[plan->stage_index[st_i]];
            sp.pred_col[sp.n_preds] = pr.col;
            sp.pred[sp.n_preds] = lower_pred(pr);
            ++sp.n_preds;
        }
        sp.hist = (uint32_t*)(slice_base + SL.hist);
        sp.part_count = (uint32_t*)(slice_base + SL.part_count);
        sp.part_start = (uint32_t*)(slice_base + SL.part_start);
        sp.chunk_start = (uint32_t*)(slice_base + SL.chunk_start);
        sp.out_key = (int32_t*)(slice_base + SL.out_key);
        sp.out_val = (int32_t*)(slice_base + SL.out_val);
        sp.out_val2 = sp.val2_col >= 0 ? (int32_t*)(slice_base + SL.out_val2) : nullptr;
        if (plan->slice_prefilter) {
            const sdb_dim* fd = q->joins[plan->stage_index[ss]].dim;
            sp.filt = (const uint32_t*)fd->filter;
            sp.filt_bits = fd->filter_bits;
            sp.filt_kind = fd->filter_kind;
            sp.filt_key_min = fd->key_min;
            sp.keep = slice_base + SL.keep;
        }
        sp.tile_rows = SL.tile_rows;
        sp.tile_base = (uint32_t*)(slice_base + SL.tile_base);
        sp.tile_map = (int32_t*)(slice_base + SL.tile_map);
        sp.n_vtiles = SL.n_vtiles;
        StageDev hs = p.st[ss];
        hs.col = 0;
        hs.eg_slot = -1;
        hs.op = OP_HASH_PAIR;   // its slots are mostly in L2: fewer requests pay
        FusedParams p3;
        std::memset(&p3, 0, sizeof p3);
        p3.cols[0] = sp.out_key;
        p3.cols[1] = sp.out_val;
        p3.cols[2] = sp.out_val2;   // two-column aggregates only
        p3.n = q->n_fact;
        p3.n_dev = sp.part_start + (1u << plan->slice_bits);
        p3.tile_map = sp.tile_map;
        p3.n_vtiles = sp.n_vtiles;
        p3.nstages = 1;
        p3.st[0] = hs;
        p3.agg_kind = q->agg.kind;
        p3.agg_a = 1;
        p3.agg_b = sp.val2_col >= 0 ? 2 : 1;
        p3.agg_a_slot = -1;
        p3.agg_b_slot = -1;
        p3.defer_stage = -1;
        p3.n_groups = p.n_groups;
        p3.ring_off = p.ring_off;
        p = p3;
    }
    {
        // the rank tables of LDS_RANK stages and the coarse bitmaps of
        // LDS_COARSE stages, derived from their pass bitmaps and maps
        uint64_t off = 0;
        for (int st_i = 0; st_i < plan->n_stages; ++st_i) {
            if (plan->stage_lds[st_i] == LDS_COARSE) {
                const sdb_dim* d = q->joins[plan->stage_index[st_i]].dim;
                CoarseParams cp;
                cp.bits = (const uint32_t*)d->bits;
                cp.nslots = (uint32_t)d->n_slots;
                cp.shift = (uint32_t)plan->stage_coarse[st_i];
                cp.out = (uint32_t*)((uint8_t*)scratch + off);
                cp.n_words = (uint32_t)(coarse_bits_bytes(d, plan->stage_coarse[st_i]) / 4);
                off += scratch_part(coarse_bits_bytes(d, plan->stage_coarse[st_i]));
                p.st[st_i].bits = cp.out;
                if (q->n_fact > 0) SDB_HIP(launch_coarse_build(cp, s), "coarse bitmap launch");
                continue;
            }
            if (plan->stage_lds[st_i] != LDS_RANK) continue;
            const sdb_dim* d = q->joins[plan->stage_index[st_i]].dim;
            RankParams rp;
            rp.bits = (const uint32_t*)d->bits;
            rp.map = d->map;
            rp.width = d->width;
            rp.nslots = (uint32_t)d->n_slots;
            rp.prefix = (uint32_t*)((uint8_t*)scratch + off);
            off += scratch_part(lds_rank_bytes(d));
            rp.codes = (uint8_t*)scratch + off;
            off += scratch_part(lds_codes_bytes(d));
            p.st[st_i].rank = rp.prefix;
            p.st[st_i].codes = rp.codes;
            if (q->n_fact > 0) SDB_HIP(launch_rank_build(rp, s), "rank table launch");
        }
    }
    if (plan->xcd_copies) {
        SDB_HIP(launch_fill_u64((unsigned long long*)term_base, term_scratch / 8, s), "copy fill");
    } else {
        SDB_HIP(launch_zero_pair((unsigned long long*)sums, (unsigned long long*)counts, plan->n_groups, s),
                "output fill");
    }
    p.sums = (unsigned long long*)sums;
    p.counts = (unsigned long long*)counts;
    p.xcd_copies = plan->xcd_copies;
    p.xtab = plan->xcd_copies ? (unsigned long long*)term_base : nullptr;
    PartParams pp;
    std::memset(&pp, 0, sizeof pp);
    if (plan->terminal == TERM_PART) {
        const PartLayout L = part_layout(q, plan);
        uint8_t* base = term_base;
        p.region_count = (uint32_t*)(base + L.region_count);
        p.rec_gid = (uint32_t*)(base + L.rec_gid);
        p.rec_val = base + L.rec_val;
        p.rec_wide = records_wide(q) ? 1 : 0;
        p.part_hist = (uint32_t*)(base + L.part_hist);
        p.part_cap = (uint32_t)plan->part_cap;
        p.part_shift = plan->part_shift;
        p.n_parts = (uint32_t)plan->n_parts;
        p.part_subs = (uint32_t)plan->part_subs;
        pp.n_groups = plan->n_groups;
        pp.part_shift = plan->part_shift;
        pp.n_parts = (uint32_t)plan->n_parts;
        pp.n_regions = (uint32_t)part_regions(plan);
        pp.part_cap = (uint32_t)plan->part_cap;
        pp.region_count = p.region_count;
        pp.rec_gid = p.rec_gid;
        pp.rec_val = p.rec_val;
        pp.rec_wide = p.rec_wide;
        pp.part_hist = p.part_hist;
        pp.part_count = (uint32_t*)(base + L.part_count);
        pp.part_start = (uint32_t*)(base + L.part_start);
        pp.chunk_start = (uint32_t*)(base + L.chunk_start);
        pp.sorted_gid = (uint32_t*)(base + L.sorted_gid);
        pp.sorted_val = base + L.sorted_val;
        pp.item_sum = (unsigned long long*)(base + L.item_sum);
        pp.item_cnt = (uint32_t*)(base + L.item_cnt);
        pp.sums = p.sums;
        pp.counts = p.counts;
    }
    if (q->n_fact > 0) {
        int grid = plan->grid;
        if (grid <= 0) {
            st = choose_grid(q, plan, &grid);
            if (st != SDB_OK) return st;
        }
        const bool timed = g_fused_start && g_fused_stop;
        if (timed) SDB_HIP(hipEventRecord(g_fused_start, s), "event record");
        if (sliced) SDB_HIP(launch_slice_partition(sp, plan->slice_grid, s), "slice passes launch");
        const int segs = std::max(1, plan->n_segments);
        p.n_regions = (uint32_t)((uint64_t)grid * (uint64_t)segs * (uint64_t)plan->part_subs);
        for (int g = 0; g < segs; ++g) {
            // segment g: its rows, its stage order, its own block regions
            FusedParams pg = p;
            if (segs > 1) {
                const int64_t a = plan->segment_start[g], b = plan->segment_start[g + 1];
                for (int c = 0; c < q->n_cols; ++c) pg.cols[c] = q->cols[c] + a;
                pg.n = b - a;
                pg.defer_stage = -1;
                for (int i = 0; i < plan->n_stages; ++i) {
                    const int o = plan->segment_order[g][i];
                    pg.st[i] = p.st[o];
                    if (o == p.defer_stage) pg.defer_stage = i;
                }
                pg.region_base = (uint32_t)((uint64_t)g * (uint64_t)grid);
            }
            SDB_HIP(launch_fused(pg, plan->vector, plan->ipt, plan->terminal, plan->eager, plan->unroll, grid,
                                 plan->block, lds_bytes, s),
                    "fused kernel launch");
        }
        if (timed) SDB_HIP(hipEventRecord(g_fused_stop, s), "event record");
        if (plan->terminal == TERM_PART) SDB_HIP(launch_part_passes(pp, s), "partition passes launch");
    }
    if (plan->xcd_copies)
        SDB_HIP(launch_xcd_merge((const unsigned long long*)term_base, plan->xcd_copies, plan->n_groups,
                                 (unsigned long long*)sums, (unsigned long long*)counts, s),
                "copy merge launch");
    return ok();
}

SDB_API sdb_status sdb_run_star_query_noalloc(const sdb_query* q, const sdb_plan* plan, int64_t* sums,
                                              int64_t* counts, int64_t n_groups_capacity, void* stream) {
    sdb_status st = check_run(q, plan, sums, counts, n_groups_capacity);
    if (st != SDB_OK) return st;
    if (plan->run_scratch_bytes < 0 || (uint64_t)plan->run_scratch_bytes > kNoallocScratchBytes)
        return fail(SDB_WORKSPACE_TOO_SMALL,
                    "the plan needs %lld bytes of run scratch; the fixed scratch of the allocation-free run holds "
                    "%llu (plan with the global terminal, no per-XCD copies and no table slices)",
                    (long long)plan->run_scratch_bytes, (unsigned long long)kNoallocScratchBytes);
    void* fixed = nullptr;
    SDB_HIP(noalloc_scratch(&fixed), "fixed run scratch address");
    return sdb_run_star_query(q, plan, sums, counts, n_groups_capacity, fixed, (int64_t)kNoallocScratchBytes,
                              stream);
}

SDB_API sdb_status sdb_baseline_scratch_bytes(int64_t n_fact, int64_t* bytes) {
    if (!bytes) return fail(SDB_INVALID_ARG, "null argument");
    if (n_fact < 0) return fail(SDB_INVALID_ARG, "negative n_fact");
    *bytes = (int64_t)(align_up((uint64_t)n_fact, 256) + align_up((uint64_t)n_fact * 4, 256));
    return ok();
}

SDB_API sdb_status sdb_run_star_query_baseline(const sdb_query* q, const sdb_plan* plan, int32_t mode,
                                               int64_t* sums, int64_t* counts, int64_t n_groups_capacity,
                                               void* scratch, int64_t scratch_bytes, void* stream) {
    sdb_status st = check_run(q, plan, sums, counts, n_groups_capacity);
    if (st != SDB_OK) return st;
    if (mode != SDB_BASELINE_PER_OPERATOR && mode != SDB_BASELINE_GLOBAL_HANDOFF)
        return fail(SDB_INVALID_ARG, "unknown baseline mode %d", (int)mode);
    int64_t need = 0;
    sdb_baseline_scratch_bytes(q->n_fact, &need);
    if (need > 0) {
        if (!scratch) return fail(SDB_INVALID_ARG, "null run scratch");
        if (((uintptr_t)scratch & 255u) != 0) return fail(SDB_INVALID_ARG, "run scratch is not 256-byte aligned");
        if (scratch_bytes < need)
            return fail(SDB_WORKSPACE_TOO_SMALL, "run scratch holds %lld bytes, %lld needed", (long long)scratch_bytes,
                        (long long)need);
    }
    // stages in the plan's order, every table read in device memory
    FusedParams p;
    std::memset(&p, 0, sizeof p);
    for (int c = 0; c < q->n_cols; ++c) p.cols[c] = q->cols[c];
    p.n = q->n_fact;
    p.nstages = plan->n_stages;
    for (int s = 0; s < plan->n_stages; ++s)
        p.st[s] = make_stage(q, plan, plan->stage_kind[s], plan->stage_index[s], -1);
    p.agg_kind = q->agg.kind;
    p.agg_a = q->agg.a;
    p.agg_b = q->agg.kind == SDB_AGG_COL ? q->agg.a : q->agg.b;
    p.sums = (unsigned long long*)sums;
    p.counts = (unsigned long long*)counts;
    hipStream_t s = (hipStream_t)stream;
    SDB_HIP(launch_zero_pair(p.sums, p.counts, plan->n_groups, s), "output fill");
    uint8_t* flags = (uint8_t*)scratch;
    uint32_t* gid = (uint32_t*)((uint8_t*)scratch + align_up((uint64_t)q->n_fact, 256));
    if (mode == SDB_BASELINE_PER_OPERATOR) SDB_HIP(launch_unfused(p, flags, gid, s), "per-operator launch");
    else SDB_HIP(launch_handoff(p, flags, gid, s), "global hand-off launch");
    return ok();
}

SDB_API sdb_status sdb_set_fused_events(void* start, void* stop) {
    if ((start == nullptr) != (stop == nullptr)) return fail(SDB_INVALID_ARG, "set both events or neither");
    g_fused_start = (hipEvent_t)start;
    g_fused_stop = (hipEvent_t)stop;
    return ok();
}

SDB_API sdb_status sdb_read_columns(const int32_t* const* cols, int32_t n_cols, int64_t n, int32_t blocks_per_cu,
                                    int64_t* sum, void* stream) {
    if (!cols || !sum) return fail(SDB_INVALID_ARG, "null argument");
    if (blocks_per_cu < 0 || blocks_per_cu > 4)
        return fail(SDB_INVALID_ARG, "blocks_per_cu %d is not in [0, 4]", (int)blocks_per_cu);
    if (n_cols < 0 || n_cols > SDB_MAX_FACT_COLS)
        return fail(SDB_INVALID_ARG, "n_cols %d is not in [0, %d]", (int)n_cols, SDB_MAX_FACT_COLS);
    if (n < 0) return fail(SDB_INVALID_ARG, "negative n");
    ReadParams p;
    std::memset(&p, 0, sizeof p);
    for (int c = 0; c < n_cols; ++c) {
        if (!cols[c] && n > 0) return fail(SDB_INVALID_ARG, "column %d is null", c);
        if (!aligned16(cols[c])) return fail(SDB_INVALID_ARG, "column %d is not 16-byte aligned", c);
        p.cols[c] = cols[c];
    }
    p.n_cols = n_cols;
    p.n = n;
    p.out = (unsigned long long*)sum;
    int dev = 0, cus = 0;
    SDB_HIP(hipGetDevice(&dev), "device query");
    SDB_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev), "device query");
    const int64_t tiles = (n / 4 + 1023) / 1024;
    const int per_cu = blocks_per_cu > 0 ? blocks_per_cu : 2;
    const int grid = (int)std::max<int64_t>(1, std::min<int64_t>(tiles, (int64_t)cus * per_cu));
    SDB_HIP(launch_read_columns(p, grid, (hipStream_t)stream), "read launch");
    return ok();
}

SDB_API sdb_status sdb_finalize_scratch_bytes(const sdb_plan* plan, int64_t* bytes) {
    if (!plan || !bytes) return fail(SDB_INVALID_ARG, "null argument");
    const uint64_t nb = (plan->n_groups + kFinGroupsPerBlock - 1) / kFinGroupsPerBlock;
    *bytes = (int64_t)std::max<uint64_t>(nb * 8, 256);
    return ok();
}

SDB_API sdb_status sdb_finalize_groups(const sdb_plan* plan, const int64_t* sums, const int64_t* counts,
                                       int32_t* out_keys, int64_t* out_sums, int64_t* out_counts,
                                       int64_t out_capacity, int64_t* out_n, void* scratch,
                                       int64_t scratch_bytes, void* stream) {
    if (!plan) return fail(SDB_INVALID_ARG, "null plan");
    if (!sums || !counts || !out_sums || !out_counts || !out_n || !scratch)
        return fail(SDB_INVALID_ARG, "null argument");
    if (plan->n_group_keys < 0 || plan->n_group_keys > SDB_MAX_GROUP_KEYS)
        return fail(SDB_INVALID_ARG, "bad plan key count");
    if (plan->n_group_keys > 0 && !out_keys) return fail(SDB_INVALID_ARG, "null key output");
    if (plan->n_groups == 0 || plan->n_groups > (uint64_t)INT32_MAX)
        return fail(SDB_INVALID_ARG, "bad plan group count");
    {
        // the last key varies fastest: stride[last] = 1, stride[k] = stride[k+1] * radix[k+1]
        uint64_t g = 1;
        for (int k = plan->n_group_keys - 1; k >= 0; --k) {
            if (plan->radix[k] == 0 || plan->stride[k] != g) return fail(SDB_INVALID_ARG, "bad plan group layout");
            g *= plan->radix[k];
        }
        if (g != plan->n_groups) return fail(SDB_INVALID_ARG, "bad plan group count");
    }
    if (out_capacity < 0 || (uint64_t)out_capacity < plan->n_groups)
        return fail(SDB_CAPACITY, "output holds %lld groups, plan needs %llu", (long long)out_capacity,
                    (unsigned long long)plan->n_groups);
    int64_t need = 0;
    sdb_finalize_scratch_bytes(plan, &need);
    if (scratch_bytes < need)
        return fail(SDB_WORKSPACE_TOO_SMALL, "finalize scratch holds %lld bytes, %lld needed",
                    (long long)scratch_bytes, (long long)need);
    FinalizeParams fp;
    std::memset(&fp, 0, sizeof fp);
    fp.sums = (const long long*)sums;
    fp.counts = (const long long*)counts;
    fp.n_groups = plan->n_groups;
    fp.n_keys = plan->n_group_keys;
    fp.scalar = plan->n_group_keys == 0;
    for (int k = 0; k < plan->n_group_keys; ++k) {
        fp.key_min[k] = plan->key_min[k];
        fp.radix[k] = plan->radix[k];
        fp.stride[k] = (uint32_t)plan->stride[k];
    }
    fp.out_keys = out_keys;
    fp.out_sums = (long long*)out_sums;
    fp.out_counts = (long long*)out_counts;
    fp.out_n = (long long*)out_n;
    fp.block_off = (long long*)scratch;
    fp.n_blocks = (int64_t)((plan->n_groups + kFinGroupsPerBlock - 1) / kFinGroupsPerBlock);
    SDB_HIP(launch_finalize(fp, (hipStream_t)stream), "finalize launch");
    return ok();
}

}  // extern "C"
