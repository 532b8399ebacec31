// The fused probe-filter-aggregate pass of libsdb (gfx950, wave64;
// Sections 3.2, 4.2 and 4.3 of the paper).
//
// A grid-stride persistent loop. A lane owns IPT items per iteration; an item
// is W consecutive fact rows (W = 4: one 128-bit load per column per item).
// Stages run in plan order; a stage loads its column only for items that still
// hold a live row, and the whole wave leaves the stage list as soon as no lane
// has a live row (wave-wide vote). Probes keep the group id in a register; the
// terminal is a register accumulator, an LDS group table, global 64-bit
// atomics, or records for the partitioned aggregation passes.
//
// The kernel template is instantiated in several translation units
// (sdb_fused_*.hip), each exporting a picker for its instances, so the
// instances compile in parallel.
#pragma once

#include "sdb_device.h"

namespace sdb {

// ---------------------------------------------------------------------------
// the fused probe-filter-aggregate pass
// ---------------------------------------------------------------------------

// Hardware register XCC_ID (register id 20, bits [3:0]): the XCD the wave runs
// on. Only used to pick a private group-table copy, so a wrong value would
// cost speed, never correctness (every copy is updated with device-scope
// atomics and all copies are added up afterwards).
__device__ __forceinline__ uint32_t xcc_id() {
    return __builtin_amdgcn_s_getreg((3 << 11) | 20) & 0xFu;
}

template <int TERM>
struct TermState {
    unsigned long long sum = 0;
    unsigned long long cnt = 0;
    unsigned long long* lsum = nullptr;   // LDS terminal
    unsigned long long* lcnt = nullptr;
    unsigned long long* xt = nullptr;     // global terminal: this XCD's interleaved copy, or null
    // partitioned terminal: survivors collect in a per-wave LDS ring and leave
    // in 64-record flushes to this block's region (full coalesced stores)
    uint32_t* lfill = nullptr;            // records this block claimed in its region
    uint32_t* lhist = nullptr;            // records per partition in the region
    // this wave's ring (kRing entries): with 64-bit values a group-id array
    // and a value array; with 32-bit values one 8-byte {group id, value} each
    uint32_t* ring_gid = nullptr;
    void* ring_val = nullptr;
    uint32_t head = 0;                    // ring index of the oldest pending record (wave-uniform)
    uint32_t pend = 0;                    // pending records (wave-uniform, < kRing)
    uint32_t* rgid = nullptr;             // this block's record region
    void* rval = nullptr;
};

constexpr uint32_t kRing = 128;   // per-wave ring entries: < 64 pending + one 64-lane step
static_assert(kRing == kRingEntries, "ring layout");

// Writes `cnt` (<= 64) pending ring records to the block's region, one per
// lane; records past the region's capacity go straight into the group table.
__device__ __forceinline__ void part_flush(const FusedParams& p, TermState<TERM_PART>& ts, uint32_t cnt) {
    __builtin_amdgcn_wave_barrier();
    const uint32_t lane = threadIdx.x & 63u;
    uint32_t base = 0;
    if (lane == 0) base = atomicAdd(ts.lfill, cnt);
    base = __shfl(base, 0, 64);
    if (lane < cnt) {
        const uint32_t slot = (ts.head + lane) & (kRing - 1u);
        uint32_t g;
        long long v;
        if (p.rec_wide) {
            g = ts.ring_gid[slot];
            v = static_cast<const long long*>(ts.ring_val)[slot];
        } else {
            const unsigned long long e = static_cast<const unsigned long long*>(ts.ring_val)[slot];
            g = (uint32_t)e;
            v = (long long)(int32_t)(uint32_t)(e >> 32);
        }
        const uint32_t pos = base + lane;
        if (pos < p.part_cap) {
            // non-temporal: the records are read back only by the scatter pass,
            // so they should not take L2 lines from the lookup tables
            // (measured: c5 13.85 -> 13.68 ms per run; the same hint on the
            // scatter passes' stores made them slower)
            __builtin_nontemporal_store(g, ts.rgid + pos);
            if (p.rec_wide) __builtin_nontemporal_store((long long)v, static_cast<long long*>(ts.rval) + pos);
            else __builtin_nontemporal_store((int32_t)v, static_cast<int32_t*>(ts.rval) + pos);
            atomicAdd(&ts.lhist[g >> p.part_shift], 1u);
        } else {
            atomicAdd(&p.sums[g], (unsigned long long)v);
            atomicAdd(&p.counts[g], 1ull);
        }
    }
    __builtin_amdgcn_wave_barrier();
    ts.head = (ts.head + cnt) & (kRing - 1u);
    ts.pend -= cnt;
}

template <int TERM>
__device__ __forceinline__ void accumulate(const FusedParams& p, TermState<TERM>& ts, uint32_t g,
                                           long long v) {
    if constexpr (TERM == TERM_SCALAR) {
        ts.sum += (unsigned long long)v;
        ts.cnt += 1ull;
    } else if constexpr (TERM == TERM_LDS) {
        atomicAdd(&ts.lsum[g], (unsigned long long)v);
        atomicAdd(&ts.lcnt[g], 1ull);
    } else {
        if (ts.xt) {   // sum and count of a group share a cache line
            atomicAdd(&ts.xt[2u * g], (unsigned long long)v);
            atomicAdd(&ts.xt[2u * g + 1u], 1ull);
        } else {
            atomicAdd(&p.sums[g], (unsigned long long)v);
            atomicAdd(&p.counts[g], 1ull);
        }
    }
}

template <int WB>
__device__ __forceinline__ uint32_t ld_code(const void* base, uint32_t idx) {
    if constexpr (WB == 1) return static_cast<const uint8_t*>(base)[idx];
    else if constexpr (WB == 2) return static_cast<const uint16_t*>(base)[idx];
    else return static_cast<const uint32_t*>(base)[idx];
}

// Row loops over the IPT items of W rows a lane owns. Liveness is one bool
// per row; rows that are no longer live still execute the (branch-free) code
// but read a fixed, valid slot so they cost no extra memory lines.
#define SDB_ROWS(j, r)                        \
    _Pragma("unroll") for (int j = 0; j < IPT; ++j) \
    _Pragma("unroll") for (int r = 0; r < W; ++r)

template <int W, int IPT>
__device__ __forceinline__ void load_column(const int32_t* col, const int64_t (&item)[IPT],
                                            const bool (&al)[IPT][W], int32_t (&x)[IPT][W]) {
#pragma unroll
    for (int j = 0; j < IPT; ++j) {
        bool any = false;
#pragma unroll
        for (int r = 0; r < W; ++r) any = any || al[j][r];
        // an item with no live row reads item 0, a line every such item shares
        load_item<W>(col, any ? item[j] : 0, x[j]);
    }
}

// A column for the current items: from its eager slot (loaded with the
// other eager columns when the items started; the slot number is
// wave-uniform) or loaded now, skipping items without a live row.
template <int W, int IPT, bool EG>
__device__ __forceinline__ void fetch_column(const FusedParams& p, int col, int slot, const int64_t (&item)[IPT],
                                             const bool (&al)[IPT][W], const int32_t (&eg)[kMaxEager][IPT][W],
                                             int32_t (&x)[IPT][W]) {
    if constexpr (EG) {
        if (slot >= 0) {
#pragma unroll
            for (int k = 0; k < kMaxEager; ++k)
                if (slot == k) {
                    SDB_ROWS(j, r) x[j][r] = eg[k][j][r];
                }
            return;
        }
    }
    load_column<W, IPT>(p.cols[col], item, al, x);
}

// Issues the loads of every eager column for the current items at once, so
// their latencies overlap instead of adding up stage after stage.
template <int W, int IPT>
__device__ __forceinline__ void load_eager(const FusedParams& p, const int64_t (&item)[IPT], const bool (&al)[IPT][W],
                                           int32_t (&eg)[kMaxEager][IPT][W]) {
#pragma unroll
    for (int k = 0; k < kMaxEager; ++k) {
        if (k < p.eg_n) load_column<W, IPT>(p.cols[p.eg_col[k]], item, al, eg[k]);
    }
}

template <int W, int IPT>
__device__ __forceinline__ void add_group(const StageDev& S, const uint32_t (&c)[IPT][W], uint32_t (&gid)[IPT][W]) {
    // dead rows may add garbage: their group id is never used
    if (S.gk_mode == GK_ONE) {
        SDB_ROWS(j, r) gid[j][r] += c[j][r] * S.gk_stride[0];
    } else if (S.gk_mode == GK_GENERAL) {
        SDB_ROWS(j, r) gid[j][r] += code_contribution(S, c[j][r]);
    }
}

// Dense map lookup (device memory or LDS): the code doubles as the filter.
template <int W, int IPT, int WB, bool IN_LDS>
__device__ __forceinline__ void stage_map(const StageDev& S, const unsigned char* lds, const int32_t (&x)[IPT][W],
                                          bool (&al)[IPT][W], uint32_t (&gid)[IPT][W]) {
    const void* base = IN_LDS ? static_cast<const void*>(lds + S.lds_off) : S.map;
    uint32_t c[IPT][W];
    SDB_ROWS(j, r) {
        const uint32_t idx = (uint32_t)(x[j][r] - S.kmin);
        const bool ok = al[j][r] && idx < S.nslots;
        c[j][r] = ld_code<WB>(base, ok ? idx : 0u);
        al[j][r] = ok;
    }
    SDB_ROWS(j, r) al[j][r] = al[j][r] && c[j][r] < S.sentinel;
    add_group<W, IPT>(S, c, gid);
}

template <int W, int IPT>
__device__ __forceinline__ void stage_bits(const StageDev& S, const unsigned char* lds, const int32_t (&x)[IPT][W],
                                           bool (&al)[IPT][W], uint32_t (&gid)[IPT][W], uint32_t (&didx)[IPT][W]) {
    const uint32_t* words = reinterpret_cast<const uint32_t*>(lds + S.lds_off);
    uint32_t idc[IPT][W];
    SDB_ROWS(j, r) {
        const uint32_t idx = (uint32_t)(x[j][r] - S.kmin);
        const bool ok = al[j][r] && idx < S.nslots;
        idc[j][r] = ok ? idx : 0u;
        al[j][r] = ok && ((words[idc[j][r] >> 5] >> (idc[j][r] & 31u)) & 1u);
    }
    if (S.defer == 0) {
        SDB_ROWS(j, r) didx[j][r] = idc[j][r];
    } else if (S.gk_mode != GK_NONE) {
        // gather the code now, from the device map, for the rows that passed
        uint32_t c[IPT][W];
        if (S.width == 1) {
            SDB_ROWS(j, r) c[j][r] = ld_code<1>(S.map, al[j][r] ? idc[j][r] : 0u);
        } else if (S.width == 2) {
            SDB_ROWS(j, r) c[j][r] = ld_code<2>(S.map, al[j][r] ? idc[j][r] : 0u);
        } else {
            SDB_ROWS(j, r) c[j][r] = ld_code<4>(S.map, al[j][r] ? idc[j][r] : 0u);
        }
        add_group<W, IPT>(S, c, gid);
    }
}

// Pass bitmap, ranks and passing codes in LDS: a passing key's code is the
// rank-th code (rank = passing slots before it).
template <int W, int IPT, int WB>
__device__ __forceinline__ void stage_rank(const StageDev& S, const unsigned char* lds, const int32_t (&x)[IPT][W],
                                           bool (&al)[IPT][W], uint32_t (&gid)[IPT][W]) {
    const uint32_t* words = reinterpret_cast<const uint32_t*>(lds + S.lds_off);
    const uint32_t* pre = reinterpret_cast<const uint32_t*>(lds + S.lds_rank_off);
    const void* codes = static_cast<const void*>(lds + S.lds_codes_off);
    uint32_t c[IPT][W];
    SDB_ROWS(j, r) {
        const uint32_t idx = (uint32_t)(x[j][r] - S.kmin);
        const bool ok = al[j][r] && idx < S.nslots;
        const uint32_t i = ok ? idx : 0u;
        const uint32_t w = words[i >> 5];
        const bool pass = ok && ((w >> (i & 31u)) & 1u);
        const uint32_t lower = (i & 32u) ? (uint32_t)__popc(words[(i >> 5) - 1u]) : 0u;
        const uint32_t rank = pre[i >> 6] + lower + (uint32_t)__popc(w & ((1u << (i & 31u)) - 1u));
        c[j][r] = ld_code<WB>(codes, pass ? rank : 0u);
        al[j][r] = pass;
    }
    add_group<W, IPT>(S, c, gid);
}

// Device map behind a coarse pass bitmap in LDS: a row whose coarse bit is
// clear dies without a device-memory gather.
template <int W, int IPT, int WB>
__device__ __forceinline__ void stage_coarse(const StageDev& S, const unsigned char* lds, const int32_t (&x)[IPT][W],
                                             bool (&al)[IPT][W], uint32_t (&gid)[IPT][W]) {
    const uint32_t* words = reinterpret_cast<const uint32_t*>(lds + S.lds_off);
    uint32_t c[IPT][W];
    SDB_ROWS(j, r) {
        const uint32_t idx = (uint32_t)(x[j][r] - S.kmin);
        bool ok = al[j][r] && idx < S.nslots;
        const uint32_t cb = (ok ? idx : 0u) >> S.coarse_shift;
        ok = ok && ((words[cb >> 5] >> (cb & 31u)) & 1u);
        c[j][r] = ld_code<WB>(S.map, ok ? idx : 0u);
        al[j][r] = ok;
    }
    SDB_ROWS(j, r) al[j][r] = al[j][r] && c[j][r] < S.sentinel;
    add_group<W, IPT>(S, c, gid);
}

// Pass bitmap of a window of the key range in LDS, the device map behind it:
// a row whose slot falls in the window and whose bit is clear dies without a
// device-memory gather; every other live row gathers its code (for a row in
// the window that passed, only for its group key). One gather instruction
// serves both; rows that do not gather read slot 0, a line every such lane
// shares.
template <int W, int IPT, int WB>
__device__ __forceinline__ void stage_window(const StageDev& S, const unsigned char* lds, const int32_t (&x)[IPT][W],
                                             bool (&al)[IPT][W], uint32_t (&gid)[IPT][W]) {
    const uint32_t* words = reinterpret_cast<const uint32_t*>(lds + S.lds_off);
    uint32_t c[IPT][W];
    SDB_ROWS(j, r) {
        const uint32_t idx = (uint32_t)(x[j][r] - S.kmin);
        const bool ok = al[j][r] && idx < S.nslots;
        const uint32_t w = idx - S.win_lo;
        const bool inw = w < S.win_slots;
        const uint32_t wi = inw ? w : 0u;
        const bool bit = ((words[wi >> 5] >> (wi & 31u)) & 1u) != 0u;
        const bool need = ok && (bit || !inw);
        c[j][r] = ld_code<WB>(S.map, need ? idx : 0u);
        al[j][r] = need;
    }
    SDB_ROWS(j, r) al[j][r] = al[j][r] && c[j][r] < S.sentinel;
    add_group<W, IPT>(S, c, gid);
}

// PAIR: the home slot and the next one come from one 16-byte load at 8-byte
// alignment (global loads on gfx950 need 4-byte alignment only): one memory
// request instead of two. Measured on c5, it pays when the slots are in L2,
// as with the sliced probe (13.67 -> 13.15 ms per run), and not when they
// come from HBM (16.13 -> 16.22 ms). The table's last slot, whose successor
// is slot 0, still takes two loads, so no load reaches past the table.
template <int W, int IPT, bool PAIR>
__device__ __forceinline__ void stage_hash(const StageDev& S, const int32_t (&x)[IPT][W], bool (&al)[IPT][W],
                                           uint32_t (&gid)[IPT][W]) {
    // open addressing: first slots of two items in flight, then resolve
    const unsigned long long* tab = static_cast<const unsigned long long*>(S.map);
    constexpr int HJ = IPT < 2 ? IPT : 2;
#pragma unroll
    for (int j0 = 0; j0 < IPT; j0 += HJ) {
        uint32_t h[HJ][W];
        unsigned long long sl[HJ][W], sn[HJ][W];
#pragma unroll
        for (int jj = 0; jj < HJ; ++jj)
#pragma unroll
            for (int r = 0; r < W; ++r) {
                h[jj][r] = hash_slot(S, x[j0 + jj][r]);
                sl[jj][r] = 0ull;
                sn[jj][r] = 0ull;
                if (al[j0 + jj][r]) {
                    // the home slot and the next one (mostly the same cache line)
                    if (PAIR && h[jj][r] != S.hmask) {
                        const u64x2 pr = *reinterpret_cast<const u64x2_a8*>(tab + h[jj][r]);
                        sl[jj][r] = pr.x;
                        sn[jj][r] = pr.y;
                    } else {
                        sl[jj][r] = tab[h[jj][r]];
                        sn[jj][r] = tab[(h[jj][r] + 1u) & S.hmask];
                    }
                }
            }
#pragma unroll
        for (int jj = 0; jj < HJ; ++jj)
#pragma unroll
            for (int r = 0; r < W; ++r) {
                uint32_t c = S.sentinel;
                if (al[j0 + jj][r]) {
                    const unsigned long long a = sl[jj][r];
                    const uint32_t ahi = (uint32_t)(a >> 32);
                    if (ahi == 0u) c = S.sentinel;
                    else if ((int32_t)(uint32_t)a == x[j0 + jj][r]) c = ahi - 1u;
                    else c = hash_resolve(S, x[j0 + jj][r], (h[jj][r] + 1u) & S.hmask, sn[jj][r]);
                }
                al[j0 + jj][r] = al[j0 + jj][r] && c < S.sentinel;
                if (S.gk_mode == GK_ONE) gid[j0 + jj][r] += c * S.gk_stride[0];
                else if (S.gk_mode == GK_GENERAL) gid[j0 + jj][r] += code_contribution(S, c);
            }
    }
}

// The deferred stage's codes for the rows still live (dead rows read slot 0,
// a line every such row shares).
template <int W, int IPT>
__device__ __forceinline__ void load_deferred(const StageDev& S, const bool (&al)[IPT][W],
                                              const uint32_t (&didx)[IPT][W], uint32_t (&c)[IPT][W]) {
    if (S.width == 1) {
        SDB_ROWS(j, r) c[j][r] = ld_code<1>(S.map, al[j][r] ? didx[j][r] : 0u);
    } else if (S.width == 2) {
        SDB_ROWS(j, r) c[j][r] = ld_code<2>(S.map, al[j][r] ? didx[j][r] : 0u);
    } else {
        SDB_ROWS(j, r) c[j][r] = ld_code<4>(S.map, al[j][r] ? didx[j][r] : 0u);
    }
}

template <int W, int IPT>
__device__ __forceinline__ bool wave_has_live(const bool (&al)[IPT][W]) {
    bool any = false;
    SDB_ROWS(j, r) any = any || al[j][r];
    return __any(any) != 0;
}

// One stage of the plan for the current items: fetch its column, then apply
// its predicate or lookup.
template <int W, int IPT, bool EG>
__device__ __forceinline__ void run_stage(const FusedParams& p, const unsigned char* lds, const StageDev& S,
                                          const int64_t (&item)[IPT], bool (&al)[IPT][W], uint32_t (&gid)[IPT][W],
                                          uint32_t (&didx)[IPT][W], const int32_t (&eg)[kMaxEager][IPT][W]) {
    int32_t x[IPT][W];
    fetch_column<W, IPT, EG>(p, S.col, S.eg_slot, item, al, eg, x);
    switch (S.op) {
        case OP_PRED:
            SDB_ROWS(j, r) al[j][r] = al[j][r] && range_pass(S.test, x[j][r]);
            break;
        case OP_LDS_BITS: stage_bits<W, IPT>(S, lds, x, al, gid, didx); break;
        case OP_LDS_MAP1: stage_map<W, IPT, 1, true>(S, lds, x, al, gid); break;
        case OP_LDS_MAP2: stage_map<W, IPT, 2, true>(S, lds, x, al, gid); break;
        case OP_LDS_MAP4: stage_map<W, IPT, 4, true>(S, lds, x, al, gid); break;
        case OP_MAP1: stage_map<W, IPT, 1, false>(S, lds, x, al, gid); break;
        case OP_MAP2: stage_map<W, IPT, 2, false>(S, lds, x, al, gid); break;
        case OP_MAP4: stage_map<W, IPT, 4, false>(S, lds, x, al, gid); break;
        case OP_HASH: stage_hash<W, IPT, false>(S, x, al, gid); break;
        case OP_HASH_PAIR: stage_hash<W, IPT, true>(S, x, al, gid); break;
        case OP_LDS_RANK1: stage_rank<W, IPT, 1>(S, lds, x, al, gid); break;
        case OP_LDS_RANK2: stage_rank<W, IPT, 2>(S, lds, x, al, gid); break;
        case OP_LDS_RANK4: stage_rank<W, IPT, 4>(S, lds, x, al, gid); break;
        case OP_COARSE1: stage_coarse<W, IPT, 1>(S, lds, x, al, gid); break;
        case OP_COARSE2: stage_coarse<W, IPT, 2>(S, lds, x, al, gid); break;
        case OP_COARSE4: stage_coarse<W, IPT, 4>(S, lds, x, al, gid); break;
        case OP_WINDOW1: stage_window<W, IPT, 1>(S, lds, x, al, gid); break;
        case OP_WINDOW2: stage_window<W, IPT, 2>(S, lds, x, al, gid); break;
        case OP_WINDOW4: stage_window<W, IPT, 4>(S, lds, x, al, gid); break;
        default:   // OP_NEVER
            SDB_ROWS(j, r) al[j][r] = false;
            break;
    }
}

// Runs every stage and the terminal for IPT items of W rows each. All lanes
// of the wave must call this together (the early exit is a wave-wide vote).
template <int W, int IPT, int TERM, bool EG, int UNR = 0>
__device__ __forceinline__ void process_items(const FusedParams& p, const unsigned char* lds,
                                              const int64_t (&item)[IPT], bool (&al)[IPT][W],
                                              TermState<TERM>& ts) {
    uint32_t gid[IPT][W];
    uint32_t didx[IPT][W];   // deferred gather: slot in the deferred stage's map
    SDB_ROWS(j, r) {
        gid[j][r] = 0u;
        didx[j][r] = 0u;
    }
    int32_t eg[kMaxEager][IPT][W];
    if constexpr (EG) load_eager<W, IPT>(p, item, al, eg);

    if constexpr (UNR > 0) {
        // the stage loop written out UNR times: each copy's stage parameters
        // stay in scalar registers across tiles instead of being reloaded
#pragma unroll
        for (int s = 0; s < UNR; ++s) {
            if (s >= p.nstages) break;
            if (!wave_has_live<W, IPT>(al)) return;
            run_stage<W, IPT, EG>(p, lds, p.st[s], item, al, gid, didx, eg);
        }
    } else {
        for (int s = 0; s < p.nstages; ++s) {
            if (!wave_has_live<W, IPT>(al)) return;
            run_stage<W, IPT, EG>(p, lds, p.st[s], item, al, gid, didx, eg);
        }
    }
    if (!wave_has_live<W, IPT>(al)) return;
    // deferred codes and the aggregate column are loaded together, used after
    uint32_t dc[IPT][W];
    if (p.defer_stage >= 0) load_deferred<W, IPT>(p.st[p.defer_stage], al, didx, dc);

    int32_t a[IPT][W], b[IPT][W];
    fetch_column<W, IPT, EG>(p, p.agg_a, p.agg_a_slot, item, al, eg, a);
    if (p.defer_stage >= 0) add_group<W, IPT>(p.st[p.defer_stage], dc, gid);
    long long v[IPT][W];
    switch (p.agg_kind) {
        case SDB_AGG_COL:
            SDB_ROWS(j, r) v[j][r] = a[j][r];
            break;
        case SDB_AGG_MUL:
            fetch_column<W, IPT, EG>(p, p.agg_b, p.agg_b_slot, item, al, eg, b);
            SDB_ROWS(j, r) v[j][r] = (long long)a[j][r] * (long long)b[j][r];
            break;
        case SDB_AGG_SUB:
            fetch_column<W, IPT, EG>(p, p.agg_b, p.agg_b_slot, item, al, eg, b);
            SDB_ROWS(j, r) v[j][r] = (long long)a[j][r] - (long long)b[j][r];
            break;
        default:
            fetch_column<W, IPT, EG>(p, p.agg_b, p.agg_b_slot, item, al, eg, b);
            SDB_ROWS(j, r) v[j][r] = (long long)a[j][r] + (long long)b[j][r];
            break;
    }
    if constexpr (TERM == TERM_SCALAR) {
        SDB_ROWS(j, r) {
            ts.sum += al[j][r] ? (unsigned long long)v[j][r] : 0ull;
            ts.cnt += al[j][r] ? 1ull : 0ull;
        }
    } else if constexpr (TERM == TERM_PART) {
        // append the wave's survivors to its ring; flush every full 64
        const uint32_t lane = threadIdx.x & 63u;
        const unsigned long long below = (1ull << lane) - 1ull;
        SDB_ROWS(j, r) {
            const unsigned long long m = __ballot(al[j][r]);
            if (al[j][r]) {
                const uint32_t slot = (ts.head + ts.pend + (uint32_t)__popcll(m & below)) & (kRing - 1u);
                if (p.rec_wide) {
                    ts.ring_gid[slot] = gid[j][r];
                    static_cast<long long*>(ts.ring_val)[slot] = v[j][r];
                } else {
                    static_cast<unsigned long long*>(ts.ring_val)[slot] =
                        ((unsigned long long)(uint32_t)(int32_t)v[j][r] << 32) | gid[j][r];
                }
            }
            ts.pend += (uint32_t)__popcll(m);
            if (ts.pend >= 64u) part_flush(p, ts, 64u);
        }
    } else {
        SDB_ROWS(j, r) if (al[j][r]) accumulate<TERM>(p, ts, gid[j][r], v[j][r]);
    }
}

// The kernel reads its parameters in place from the kernel-argument segment
// (constant memory, scalar loads); indexing the by-value copy with a runtime
// stage number could otherwise make the compiler copy it to scratch.
template <int W, int IPT, int TERM, bool EG, int LB, int UNR = 0>
__global__ void __launch_bounds__(LB) star_fused_kernel(FusedParams kernel_args) {
    (void)kernel_args;
    const FusedParams& p = *(const FusedParams*)__builtin_amdgcn_kernarg_segment_ptr();
    extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
    TermState<TERM> ts;
    if constexpr (TERM == TERM_LDS) {
        ts.lsum = reinterpret_cast<unsigned long long*>(lds);
        ts.lcnt = ts.lsum + p.n_groups;
        for (uint32_t g = threadIdx.x; g < 2u * p.n_groups; g += blockDim.x) ts.lsum[g] = 0ull;
    }
    if constexpr (TERM == TERM_GLOBAL) {
        if (p.xcd_copies > 0)
            ts.xt = p.xtab + 2ull * p.n_groups * (xcc_id() & (uint32_t)(p.xcd_copies - 1));
    }
    if constexpr (TERM == TERM_PART) {
        // the block's part_subs fill counters, then a histogram each
        uint32_t* fills = reinterpret_cast<uint32_t*>(lds);
        for (uint32_t i = threadIdx.x; i < p.part_subs * (1u + p.n_parts); i += blockDim.x) fills[i] = 0u;
        // rings: every wave's 8-byte entries (values, or {group id, value}),
        // then (64-bit values) every wave's group ids
        const uint32_t wave = threadIdx.x >> 6;
        const uint32_t sub = wave % p.part_subs;
        ts.lfill = fills + sub;
        ts.lhist = fills + p.part_subs + sub * p.n_parts;
        const uint32_t vbytes = p.rec_wide ? 8u : 4u;
        ts.ring_val = lds + p.ring_off + (size_t)wave * kRing * 8u;
        ts.ring_gid = reinterpret_cast<uint32_t*>(lds + p.ring_off + (blockDim.x >> 6) * kRing * 8u) +
                      (size_t)wave * kRing;
        // launches of a segmented plan start at region_base
        const uint64_t region = ((uint64_t)p.region_base + blockIdx.x) * p.part_subs + sub;
        ts.rgid = p.rec_gid + region * p.part_cap;
        ts.rval = static_cast<unsigned char*>(p.rec_val) + region * p.part_cap * vbytes;
    }
    // stage the LDS-resident dimension tables (16-byte copies; sources are padded)
    for (int s = 0; s < p.nstages; ++s) {
        const StageDev& S = p.st[s];
        if (S.lds_mode == LDS_GLOBAL) continue;
        const v4i* src = reinterpret_cast<const v4i*>(S.lds_mode == LDS_MAP ? S.map : S.bits);
        v4i* dst = reinterpret_cast<v4i*>(lds + S.lds_off);
        for (uint32_t i = threadIdx.x; i < S.lds_bytes / 16u; i += blockDim.x) dst[i] = src[i];
        if (S.lds_mode == LDS_RANK) {
            const v4i* rsrc = reinterpret_cast<const v4i*>(S.rank);
            v4i* rdst = reinterpret_cast<v4i*>(lds + S.lds_rank_off);
            for (uint32_t i = threadIdx.x; i < S.lds_rank_bytes / 16u; i += blockDim.x) rdst[i] = rsrc[i];
            const v4i* csrc = reinterpret_cast<const v4i*>(S.codes);
            v4i* cdst = reinterpret_cast<v4i*>(lds + S.lds_codes_off);
            for (uint32_t i = threadIdx.x; i < S.lds_codes_bytes / 16u; i += blockDim.x) cdst[i] = csrc[i];
        }
    }
    __syncthreads();

    int64_t n_rows = p.n;
    if (p.n_dev) n_rows = min(n_rows, (int64_t)*p.n_dev);
    const int64_t n_items = n_rows / W;
    const int64_t tile = (int64_t)blockDim.x * IPT;
    const int64_t n_tiles = (n_items + tile - 1) / tile;
    const int64_t n_loop = p.tile_map ? p.n_vtiles : n_tiles;
    for (int64_t t = blockIdx.x; t < n_loop; t += gridDim.x) {
        int64_t tt = t;
        if (p.tile_map) {   // the sliced probe's XCD-aware tile order
            tt = p.tile_map[t];
            if (tt < 0) continue;
        }
        int64_t item[IPT];
        bool al[IPT][W];
#pragma unroll
        for (int j = 0; j < IPT; ++j) {
            item[j] = tt * tile + (int64_t)j * blockDim.x + threadIdx.x;
#pragma unroll
            for (int r = 0; r < W; ++r) al[j][r] = item[j] < n_items;
        }
        process_items<W, IPT, TERM, EG, UNR>(p, lds, item, al, ts);
    }
    if constexpr (W > 1) {
        // the last n mod W rows, one per lane, by the last block
        if (blockIdx.x == gridDim.x - 1) {
            int64_t row[1] = {n_items * W + (int64_t)threadIdx.x};
            bool al1[1][1] = {{row[0] < n_rows}};
            process_items<1, 1, TERM, false>(p, lds, row, al1, ts);
        }
    }

    if constexpr (TERM == TERM_SCALAR) {
        __shared__ unsigned long long red[2][LB / 64];
        const unsigned long long s = wave_sum_u64(ts.sum);
        const unsigned long long c = wave_sum_u64(ts.cnt);
        if ((threadIdx.x & 63) == 0) {
            red[0][threadIdx.x >> 6] = s;
            red[1][threadIdx.x >> 6] = c;
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            unsigned long long bs = 0, bc = 0;
            for (uint32_t w = 0; w < blockDim.x / 64u; ++w) {
                bs += red[0][w];
                bc += red[1][w];
            }
            if (bc) {
                atomicAdd(&p.sums[0], bs);
                atomicAdd(&p.counts[0], bc);
            }
        }
    } else if constexpr (TERM == TERM_LDS) {
        __syncthreads();
        for (uint32_t g = threadIdx.x; g < p.n_groups; g += blockDim.x) {
            const unsigned long long c = ts.lcnt[g];
            if (c) {
                atomicAdd(&p.sums[g], ts.lsum[g]);
                atomicAdd(&p.counts[g], c);
            }
        }
    } else if constexpr (TERM == TERM_PART) {
        if (ts.pend) part_flush(p, ts, ts.pend);
        __syncthreads();
        const uint32_t* fills = reinterpret_cast<const uint32_t*>(lds);
        const uint32_t region0 = (p.region_base + blockIdx.x) * p.part_subs;
        if (threadIdx.x < p.part_subs) p.region_count[region0 + threadIdx.x] = min(fills[threadIdx.x], p.part_cap);
        // this block's columns of the partition x region histogram
        for (uint32_t i = threadIdx.x; i < p.part_subs * p.n_parts; i += blockDim.x) {
            const uint32_t sub = i / p.n_parts, q = i - sub * p.n_parts;
            p.part_hist[(uint64_t)q * p.n_regions + region0 + sub] = fills[p.part_subs + i];
        }
    }
}

template <int W, int IPT, int TERM, bool EG, int LB = kMaxBlock, int UNR = 0>
const void* fused_fn() {
    return reinterpret_cast<const void*>(&star_fused_kernel<W, IPT, TERM, EG, LB, UNR>);
}

// The instance of every terminal for one item shape (inside a picker that
// takes `terminal`).
#define SDB_FUSED_TERMINALS(Wv, I, EGv, LBv, UNRv)                                         \
    if (terminal == TERM_SCALAR) return fused_fn<Wv, I, TERM_SCALAR, EGv, LBv, UNRv>();  \
    if (terminal == TERM_LDS) return fused_fn<Wv, I, TERM_LDS, EGv, LBv, UNRv>();        \
    if (terminal == TERM_GLOBAL) return fused_fn<Wv, I, TERM_GLOBAL, EGv, LBv, UNRv>();  \
    if (terminal == TERM_PART) return fused_fn<Wv, I, TERM_PART, EGv, LBv, UNRv>();

// Pickers of the instance files (nullptr for a shape they do not hold):
// the stage loop written out kUnrollStages times, 4-row items, ipt 2, no
// eager loads, blocks of kMaxBlock ...
const void* pick_fused_unrolled(int terminal);
// ... or of kBigBlock threads;
const void* pick_fused_unrolled_big(int terminal);
// 4-row items, ipt 1, 2 or 4, launch bound kMaxBlock;
const void* pick_fused_vec(int ipt, int terminal);
// 4-row items, ipt 1 or 2, blocks of kBigBlock;
const void* pick_fused_big(int ipt, int terminal);
// 4-row items with eager column loads, ipt 1 or 2, launch bound kMaxBlock;
const void* pick_fused_eager(int ipt, int terminal);
// 1-row items, ipt 1, 2 or 4, launch bound kMaxBlock.
const void* pick_fused_rows(int ipt, int terminal);

}  // namespace sdb
