// Device kernels of libsdb for CDNA4 (gfx950, wave64), except the fused pass
// itself (sdb_fused.h, instantiated in sdb_fused_*.hip):
//
//  * dimension build: statistics pass, direct-mapped packed map scatter, and
//    open-addressing insert with 64-bit compare-and-swap (Section 3.3);
//  * plan sampling: each stage evaluated on its own over a strided fact sample;
//  * the fused pass's launch, the per-XCD copies' merge, the partitioned
//    terminal's passes and the sliced hash probe's partition passes;
//  * the kernel-at-a-time baselines, the streaming-read reference and
//    group-table compaction.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <climits>
#include <mutex>

#include "sdb_fused.h"

namespace sdb {
// ---------------------------------------------------------------------------
// fills
// ---------------------------------------------------------------------------

__global__ void fill_u32_kernel(uint32_t* p, uint64_t n, uint32_t v) {
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = v;
}

__global__ void fill_u64_kernel(unsigned long long* p, uint64_t n) {
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = 0ull;
}

__global__ void zero_pair_kernel(unsigned long long* a, unsigned long long* b, uint64_t n) {
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
        a[i] = 0ull;
        b[i] = 0ull;
    }
}

static int fill_grid(uint64_t n) {
    uint64_t g = (n + 255) / 256;
    if (g > 4096) g = 4096;
    if (g < 1) g = 1;
    return (int)g;
}

hipError_t launch_fill_u32(uint32_t* p, uint64_t n_words, uint32_t value, hipStream_t s) {
    if (n_words == 0) return hipSuccess;
    hipLaunchKernelGGL(fill_u32_kernel, dim3(fill_grid(n_words)), dim3(256), 0, s, p, n_words, value);
    return hipGetLastError();
}

hipError_t launch_fill_u64(unsigned long long* p, uint64_t n, hipStream_t s) {
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(fill_u64_kernel, dim3(fill_grid(n)), dim3(256), 0, s, p, n);
    return hipGetLastError();
}

hipError_t launch_zero_pair(unsigned long long* a, unsigned long long* b, uint64_t n, hipStream_t s) {
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(zero_pair_kernel, dim3(fill_grid(n)), dim3(256), 0, s, a, b, n);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// dimension build
// ---------------------------------------------------------------------------

__device__ __forceinline__ bool dim_row_passes(const BuildParams& bp, int64_t i) {
    bool pass = true;
    for (int q = 0; q < bp.n_preds; ++q) pass = pass && range_pass(bp.pred[q], bp.cols[bp.pred_col[q]][i]);
    return pass;
}

// The build kernels read their table's parameters in place from the batch in
// the kernel-argument segment (table = blockIdx.y).
#define SDB_BATCH_TABLE                                                                     \
    (void)kernel_args;                                                                      \
    const BuildBatch& bb = *(const BuildBatch*)__builtin_amdgcn_kernarg_segment_ptr();      \
    const BuildParams& bp = bb.bp[blockIdx.y];                                              \
    (void)bb

// Key range over all rows; pass count and payload ranges over passing rows.
// Block b of a table's stats_blocks reduces its rows in registers and LDS and
// writes its partial statistics to stats_part[b]; stats_reduce_kernel then
// combines the partials (no atomics, however many blocks).
__global__ void __launch_bounds__(256) dim_stats_kernel(BuildBatch kernel_args) {
    SDB_BATCH_TABLE;
    if ((int)blockIdx.x >= bp.stats_blocks) return;
    constexpr int kWaves = 256 / 64;
    __shared__ int32_t s_kmin[kWaves], s_kmax[kWaves], s_pkmin[kWaves], s_pkmax[kWaves];
    __shared__ unsigned long long s_np[kWaves];
    __shared__ int32_t s_pmin[SDB_MAX_PAYLOADS][kWaves], s_pmax[SDB_MAX_PAYLOADS][kWaves];
    int32_t kmin = INT_MAX, kmax = INT_MIN, pkmin = INT_MAX, pkmax = INT_MIN;
    unsigned long long npass = 0;
    int32_t pmin[SDB_MAX_PAYLOADS], pmax[SDB_MAX_PAYLOADS];
    for (int p = 0; p < SDB_MAX_PAYLOADS; ++p) {
        pmin[p] = INT_MAX;
        pmax[p] = INT_MIN;
    }
    // kBuildRows rows per thread per step, each column's loads issued together
    constexpr int U = kBuildRows;
    const int64_t stride = (int64_t)bp.stats_blocks * blockDim.x * U;
    for (int64_t i0 = (int64_t)blockIdx.x * blockDim.x * U + threadIdx.x; i0 < bp.n; i0 += stride) {
        bool ok[U], pass[U];
        int32_t x[U], key[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t i = i0 + (int64_t)u * blockDim.x;
            ok[u] = i < bp.n;
            key[u] = ok[u] ? bp.key[i] : 0;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (ok[u]) {
                kmin = min(kmin, key[u]);
                kmax = max(kmax, key[u]);
            }
            pass[u] = ok[u];
        }
        for (int q = 0; q < bp.n_preds; ++q) {
            const int32_t* col = bp.cols[bp.pred_col[q]];
#pragma unroll
            for (int u = 0; u < U; ++u) x[u] = ok[u] ? col[i0 + (int64_t)u * blockDim.x] : 0;
#pragma unroll
            for (int u = 0; u < U; ++u) pass[u] = pass[u] && range_pass(bp.pred[q], x[u]);
        }
        for (int p = 0; p < bp.n_payloads; ++p) {
            const int32_t* col = bp.cols[bp.payload_col[p]];
#pragma unroll
            for (int u = 0; u < U; ++u) x[u] = pass[u] ? col[i0 + (int64_t)u * blockDim.x] : 0;
#pragma unroll
            for (int u = 0; u < U; ++u)
                if (pass[u]) {
                    pmin[p] = min(pmin[p], x[u]);
                    pmax[p] = max(pmax[p], x[u]);
                }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            npass += pass[u] ? 1ull : 0ull;
            if (pass[u]) {
                pkmin = min(pkmin, key[u]);
                pkmax = max(pkmax, key[u]);
            }
        }
    }
    kmin = wave_min_i32(kmin);
    kmax = wave_max_i32(kmax);
    pkmin = wave_min_i32(pkmin);
    pkmax = wave_max_i32(pkmax);
    npass = wave_sum_u64(npass);
    for (int p = 0; p < SDB_MAX_PAYLOADS; ++p) {
        pmin[p] = wave_min_i32(pmin[p]);
        pmax[p] = wave_max_i32(pmax[p]);
    }
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
        s_kmin[wave] = kmin;
        s_kmax[wave] = kmax;
        s_pkmin[wave] = pkmin;
        s_pkmax[wave] = pkmax;
        s_np[wave] = npass;
        for (int p = 0; p < SDB_MAX_PAYLOADS; ++p) {
            s_pmin[p][wave] = pmin[p];
            s_pmax[p][wave] = pmax[p];
        }
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < kWaves; ++w) {
            kmin = min(kmin, s_kmin[w]);
            kmax = max(kmax, s_kmax[w]);
            pkmin = min(pkmin, s_pkmin[w]);
            pkmax = max(pkmax, s_pkmax[w]);
            npass += s_np[w];
            for (int p = 0; p < SDB_MAX_PAYLOADS; ++p) {
                pmin[p] = min(pmin[p], s_pmin[p][w]);
                pmax[p] = max(pmax[p], s_pmax[p][w]);
            }
        }
        DimStats part;
        part.kmin = kmin;
        part.kmax = kmax;
        part.npass = npass;
        for (int p = 0; p < SDB_MAX_PAYLOADS; ++p) {
            part.pmin[p] = pmin[p];
            part.pmax[p] = pmax[p];
        }
        part.dup = 0u;
        part.pad_ = 0u;
        part.occupied = 0ull;
        part.pkmin = pkmin;
        part.pkmax = pkmax;
        bp.stats_part[blockIdx.x] = part;
    }
}

// One block per table: the table's statistics from its blocks' partials
// (and the duplicate and occupancy counters the build passes add to, zeroed).
__global__ void __launch_bounds__(256) stats_reduce_kernel(BuildBatch kernel_args) {
    SDB_BATCH_TABLE;
    __shared__ DimStats red[256 / 64];
    DimStats acc;
    acc.kmin = INT_MAX;
    acc.kmax = INT_MIN;
    acc.npass = 0ull;
    for (int p = 0; p < SDB_MAX_PAYLOADS; ++p) {
        acc.pmin[p] = INT_MAX;
        acc.pmax[p] = INT_MIN;
    }
    acc.dup = 0u;
    acc.pad_ = 0u;
    acc.occupied = 0ull;
    acc.pkmin = INT_MAX;
    acc.pkmax = INT_MIN;
    // up to kStatsMaxBlocks / 256 partials per thread, loaded together
    constexpr int kPer = kStatsMaxBlocks / 256;
    static_assert(kPer * 256 == kStatsMaxBlocks, "whole partials per thread");
    DimStats part[kPer];
    bool have[kPer];
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
        const int b = (int)threadIdx.x + u * 256;
        have[u] = b < bp.stats_blocks;
        if (have[u]) part[u] = bp.stats_part[b];
    }
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
        if (!have[u]) continue;
        const DimStats& s = part[u];
        acc.kmin = min(acc.kmin, s.kmin);
        acc.kmax = max(acc.kmax, s.kmax);
        acc.npass += s.npass;
        acc.pkmin = min(acc.pkmin, s.pkmin);
        acc.pkmax = max(acc.pkmax, s.pkmax);
        for (int p = 0; p < SDB_MAX_PAYLOADS; ++p) {
            acc.pmin[p] = min(acc.pmin[p], s.pmin[p]);
            acc.pmax[p] = max(acc.pmax[p], s.pmax[p]);
        }
    }
    // wave reductions, then the 4 waves' results in LDS
    acc.kmin = wave_min_i32(acc.kmin);
    acc.kmax = wave_max_i32(acc.kmax);
    acc.npass = wave_sum_u64(acc.npass);
    acc.pkmin = wave_min_i32(acc.pkmin);
    acc.pkmax = wave_max_i32(acc.pkmax);
    for (int p = 0; p < SDB_MAX_PAYLOADS; ++p) {
        acc.pmin[p] = wave_min_i32(acc.pmin[p]);
        acc.pmax[p] = wave_max_i32(acc.pmax[p]);
    }
    if ((threadIdx.x & 63u) == 0u) red[threadIdx.x >> 6] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        DimStats a = red[0];
        for (uint32_t w = 1; w < blockDim.x / 64u; ++w) {
            const DimStats& s = red[w];
            a.kmin = min(a.kmin, s.kmin);
            a.kmax = max(a.kmax, s.kmax);
            a.npass += s.npass;
            a.pkmin = min(a.pkmin, s.pkmin);
            a.pkmax = max(a.pkmax, s.pkmax);
            for (int p = 0; p < SDB_MAX_PAYLOADS; ++p) {
                a.pmin[p] = min(a.pmin[p], s.pmin[p]);
                a.pmax[p] = max(a.pmax[p], s.pmax[p]);
            }
        }
        *bp.stats = a;
        if (bb.host_stats) bb.host_stats[blockIdx.y] = a;
    }
}

// One block: every table's statistics block, word by word, to pinned host memory.
__global__ void __launch_bounds__(256) export_stats_kernel(BuildBatch kernel_args) {
    (void)kernel_args;
    const BuildBatch& bb = *(const BuildBatch*)__builtin_amdgcn_kernarg_segment_ptr();
    constexpr int kWords = sizeof(DimStats) / 4;
    for (int i = threadIdx.x; i < bb.n * kWords; i += blockDim.x) {
        const uint32_t* src = reinterpret_cast<const uint32_t*>(bb.bp[i / kWords].stats);
        reinterpret_cast<uint32_t*>(bb.host_stats + i / kWords)[i % kWords] = src[i % kWords];
    }
}

__global__ void __launch_bounds__(256) copy_out_kernel(const uint32_t* src0, uint32_t words0, const uint32_t* src1,
                                                       uint32_t words1, uint32_t* dst) {
    const uint32_t stride = gridDim.x * blockDim.x;
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < words0 + words1; i += stride)
        dst[i] = i < words0 ? src0[i] : src1[i - words0];
}

__device__ __forceinline__ uint32_t dim_row_code(const BuildParams& bp, int64_t i) {
    uint32_t c = 0;
    for (int p = 0; p < bp.n_payloads; ++p)
        c += (uint32_t)(bp.cols[bp.payload_col[p]][i] - bp.pmin[p]) * bp.pdiv[p];
    return c;
}

// Direct-mapped map over the keys [kmin, kmin + nslots): the fill leaves
// every slot at `missing` (all ones: no row holds the key); a passing row then
// stores its code and a filtered row the sentinel (`missing` - 1). Plain
// stores, no atomics: each key owns its slot.
__global__ void __launch_bounds__(256) fill_table_kernel(BuildBatch kernel_args) {
    SDB_BATCH_TABLE;
    uint32_t* w = static_cast<uint32_t*>(bp.map);
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < bp.fill_words; i += stride)
        w[i] = bp.fill_value;
}

__global__ void __launch_bounds__(256) dense_scatter_kernel(BuildBatch kernel_args) {
    SDB_BATCH_TABLE;
    if (!bp.dense) return;
    // kBuildRows rows per thread per step, each column's loads issued together
    // (a row at a time, the key, predicate and payload loads form one chain)
    constexpr int U = kBuildRows;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x * U;
    for (int64_t i0 = (int64_t)blockIdx.x * blockDim.x * U + threadIdx.x; i0 < bp.n; i0 += stride) {
        bool ok[U], pass[U];
        int32_t x[U];
        uint32_t idx[U], code[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t i = i0 + (int64_t)u * blockDim.x;
            ok[u] = i < bp.n;
            x[u] = ok[u] ? bp.key[i] : 0;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            idx[u] = (uint32_t)((int64_t)x[u] - (int64_t)bp.kmin);
            pass[u] = ok[u];
            code[u] = 0u;
        }
        for (int q = 0; q < bp.n_preds; ++q) {
            const int32_t* col = bp.cols[bp.pred_col[q]];
#pragma unroll
            for (int u = 0; u < U; ++u) x[u] = ok[u] ? col[i0 + (int64_t)u * blockDim.x] : 0;
#pragma unroll
            for (int u = 0; u < U; ++u) pass[u] = pass[u] && range_pass(bp.pred[q], x[u]);
        }
        for (int p = 0; p < bp.n_payloads; ++p) {
            const int32_t* col = bp.cols[bp.payload_col[p]];
#pragma unroll
            for (int u = 0; u < U; ++u) x[u] = pass[u] ? col[i0 + (int64_t)u * blockDim.x] : 0;
#pragma unroll
            for (int u = 0; u < U; ++u) code[u] += (uint32_t)((int64_t)x[u] - (int64_t)bp.pmin[p]) * bp.pdiv[p];
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (!ok[u]) continue;
            if ((uint64_t)idx[u] >= bp.nslots) {          // cannot happen: kmin/kmax cover all keys
                atomicOr(&bp.stats->dup, 4u);
                continue;
            }
            const uint32_t c = pass[u] ? code[u] : bp.sentinel;
            if (bp.width == 1) static_cast<uint8_t*>(bp.map)[idx[u]] = (uint8_t)c;
            else if (bp.width == 2) static_cast<uint16_t*>(bp.map)[idx[u]] = (uint16_t)c;
            else static_cast<uint32_t*>(bp.map)[idx[u]] = c;
        }
    }
}

// One thread per 32 slots: the pass bitmap word (code below the sentinel)
// and the number of occupied slots. Distinct keys occupy n slots; a duplicate
// key leaves fewer, which the host detects from the total.
__global__ void __launch_bounds__(256) dense_bits_kernel(BuildBatch kernel_args) {
    SDB_BATCH_TABLE;
    if (!bp.dense) return;
    const uint64_t n_words = (bp.nslots + 31) / 32;
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    unsigned long long occupied = 0;
    for (uint64_t w = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; w < n_words; w += stride) {
        // the word's 32 map entries as 16-byte loads (the map is padded to 256
        // bytes and filled, so the last word's loads stay inside it)
        uint32_t bits = 0u;
        const uint32_t valid = (uint32_t)min<uint64_t>(32, bp.nslots - w * 32);
        if (bp.width == 1) {
            const v4u* src = reinterpret_cast<const v4u*>(static_cast<const uint8_t*>(bp.map) + w * 32);
            const v4u a = src[0], b = src[1];
            const uint32_t d[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
            for (uint32_t e = 0; e < 32u; ++e) {
                const uint32_t c = (d[e >> 2] >> ((e & 3u) * 8u)) & 0xFFu;
                if (e < valid) {
                    bits |= (c < bp.sentinel ? 1u : 0u) << e;
                    occupied += c != bp.missing;
                }
            }
        } else if (bp.width == 2) {
            const v4u* src = reinterpret_cast<const v4u*>(static_cast<const uint16_t*>(bp.map) + w * 32);
            uint32_t d[16];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const v4u a = src[k];
                d[4 * k] = a.x;
                d[4 * k + 1] = a.y;
                d[4 * k + 2] = a.z;
                d[4 * k + 3] = a.w;
            }
#pragma unroll
            for (uint32_t e = 0; e < 32u; ++e) {
                const uint32_t c = (d[e >> 1] >> ((e & 1u) * 16u)) & 0xFFFFu;
                if (e < valid) {
                    bits |= (c < bp.sentinel ? 1u : 0u) << e;
                    occupied += c != bp.missing;
                }
            }
        } else {
            const v4u* src = reinterpret_cast<const v4u*>(static_cast<const uint32_t*>(bp.map) + w * 32);
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const v4u a = src[k];
                const uint32_t d[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
                for (uint32_t e4 = 0; e4 < 4u; ++e4) {
                    const uint32_t e = (uint32_t)k * 4u + e4;
                    if (e < valid) {
                        bits |= (d[e4] < bp.sentinel ? 1u : 0u) << e;
                        occupied += d[e4] != bp.missing;
                    }
                }
            }
        }
        bp.pass_bits[w] = bits;
    }
    occupied = wave_sum_u64(occupied);
    __shared__ unsigned long long s_occ[4];
    if ((threadIdx.x & 63) == 0) s_occ[threadIdx.x >> 6] = occupied;
    __syncthreads();
    if (threadIdx.x == 0) {
        const unsigned long long t = s_occ[0] + s_occ[1] + s_occ[2] + s_occ[3];
        if (t) atomicAdd(&bp.stats->occupied, t);
    }
}

// Pass filter of a hash table's keys. SDB_FILTER_BITMAP: bit k - key_min of
// the key range. SDB_FILTER_BLOOM: three bits of one 32-bit word, the word
// and the bits from two mixes of the key (a blocked Bloom filter: one word
// read per test).
// The key mix is MurmurHash3's 32-bit finalizer.
__device__ __forceinline__ uint32_t filter_mix(int32_t k) {
    uint32_t m = (uint32_t)k;
    m = (m ^ (m >> 16)) * 0x85EBCA6Bu;
    m ^= m >> 13;
    m *= 0xC2B2AE35u;
    return m ^ (m >> 16);
}

// Word index and bit mask of key k in a filter of `nbits` bits; false when a
// bitmap's key range does not hold k.
__device__ __forceinline__ bool filter_slot(int32_t kind, uint64_t nbits, int32_t kmin, int32_t k, uint32_t& word,
                                            uint32_t& mask) {
    if (kind == SDB_FILTER_BITMAP) {
        const uint32_t idx = (uint32_t)k - (uint32_t)kmin;
        word = idx >> 5;
        mask = 1u << (idx & 31u);
        return (uint64_t)idx < nbits;
    }
    const uint32_t m = filter_mix(k);
    const uint32_t t = ((m << 16) | (m >> 16)) * 0x9E3779B1u;
    word = m & (uint32_t)((nbits >> 5) - 1u);
    mask = (1u << (t >> 27)) | (1u << ((t >> 22) & 31u)) | (1u << ((t >> 17) & 31u));
    return true;
}

// Open addressing, linear probing, 8-byte slots {key, code + 1 | 0xFFFFFFFF};
// a passing row's key also goes into the table's pass filter.
__global__ void __launch_bounds__(256) hash_insert_kernel(BuildBatch kernel_args) {
    SDB_BATCH_TABLE;
    if (bp.dense) return;
    unsigned long long* tab = static_cast<unsigned long long*>(bp.map);
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < bp.n; i += stride) {
        const int32_t k = bp.key[i];
        const uint32_t enc = dim_row_passes(bp, i) ? dim_row_code(bp, i) + 1u : 0xFFFFFFFFu;
        const unsigned long long slot = ((unsigned long long)enc << 32) | (uint32_t)k;
        uint32_t fw, fm;
        if (bp.filt && !bp.filt_via_bytes && enc != 0xFFFFFFFFu &&
            filter_slot(bp.filt_kind, bp.filt_bits, bp.kmin, k, fw, fm))
            atomicOr(&bp.filt[fw], fm);
        uint32_t h = ((uint32_t)k * 0x9E3779B1u) >> bp.hshift & bp.hmask;
        bool placed = false;
        for (uint64_t it = 0; it < bp.nslots; ++it) {
            const unsigned long long old = atomicCAS(&tab[h], 0ull, slot);
            if (old == 0ull) {
                placed = true;
                break;
            }
            if ((int32_t)(uint32_t)old == k) {
                atomicOr(&bp.stats->dup, 1u);
                placed = true;
                break;
            }
            h = (h + 1u) & bp.hmask;
        }
        if (!placed) atomicOr(&bp.stats->dup, 2u);
    }
}

// A hash table's pass bitmap without atomics (filt_via_bytes): the slot
// region, not yet filled, first holds one byte per key of the range, cleared,
// then set by every passing row with a plain store; the bytes are then
// packed 32 to a filter word. Each key has its own byte, so no two rows
// write the same address unless they hold the same key (a duplicate, which
// the inserts report).
__global__ void __launch_bounds__(256) filter_clear_kernel(BuildBatch kernel_args) {
    SDB_BATCH_TABLE;
    if (!bp.filt_via_bytes) return;
    uint32_t* w = static_cast<uint32_t*>(bp.map);
    const uint64_t n_words = (bp.filt_bits + 31u) / 32u * 8u;   // the bytes the packing reads
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_words; i += stride) w[i] = 0u;
}

__global__ void __launch_bounds__(256) filter_mark_kernel(BuildBatch kernel_args) {
    SDB_BATCH_TABLE;
    if (!bp.filt_via_bytes) return;
    uint8_t* b = static_cast<uint8_t*>(bp.map);
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < bp.n; i += stride) {
        const uint32_t idx = (uint32_t)bp.key[i] - (uint32_t)bp.kmin;
        if ((uint64_t)idx < bp.filt_bits && dim_row_passes(bp, i)) b[idx] = 1u;
    }
}

__global__ void __launch_bounds__(256) filter_pack_kernel(BuildBatch kernel_args) {
    SDB_BATCH_TABLE;
    if (!bp.filt_via_bytes) return;
    const v4u* b = static_cast<const v4u*>(bp.map);
    const uint64_t n_words = (bp.filt_bits + 31u) / 32u;
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t w = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; w < n_words; w += stride) {
        const v4u lo = b[2 * w], hi = b[2 * w + 1];   // the 32 key bytes of word w
        const uint32_t q[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
        uint32_t out = 0u;
#pragma unroll
        for (int j = 0; j < 8; ++j)
#pragma unroll
            for (int t = 0; t < 4; ++t)
                if ((q[j] >> (8 * t)) & 0xFFu) out |= 1u << (4 * j + t);
        if (32u * w + 32u > bp.filt_bits) out &= (1u << (uint32_t)(bp.filt_bits - 32u * w)) - 1u;   // past the range
        bp.filt[w] = out;
    }
}

static int build_grid(int64_t n) {
    int64_t g = (n + 255) / 256;
    if (g > 2048) g = 2048;
    if (g < 1) g = 1;
    return (int)g;
}

hipError_t launch_build_stats(const BuildBatch& bb, hipStream_t s) {
    if (bb.n <= 0) return hipSuccess;
    int g = 1;
    for (int d = 0; d < bb.n; ++d) {
        if (bb.bp[d].stats_blocks < 1 || bb.bp[d].stats_blocks > kStatsMaxBlocks) return hipErrorInvalidValue;
        g = std::max(g, bb.bp[d].stats_blocks);
    }
    hipLaunchKernelGGL(dim_stats_kernel, dim3(g, bb.n), dim3(256), 0, s, bb);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(stats_reduce_kernel, dim3(1, bb.n), dim3(256), 0, s, bb);
    return hipGetLastError();
}

hipError_t launch_export_stats(const BuildBatch& bb, hipStream_t s) {
    if (bb.n <= 0) return hipSuccess;
    if (!bb.host_stats || bb.n > SDB_MAX_JOINS) return hipErrorInvalidValue;
    hipLaunchKernelGGL(export_stats_kernel, dim3(1), dim3(256), 0, s, bb);
    return hipGetLastError();
}

hipError_t launch_copy_out(const uint32_t* src0, uint32_t words0, const uint32_t* src1, uint32_t words1,
                           uint32_t* dst, hipStream_t s) {
    const uint64_t total = (uint64_t)words0 + words1;
    if (total == 0) return hipSuccess;
    if (!dst || (words0 && !src0) || (words1 && !src1) || total > (1ull << 30)) return hipErrorInvalidValue;
    uint64_t g = (total + 255) / 256;
    if (g > 64) g = 64;
    hipLaunchKernelGGL(copy_out_kernel, dim3((uint32_t)g), dim3(256), 0, s, src0, words0, src1, words1, dst);
    return hipGetLastError();
}

hipError_t launch_build_tables(const BuildBatch& bb, hipStream_t s) {
    if (bb.n <= 0) return hipSuccess;
    uint64_t words = 0, n_words32 = 0, filt_words = 0;
    int64_t n_dense = 0, n_hash = 0, n_filt = 0;
    for (int d = 0; d < bb.n; ++d) {
        const BuildParams& bp = bb.bp[d];
        words = std::max<uint64_t>(words, bp.fill_words);
        if (bp.dense) {
            n_dense = std::max<int64_t>(n_dense, bp.n);
            n_words32 = std::max<uint64_t>(n_words32, (bp.nslots + 31) / 32);
        } else {
            n_hash = std::max<int64_t>(n_hash, bp.n);
        }
        if (bp.filt_via_bytes) {
            n_filt = std::max<int64_t>(n_filt, bp.n);
            filt_words = std::max<uint64_t>(filt_words, (bp.filt_bits + 31) / 32);
        }
    }
    if (filt_words > 0) {   // before the fill: the bytes live in the slot region
        hipLaunchKernelGGL(filter_clear_kernel, dim3(fill_grid(filt_words * 8), bb.n), dim3(256), 0, s, bb);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        if (n_filt > 0) {
            hipLaunchKernelGGL(filter_mark_kernel, dim3(build_grid(n_filt), bb.n), dim3(256), 0, s, bb);
            e = hipGetLastError();
            if (e != hipSuccess) return e;
        }
        hipLaunchKernelGGL(filter_pack_kernel, dim3(fill_grid(filt_words), bb.n), dim3(256), 0, s, bb);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (words > 0) {
        hipLaunchKernelGGL(fill_table_kernel, dim3(fill_grid(words), bb.n), dim3(256), 0, s, bb);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (n_dense > 0) {
        hipLaunchKernelGGL(dense_scatter_kernel, dim3(build_grid((n_dense + kBuildRows - 1) / kBuildRows), bb.n),
                           dim3(256), 0, s, bb);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (n_words32 > 0) {
        hipLaunchKernelGGL(dense_bits_kernel, dim3(build_grid((int64_t)n_words32), bb.n), dim3(256), 0, s, bb);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (n_hash > 0) {
        hipLaunchKernelGGL(hash_insert_kernel, dim3(build_grid(n_hash), bb.n), dim3(256), 0, s, bb);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

// ---------------------------------------------------------------------------
// coarse pass bitmap of a dense table (LDS_COARSE placement)
// ---------------------------------------------------------------------------

// Thread w writes coarse word w: bit b is set iff one of the 2^shift slots
// starting at slot (32 w + b) << shift passes. 2^shift divides 32, so every
// group of slots lies inside one word of the pass bitmap.
__global__ void __launch_bounds__(256) coarse_bits_kernel(CoarseParams cp) {
    const uint32_t w = blockIdx.x * blockDim.x + threadIdx.x;
    if (w >= cp.n_words) return;
    const uint32_t per = 1u << cp.shift;
    const uint32_t mask = per >= 32u ? 0xFFFFFFFFu : ((1u << per) - 1u);
    const uint32_t n_fine = (cp.nslots + 31u) / 32u;
    uint32_t out = 0u;
    for (uint32_t b = 0; b < 32u; ++b) {
        const uint64_t first = ((uint64_t)w * 32u + b) << cp.shift;
        if (first >= cp.nslots) break;
        const uint32_t fw = (uint32_t)(first >> 5);
        const uint32_t word = fw < n_fine ? cp.bits[fw] : 0u;
        if ((word >> (uint32_t)(first & 31u)) & mask) out |= 1u << b;
    }
    cp.out[w] = out;
}

hipError_t launch_coarse_build(const CoarseParams& cp, hipStream_t s) {
    if (cp.n_words == 0) return hipSuccess;
    hipLaunchKernelGGL(coarse_bits_kernel, dim3((cp.n_words + 255u) / 256u), dim3(256), 0, s, cp);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// rank tables of a dense table (LDS_RANK placement)
// ---------------------------------------------------------------------------

__device__ __forceinline__ uint32_t rank_word(const RankParams& rp, uint32_t w) {
    return w < (rp.nslots + 31u) / 32u ? rp.bits[w] : 0u;
}

// One block of 1024 threads: prefix[g] = passing slots in 64-slot groups
// before g (exclusive scan of the groups' popcounts).
__global__ void __launch_bounds__(1024) rank_prefix_kernel(RankParams rp) {
    __shared__ uint32_t wsum[16];
    const uint32_t n64 = (rp.nslots + 63u) / 64u;
    constexpr uint32_t kPer = kRankGroups / 1024;
    const uint32_t g0 = threadIdx.x * kPer;
    uint32_t c[kPer];
    uint32_t loc = 0;
#pragma unroll
    for (uint32_t k = 0; k < kPer; ++k) {
        const uint32_t g = g0 + k;
        c[k] = g < n64 ? (uint32_t)(__popc(rank_word(rp, 2 * g)) + __popc(rank_word(rp, 2 * g + 1))) : 0u;
        loc += c[k];
    }
    const uint32_t lane = threadIdx.x & 63u, wave = threadIdx.x >> 6;
    uint32_t x = loc;
    for (uint32_t off = 1; off < 64u; off <<= 1) {
        const uint32_t y = __shfl_up(x, off, 64);
        if (lane >= off) x += y;
    }
    if (lane == 63u) wsum[wave] = x;
    __syncthreads();
    uint32_t run = x - loc;
    for (uint32_t w = 0; w < wave; ++w) run += wsum[w];
#pragma unroll
    for (uint32_t k = 0; k < kPer; ++k) {
        const uint32_t g = g0 + k;
        if (g < n64) rp.prefix[g] = run;
        run += c[k];
    }
}

// One thread per bitmap word: the word's passing slots store their codes at
// their ranks.
__global__ void __launch_bounds__(256) rank_codes_kernel(RankParams rp) {
    const uint32_t n_words = (rp.nslots + 31u) / 32u;
    const uint32_t w = blockIdx.x * blockDim.x + threadIdx.x;
    if (w >= n_words) return;
    uint32_t bits = rp.bits[w];
    uint32_t r = rp.prefix[w >> 1] + ((w & 1u) ? (uint32_t)__popc(rp.bits[w - 1]) : 0u);
    while (bits) {
        const uint32_t b = (uint32_t)__ffs(bits) - 1u;
        bits &= bits - 1u;
        const uint32_t slot = w * 32u + b;
        if (rp.width == 1) static_cast<uint8_t*>(rp.codes)[r] = static_cast<const uint8_t*>(rp.map)[slot];
        else if (rp.width == 2) static_cast<uint16_t*>(rp.codes)[r] = static_cast<const uint16_t*>(rp.map)[slot];
        else static_cast<uint32_t*>(rp.codes)[r] = static_cast<const uint32_t*>(rp.map)[slot];
        ++r;
    }
}

hipError_t launch_rank_build(const RankParams& rp, hipStream_t s) {
    if (rp.nslots == 0) return hipSuccess;
    if ((rp.nslots + 63u) / 64u > kRankGroups) return hipErrorInvalidValue;
    hipLaunchKernelGGL(rank_prefix_kernel, dim3(1), dim3(1024), 0, s, rp);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const uint32_t n_words = (rp.nslots + 31u) / 32u;
    hipLaunchKernelGGL(rank_codes_kernel, dim3((n_words + 255u) / 256u), dim3(256), 0, s, rp);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// plan sampling: pass count of every stage on its own over a strided sample
// ---------------------------------------------------------------------------

// Every sampled row (row k * step) is evaluated against every stage on its
// own; the pattern of stages it passes (bit s for stage s) is counted in
// pattern_hist, and for a dense-table stage the bucket of its key in the
// table's key range (kKeyBuckets equal buckets) in key_hist[s].
__global__ void __launch_bounds__(256) sample_kernel(FusedParams kernel_args, int64_t step, int64_t n_sample,
                                                     int32_t n_ranges, uint32_t* pattern_hist, uint32_t* key_hist) {
    (void)kernel_args;
    const FusedParams& p = *(const FusedParams*)__builtin_amdgcn_kernarg_segment_ptr();
    // block-private histograms in LDS (the few pass patterns of a small plan
    // would otherwise draw every sampled row's atomic onto a handful of words)
    __shared__ uint32_t kh[kMaxStages * kKeyBuckets];
    __shared__ uint32_t ph[kSamplePatternsLds];
    const uint32_t n_patterns = (uint32_t)n_ranges << p.nstages;
    const bool lds_patterns = n_patterns <= (uint32_t)kSamplePatternsLds;
    for (int i = threadIdx.x; i < p.nstages * kKeyBuckets; i += blockDim.x) kh[i] = 0u;
    for (uint32_t i = threadIdx.x; lds_patterns && i < n_patterns; i += blockDim.x) ph[i] = 0u;
    __syncthreads();
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < n_sample; k += stride) {
        const int64_t row = k * step;
        uint32_t pattern = 0u;
        for (int s = 0; s < p.nstages; ++s) {
            const StageDev& S = p.st[s];
            const int32_t x = p.cols[S.col][row];
            if (stage_pass_one(S, x)) pattern |= 1u << s;
            if (S.sample_hist && S.kind == ST_DENSE && S.nslots > 0u) {
                const uint32_t idx = (uint32_t)(x - S.kmin);
                if (idx < S.nslots)
                    atomicAdd(&kh[s * kKeyBuckets + (uint32_t)((uint64_t)idx * kKeyBuckets / S.nslots)], 1u);
            }
        }
        const uint32_t bin = (uint32_t)(k * n_ranges / n_sample) << p.nstages | pattern;
        if (lds_patterns) atomicAdd(&ph[bin], 1u);
        else atomicAdd(&pattern_hist[bin], 1u);
    }
    __syncthreads();
    for (int i = threadIdx.x; i < p.nstages * kKeyBuckets; i += blockDim.x)
        if (kh[i]) atomicAdd(&key_hist[i], kh[i]);
    for (uint32_t i = threadIdx.x; lds_patterns && i < n_patterns; i += blockDim.x)
        if (ph[i]) atomicAdd(&pattern_hist[i], ph[i]);
}

hipError_t launch_sample(const FusedParams& p, int64_t step, int64_t n_sample, int32_t n_ranges,
                         uint32_t* pattern_hist, uint32_t* key_hist, hipStream_t s) {
    if (p.nstages < 0 || p.nstages > kMaxStages || n_ranges < 1 || ((uint64_t)n_ranges << p.nstages) > (1ull << kMaxStages))
        return hipErrorInvalidValue;
    hipError_t e;
    if (key_hist == pattern_hist + (1u << kMaxStages)) {
        e = launch_fill_u32(pattern_hist, (1u << kMaxStages) + (uint64_t)kMaxStages * kKeyBuckets, 0u, s);
    } else {
        e = launch_fill_u32(pattern_hist, (uint64_t)n_ranges << p.nstages, 0u, s);
        if (e != hipSuccess) return e;
        e = launch_fill_u32(key_hist, (uint64_t)kMaxStages * kKeyBuckets, 0u, s);
    }
    if (e != hipSuccess || n_sample == 0 || p.nstages == 0) return e;
    int64_t g = (n_sample + 255) / 256;
    if (g > 256) g = 256;
    hipLaunchKernelGGL(sample_kernel, dim3((int)g), dim3(256), 0, s, p, step, n_sample, n_ranges, pattern_hist,
                       key_hist);
    return hipGetLastError();
}

// Adds the per-XCD copies into the outputs (which it overwrites).
__global__ void __launch_bounds__(256) xcd_merge_kernel(const unsigned long long* xtab, int copies,
                                                        uint64_t n_groups, unsigned long long* sums,
                                                        unsigned long long* counts) {
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t g = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; g < n_groups; g += stride) {
        unsigned long long s = 0, c = 0;
        for (int x = 0; x < copies; ++x) {
            const unsigned long long* e = xtab + 2ull * (n_groups * (uint64_t)x + g);
            s += e[0];
            c += e[1];
        }
        sums[g] = s;
        counts[g] = c;
    }
}

hipError_t launch_xcd_merge(const unsigned long long* xtab, int copies, uint64_t n_groups,
                            unsigned long long* sums, unsigned long long* counts, hipStream_t s) {
    if (n_groups == 0) return hipSuccess;
    hipLaunchKernelGGL(xcd_merge_kernel, dim3(fill_grid(n_groups)), dim3(256), 0, s, xtab, copies, n_groups,
                       sums, counts);
    return hipGetLastError();
}


// Instances: 4-row or 1-row items, 1/2/4 items per lane, every terminal;
// eager column loads for 4-row items with 1 or 2 items per lane; blocks of
// kBigBlock threads for 4-row items with 1 or 2 items per lane; the stage
// loop written out kUnrollStages times for 4-row items, 2 items per lane,
// blocks of kMaxBlock or kBigBlock and no eager loads.
static const void* pick_fused(int vector, int ipt, int terminal, int eager, int block, int unroll) {
    if (unroll) {
        if (!vector || ipt != 2 || eager > 0) return nullptr;
        if (block == kMaxBlock) return pick_fused_unrolled(terminal);
        if (block == kBigBlock) return pick_fused_unrolled_big(terminal);
        return nullptr;
    }
    if (block == kBigBlock) return vector && eager <= 0 ? pick_fused_big(ipt, terminal) : nullptr;
    if (block > kMaxBlock) return nullptr;
    if (eager > 0) return vector ? pick_fused_eager(ipt, terminal) : nullptr;
    return vector ? pick_fused_vec(ipt, terminal) : pick_fused_rows(ipt, terminal);
}

int fused_blocks_per_cu(int vector, int ipt, int terminal, int eager, int block, int unroll, size_t lds_bytes) {
    const void* fn = pick_fused(vector, ipt, terminal, eager, block, unroll);
    if (!fn) return -1;
    int blocks = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, fn, block, lds_bytes) != hipSuccess)
        return -1;
    return blocks;
}

hipError_t launch_fused(const FusedParams& p, int vector, int ipt, int terminal, int eager, int unroll, int grid,
                        int block, size_t lds_bytes, hipStream_t s) {
    if (unroll && p.nstages > kUnrollStages) return hipErrorInvalidValue;
    const void* fn = pick_fused(vector, ipt, terminal, eager, block, unroll);
    if (!fn) return hipErrorInvalidValue;
    void* args[] = {const_cast<FusedParams*>(&p)};
    return hipLaunchKernel(fn, dim3(grid), dim3(block), args, lds_bytes, s);
}


// ---------------------------------------------------------------------------
// kernel-at-a-time execution: one kernel per operator, flags and group ids in
// global memory between them (the unfused baseline)
// ---------------------------------------------------------------------------

struct UnfusedParams {
    const int32_t* col;        // the stage's fact column (stage kernels), agg operand a (aggregate kernel)
    const int32_t* col_b;      // agg operand b
    int64_t n;
    uint8_t* flags;            // live flag per row
    uint32_t* gid;             // group id per row
    unsigned long long* sums;
    unsigned long long* counts;
    int32_t agg_kind;
    int32_t pad_;
    StageDev st;
};

__global__ void __launch_bounds__(256) unfused_init_kernel(UnfusedParams up) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < up.n; i += stride) {
        up.flags[i] = 1u;
        up.gid[i] = 0u;
    }
}

// One row of one stage with its table in device memory: whether the row
// passes, and the dimension code it gathers (pass implies c < sentinel).
__device__ __forceinline__ bool device_stage_row(const StageDev& S, int32_t x, uint32_t& c) {
    c = 0u;
    if (S.kind == ST_PRED) return range_pass(S.test, x);
    if (S.kind == ST_DENSE) {
        const uint32_t idx = (uint32_t)(x - S.kmin);
        if (idx >= S.nslots) return false;
        c = load_dense_code(S, idx);
        return c < S.sentinel;
    }
    const uint32_t h = hash_slot(S, x);
    c = hash_resolve(S, x, h, static_cast<const unsigned long long*>(S.map)[h]);
    return c < S.sentinel;
}

// The part of the mixed-radix group id that a passing row's code adds.
__device__ __forceinline__ uint32_t stage_gid_part(const StageDev& S, uint32_t c) {
    if (S.gk_mode == GK_ONE) return c * S.gk_stride[0];
    if (S.gk_mode == GK_GENERAL) return code_contribution(S, c);
    return 0u;
}

__device__ __forceinline__ long long row_value(int32_t kind, int32_t a, int32_t b) {
    const long long x = a;
    if (kind == SDB_AGG_MUL) return x * (long long)b;
    if (kind == SDB_AGG_SUB) return x - (long long)b;
    if (kind == SDB_AGG_ADD) return x + (long long)b;
    return x;
}

// One stage over every row still flagged: predicate, dense map or hash probe.
__global__ void __launch_bounds__(256) unfused_stage_kernel(UnfusedParams kernel_args) {
    (void)kernel_args;
    const UnfusedParams& up = *(const UnfusedParams*)__builtin_amdgcn_kernarg_segment_ptr();
    const StageDev& S = up.st;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < up.n; i += stride) {
        if (!up.flags[i]) continue;
        uint32_t c;
        if (!device_stage_row(S, up.col[i], c)) up.flags[i] = 0u;
        else if (S.gk_mode != GK_NONE) up.gid[i] += stage_gid_part(S, c);
    }
}

// The aggregate of every flagged row, added into the outputs with atomics.
__global__ void __launch_bounds__(256) unfused_agg_kernel(UnfusedParams up) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < up.n; i += stride) {
        if (!up.flags[i]) continue;
        const long long v = row_value(up.agg_kind, up.col[i], up.col_b[i]);
        const uint32_t g = up.gid[i];
        atomicAdd(&up.sums[g], (unsigned long long)v);
        atomicAdd(&up.counts[g], 1ull);
    }
}

static int unfused_grid(int64_t n) {
    int64_t g = (n + 255) / 256;
    if (g > 8192) g = 8192;
    if (g < 1) g = 1;
    return (int)g;
}

hipError_t launch_unfused(const FusedParams& p, uint8_t* flags, uint32_t* gid, hipStream_t s) {
    if (p.n == 0) return hipSuccess;
    UnfusedParams up;
    memset(&up, 0, sizeof up);
    up.n = p.n;
    up.flags = flags;
    up.gid = gid;
    up.sums = p.sums;
    up.counts = p.counts;
    up.agg_kind = p.agg_kind;
    const int grid = unfused_grid(p.n);
    hipLaunchKernelGGL(unfused_init_kernel, dim3(grid), dim3(256), 0, s, up);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    for (int st = 0; st < p.nstages; ++st) {
        up.st = p.st[st];
        up.col = p.cols[up.st.col];
        hipLaunchKernelGGL(unfused_stage_kernel, dim3(grid), dim3(256), 0, s, up);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    up.col = p.cols[p.agg_a];
    up.col_b = p.cols[p.agg_b];
    hipLaunchKernelGGL(unfused_agg_kernel, dim3(grid), dim3(256), 0, s, up);
    return hipGetLastError();
}

struct HandoffParams {
    uint8_t* flags;
    uint32_t* gid;
    FusedParams p;
};
static_assert(sizeof(HandoffParams) <= 4096, "kernel arguments must fit the 4 KB kernarg segment");

// The whole query in one kernel, one row per thread, but with every hand-off
// between operators a store to and a later load from the per-row flag and
// group-id arrays in global memory (volatile, so none is kept in registers).
__global__ void __launch_bounds__(256) handoff_kernel(HandoffParams kernel_args) {
    (void)kernel_args;
    const HandoffParams& hp = *(const HandoffParams*)__builtin_amdgcn_kernarg_segment_ptr();
    const FusedParams& p = hp.p;
    volatile uint8_t* flags = hp.flags;
    volatile uint32_t* gid = hp.gid;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < p.n; i += stride) {
        flags[i] = 1u;
        gid[i] = 0u;
        for (int st = 0; st < p.nstages; ++st) {
            if (!flags[i]) break;
            const StageDev& S = p.st[st];
            uint32_t c;
            if (!device_stage_row(S, p.cols[S.col][i], c)) flags[i] = 0u;
            else if (S.gk_mode != GK_NONE) gid[i] = gid[i] + stage_gid_part(S, c);
        }
        if (!flags[i]) continue;
        const long long v = row_value(p.agg_kind, p.cols[p.agg_a][i], p.cols[p.agg_b][i]);
        const uint32_t g = gid[i];
        atomicAdd(&p.sums[g], (unsigned long long)v);
        atomicAdd(&p.counts[g], 1ull);
    }
}

hipError_t launch_handoff(const FusedParams& p, uint8_t* flags, uint32_t* gid, hipStream_t s) {
    if (p.n == 0) return hipSuccess;
    HandoffParams hp;
    memset(&hp, 0, sizeof hp);
    hp.flags = flags;
    hp.gid = gid;
    hp.p = p;
    hipLaunchKernelGGL(handoff_kernel, dim3(unfused_grid(p.n)), dim3(256), 0, s, hp);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// streaming read of fact columns: the bandwidth the fused pass is compared with
// ---------------------------------------------------------------------------

// Adds every int32 of n_cols columns of n rows into *out (mod 2^64), reading
// the columns four at a time with 128-bit non-temporal loads, two 4-row
// items per lane: the fused kernel's load shape without any of its work.
__global__ void __launch_bounds__(512) read_columns_kernel(ReadParams kernel_args) {
    (void)kernel_args;
    const ReadParams& p = *(const ReadParams*)__builtin_amdgcn_kernarg_segment_ptr();
    const int64_t n_items = p.n / 4;
    const int64_t tile = (int64_t)blockDim.x * 2;
    unsigned long long acc = 0;
    for (int64_t base = (int64_t)blockIdx.x * tile; base < n_items; base += (int64_t)gridDim.x * tile) {
        for (int c0 = 0; c0 < p.n_cols; c0 += 4) {
            v4i x[4][2];
#pragma unroll
            for (int k = 0; k < 4; ++k)
#pragma unroll
                for (int j = 0; j < 2; ++j) {
                    const int64_t it = base + (int64_t)j * blockDim.x + threadIdx.x;
                    x[k][j] = v4i{0, 0, 0, 0};
                    if (c0 + k < p.n_cols && it < n_items)
                        x[k][j] = __builtin_nontemporal_load(reinterpret_cast<const v4i*>(p.cols[c0 + k]) + it);
                }
#pragma unroll
            for (int k = 0; k < 4; ++k)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc += (unsigned long long)((long long)x[k][j].x + x[k][j].y + x[k][j].z + x[k][j].w);
        }
    }
    if (blockIdx.x == 0) {   // the last n mod 4 rows
        const int64_t r = n_items * 4 + (int64_t)threadIdx.x;
        if (r < p.n)
            for (int c = 0; c < p.n_cols; ++c) acc += (unsigned long long)(long long)p.cols[c][r];
    }
    acc = wave_sum_u64(acc);
    if ((threadIdx.x & 63u) == 0u) atomicAdd(p.out, acc);
}

hipError_t launch_read_columns(const ReadParams& p, int grid, hipStream_t s) {
    hipError_t e = launch_fill_u64(p.out, 1, s);
    if (e != hipSuccess || p.n == 0 || p.n_cols == 0) return e;
    hipLaunchKernelGGL(read_columns_kernel, dim3(grid), dim3(512), 0, s, p);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// partitioned aggregation: scan, scatter by partition, LDS aggregation
// ---------------------------------------------------------------------------

// One block: exclusive scan of the partition counts into part_start, and of
// the per-partition work items into chunk_start.
__global__ void __launch_bounds__(1024) part_scan_kernel(PartParams pp) {
    __shared__ uint32_t buf_r[1024], buf_c[1024];
    __shared__ uint32_t carry_r, carry_c;
    if (threadIdx.x == 0) {
        carry_r = 0u;
        carry_c = 0u;
    }
    __syncthreads();
    for (uint32_t base = 0; base < pp.n_parts; base += 1024u) {
        const uint32_t i = base + threadIdx.x;
        const uint32_t vr = i < pp.n_parts ? pp.part_count[i] : 0u;
        const uint32_t vc = (vr + (uint32_t)kPartChunk - 1u) / (uint32_t)kPartChunk;
        buf_r[threadIdx.x] = vr;
        buf_c[threadIdx.x] = vc;
        __syncthreads();
        for (uint32_t off = 1; off < 1024u; off <<= 1) {
            const uint32_t ar = threadIdx.x >= off ? buf_r[threadIdx.x - off] : 0u;
            const uint32_t ac = threadIdx.x >= off ? buf_c[threadIdx.x - off] : 0u;
            __syncthreads();
            buf_r[threadIdx.x] += ar;
            buf_c[threadIdx.x] += ac;
            __syncthreads();
        }
        if (i < pp.n_parts) {
            pp.part_start[i] = carry_r + buf_r[threadIdx.x] - vr;
            pp.chunk_start[i] = carry_c + buf_c[threadIdx.x] - vc;
        }
        __syncthreads();
        if (threadIdx.x == 1023) {
            carry_r += buf_r[1023];
            carry_c += buf_c[1023];
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        pp.part_start[pp.n_parts] = carry_r;
        pp.chunk_start[pp.n_parts] = carry_c;
    }
}

// Exclusive scan of n values by a 256-thread block: out[i] = carry + sum of
// in[0..i). in and out may be the same array (each thread reads its own run
// before writing it). Every thread must call it; returns the sum of in[0..n).
__device__ uint32_t block_scan_256(const uint32_t* in, uint32_t* out, uint32_t n, uint32_t carry,
                                   uint32_t* wtmp) {
    const uint32_t lane = threadIdx.x & 63u, wave = threadIdx.x >> 6;
    const uint32_t per = (n + 255u) / 256u;
    const uint32_t b0 = threadIdx.x * per;
    uint32_t loc = 0;
    for (uint32_t k = 0; k < per; ++k)
        if (b0 + k < n) loc += in[b0 + k];
    uint32_t x = loc;
    for (uint32_t off = 1; off < 64u; off <<= 1) {
        const uint32_t y = __shfl_up(x, off, 64);
        if (lane >= off) x += y;
    }
    if (lane == 63u) wtmp[wave] = x;
    __syncthreads();
    uint32_t before = 0, total = 0;
    for (uint32_t w = 0; w < 4u; ++w) {
        const uint32_t t = wtmp[w];
        if (w < wave) before += t;
        total += t;
    }
    uint32_t run = carry + before + x - loc;
    for (uint32_t k = 0; k < per; ++k)
        if (b0 + k < n) {
            const uint32_t v = in[b0 + k];
            out[b0 + k] = run;
            run += v;
        }
    __syncthreads();
    return total;
}

// One block per partition q: the fused kernel's per-block counts of q become
// exclusive offsets within q (in place); their sum is q's record count.
__global__ void __launch_bounds__(256) part_offsets_kernel(PartParams pp) {
    __shared__ uint32_t wtmp[4];
    uint32_t* h = pp.part_hist + (uint64_t)blockIdx.x * pp.n_regions;
    uint32_t carry = 0;
    for (uint32_t b0 = 0; b0 < pp.n_regions; b0 += 4096u) {
        const uint32_t n = min(4096u, pp.n_regions - b0);
        carry += block_scan_256(h + b0, h + b0, n, carry, wtmp);
    }
    if (threadIdx.x == 0) pp.part_count[blockIdx.x] = carry;
}

// One block per fused-kernel region: the region's records, kScatterChunk at a
// time, are counting-sorted by partition in LDS and written out so that each
// partition's records of the chunk form one contiguous run.
template <typename VT>
__global__ void __launch_bounds__(256) part_scatter_kernel(PartParams pp) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    __shared__ uint32_t wtmp[4];
    constexpr int PER = kScatterChunk / 256;
    const uint32_t P = pp.n_parts;
    const int shift = pp.part_shift;
    VT* sval = reinterpret_cast<VT*>(smem);
    uint32_t* sgid = reinterpret_cast<uint32_t*>(sval + kScatterChunk);
    uint32_t* lcnt = sgid + kScatterChunk;
    uint32_t* lstart = lcnt + P;
    uint32_t* lcur = lstart + P;
    const uint32_t b = blockIdx.x;
    for (uint32_t q = threadIdx.x; q < P; q += blockDim.x) {
        lcur[q] = pp.part_start[q] + pp.part_hist[(uint64_t)q * pp.n_regions + b];
        lcnt[q] = 0u;
    }
    __syncthreads();
    const uint32_t n = pp.region_count[b];
    const uint32_t* rg = pp.rec_gid + (uint64_t)b * pp.part_cap;
    const VT* rv = static_cast<const VT*>(pp.rec_val) + (uint64_t)b * pp.part_cap;
    VT* out_val = static_cast<VT*>(pp.sorted_val);
    for (uint32_t c0 = 0; c0 < n; c0 += (uint32_t)kScatterChunk) {
        const uint32_t cn = min((uint32_t)kScatterChunk, n - c0);
        uint32_t g[PER], rk[PER];
        VT v[PER];
#pragma unroll
        for (int k = 0; k < PER; ++k) {
            const uint32_t i = (uint32_t)k * 256u + threadIdx.x;
            g[k] = 0u;
            v[k] = 0;
            rk[k] = 0u;
            if (i < cn) {
                g[k] = rg[c0 + i];
                v[k] = rv[c0 + i];
            }
        }
#pragma unroll
        for (int k = 0; k < PER; ++k)
            if ((uint32_t)k * 256u + threadIdx.x < cn) rk[k] = atomicAdd(&lcnt[g[k] >> shift], 1u);
        __syncthreads();
        block_scan_256(lcnt, lstart, P, 0u, wtmp);
#pragma unroll
        for (int k = 0; k < PER; ++k)
            if ((uint32_t)k * 256u + threadIdx.x < cn) {
                const uint32_t pos = lstart[g[k] >> shift] + rk[k];
                sgid[pos] = g[k];
                sval[pos] = v[k];
            }
        __syncthreads();
        for (uint32_t i = threadIdx.x; i < cn; i += blockDim.x) {
            const uint32_t gi = sgid[i];
            const uint32_t q = gi >> shift;
            const uint32_t dest = lcur[q] + (i - lstart[q]);
            pp.sorted_gid[dest] = gi;
            out_val[dest] = sval[i];
        }
        __syncthreads();
        for (uint32_t q = threadIdx.x; q < P; q += blockDim.x) {
            lcur[q] += lcnt[q];
            lcnt[q] = 0u;
        }
        __syncthreads();
    }
}

size_t part_scatter_lds_bytes(uint32_t n_parts, bool wide) {
    return (size_t)kScatterChunk * (wide ? 12u : 8u) + (size_t)n_parts * 12u;
}

// Work item c covers up to kPartChunk records of one partition q: sum them in
// an LDS table of q's groups. A partition with one work item adds its table
// straight into the outputs; otherwise each item stores its table as a partial
// that part_merge_kernel adds up. Either way each output group has exactly one
// writer in this pass, so plain read-add-write suffices (the outputs already
// hold what the fused kernel added for records past a region's capacity).
constexpr int kAggUnroll = 8;
constexpr int kAggBlock = 1024;   // one work item is summed by 16 waves sharing its LDS table

template <typename VT>
__global__ void __launch_bounds__(kAggBlock) part_agg_kernel(PartParams pp) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    const uint32_t gpp = 1u << pp.part_shift;
    unsigned long long* lsum = reinterpret_cast<unsigned long long*>(smem);
    uint32_t* lcnt = reinterpret_cast<uint32_t*>(lsum + gpp);
    const uint32_t* sg = pp.sorted_gid;
    const VT* sv = static_cast<const VT*>(pp.sorted_val);
    const uint32_t n_items = pp.chunk_start[pp.n_parts];
    for (uint32_t c = blockIdx.x; c < n_items; c += gridDim.x) {
        // partition holding work item c: last q with chunk_start[q] <= c
        uint32_t lo = 0, hi = pp.n_parts;
        while (hi - lo > 1u) {
            const uint32_t mid = (lo + hi) >> 1;
            if (pp.chunk_start[mid] <= c) lo = mid;
            else hi = mid;
        }
        const uint32_t q = lo;
        const uint32_t r0 = pp.part_start[q] + (c - pp.chunk_start[q]) * (uint32_t)kPartChunk;
        const uint32_t r1 = min(r0 + (uint32_t)kPartChunk, pp.part_start[q + 1]);
        for (uint32_t k = threadIdx.x; k < gpp; k += blockDim.x) {
            lsum[k] = 0ull;
            lcnt[k] = 0u;
        }
        __syncthreads();
        const uint32_t g0 = q << pp.part_shift;
        // kAggUnroll records per thread in flight per step
        for (uint32_t i0 = r0; i0 < r1; i0 += kAggUnroll * blockDim.x) {
            uint32_t k[kAggUnroll];
            VT v[kAggUnroll];
#pragma unroll
            for (int u = 0; u < kAggUnroll; ++u) {
                const uint32_t i = i0 + (uint32_t)u * blockDim.x + threadIdx.x;
                k[u] = 0xFFFFFFFFu;
                v[u] = 0;
                if (i < r1) {
                    k[u] = sg[i] - g0;
                    v[u] = sv[i];
                }
            }
#pragma unroll
            for (int u = 0; u < kAggUnroll; ++u) {
                if (k[u] != 0xFFFFFFFFu) {
                    atomicAdd(&lsum[k[u]], (unsigned long long)(long long)v[u]);
                    atomicAdd(&lcnt[k[u]], 1u);
                }
            }
        }
        __syncthreads();
        const bool single = pp.chunk_start[q + 1] - pp.chunk_start[q] == 1u;
        const uint32_t kend = (uint32_t)min((uint64_t)gpp, pp.n_groups - g0);
        if (single) {
            for (uint32_t k = threadIdx.x; k < kend; k += blockDim.x) {
                pp.sums[g0 + k] += lsum[k];
                pp.counts[g0 + k] += lcnt[k];
            }
        } else {
            for (uint32_t k = threadIdx.x; k < kend; k += blockDim.x) {
                pp.item_sum[(uint64_t)c * gpp + k] = lsum[k];
                pp.item_cnt[(uint64_t)c * gpp + k] = lcnt[k];
            }
        }
        __syncthreads();
    }
}

// Groups of partitions with several work items: add the items' partials.
__global__ void __launch_bounds__(256) part_merge_kernel(PartParams pp) {
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    const uint32_t gpp = 1u << pp.part_shift;
    for (uint64_t g = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; g < pp.n_groups; g += stride) {
        const uint32_t q = (uint32_t)(g >> pp.part_shift);
        const uint32_t k = (uint32_t)g & (gpp - 1u);
        const uint32_t c0 = pp.chunk_start[q], c1 = pp.chunk_start[q + 1];
        if (c1 - c0 < 2u) continue;
        unsigned long long s = 0;
        unsigned long long n = 0;
        for (uint32_t c = c0; c < c1; ++c) {
            s += pp.item_sum[(uint64_t)c * gpp + k];
            n += pp.item_cnt[(uint64_t)c * gpp + k];
        }
        pp.sums[g] += s;
        pp.counts[g] += n;
    }
}

hipError_t launch_part_passes(const PartParams& pp, hipStream_t s) {
    hipLaunchKernelGGL(part_offsets_kernel, dim3(pp.n_parts), dim3(256), 0, s, pp);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(part_scan_kernel, dim3(1), dim3(1024), 0, s, pp);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const bool wide = pp.rec_wide != 0;
    const size_t agg_lds = (size_t)12u << pp.part_shift;
    if (wide) {
        hipLaunchKernelGGL(part_scatter_kernel<long long>, dim3(pp.n_regions), dim3(256),
                           part_scatter_lds_bytes(pp.n_parts, true), s, pp);
    } else {
        hipLaunchKernelGGL(part_scatter_kernel<int32_t>, dim3(pp.n_regions), dim3(256),
                           part_scatter_lds_bytes(pp.n_parts, false), s, pp);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (wide) hipLaunchKernelGGL(part_agg_kernel<long long>, dim3(512), dim3(kAggBlock), agg_lds, s, pp);
    else hipLaunchKernelGGL(part_agg_kernel<int32_t>, dim3(512), dim3(kAggBlock), agg_lds, s, pp);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(part_merge_kernel, dim3(fill_grid(pp.n_groups)), dim3(256), 0, s, pp);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// sliced hash probe: fact rows partitioned by the top bits of the key's hash
// ---------------------------------------------------------------------------

// Partition of key k: the top `bits` bits of its 32-bit multiplicative hash,
// which are also the top bits of its home slot in a table of at least 2^bits
// slots, so partition q probes only slice q of the table (and the slots
// that linear probing runs into past its end).
__device__ __forceinline__ uint32_t slice_of(int32_t k, int bits) {
    return ((uint32_t)k * 0x9E3779B1u) >> (32 - bits);
}

// Rows r .. r + 3 of a column (r a multiple of 4, the column 16-byte
// aligned): one 128-bit load, or row by row below r1 in a last partial group.
__device__ __forceinline__ void slice_load4(const int32_t* col, int64_t r, int64_t r1, int32_t* x) {
    if (r + 3 < r1) {
        const v4i v = __builtin_nontemporal_load(reinterpret_cast<const v4i*>(col + r));
        x[0] = v.x;
        x[1] = v.y;
        x[2] = v.z;
        x[3] = v.w;
    } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) x[j] = r + j < r1 ? __builtin_nontemporal_load(col + r + j) : 0;
    }
}

// A thread's rows of the chunk at c0: kSliceRowsPerThread / 4 groups of 4,
// group i at c0 + 4 * (i * kSliceBlock + threadIdx.x). Which of them lie below
// r1 and pass every fact predicate, and their keys (0 for the others).
template <int RPT>
__device__ __forceinline__ void slice_load_keys(const SliceParams& sp, int64_t c0, int64_t r1, int32_t (&k)[RPT],
                                                bool (&ok)[RPT]) {
    constexpr int G = RPT / 4;
#pragma unroll
    for (int i = 0; i < G; ++i) {
        const int64_t r = c0 + 4 * ((int64_t)i * kSliceBlock + threadIdx.x);
#pragma unroll
        for (int j = 0; j < 4; ++j) ok[4 * i + j] = r + j < r1;
    }
    for (int pi = 0; pi < sp.n_preds; ++pi) {
        const int32_t* col = sp.cols[sp.pred_col[pi]];
        const RangeTest t = sp.pred[pi];
#pragma unroll
        for (int i = 0; i < G; ++i) {
            const int64_t r = c0 + 4 * ((int64_t)i * kSliceBlock + threadIdx.x);
            if (!(ok[4 * i] || ok[4 * i + 1] || ok[4 * i + 2] || ok[4 * i + 3])) continue;
            int32_t x[4];
            slice_load4(col, r, r1, x);
#pragma unroll
            for (int j = 0; j < 4; ++j) ok[4 * i + j] = ok[4 * i + j] && range_pass(t, x[j]);
        }
    }
    const int32_t* key = sp.cols[sp.key_col];
#pragma unroll
    for (int i = 0; i < G; ++i) {
        const int64_t r = c0 + 4 * ((int64_t)i * kSliceBlock + threadIdx.x);
        int32_t x[4] = {0, 0, 0, 0};
        if (ok[4 * i] || ok[4 * i + 1] || ok[4 * i + 2] || ok[4 * i + 3]) slice_load4(key, r, r1, x);
#pragma unroll
        for (int j = 0; j < 4; ++j) k[4 * i + j] = ok[4 * i + j] ? x[j] : 0;
    }
}

// The pre-filter of the count pass: drops the rows whose key the table's
// pass filter rejects, and records for each of the thread's 4-row groups
// below r1 which of its rows stay (bit j: row 4 g + j), for the scatter pass.
template <int RPT>
__device__ __forceinline__ void slice_prefilter(const SliceParams& sp, int64_t c0, int64_t r1, const int32_t (&k)[RPT],
                                                bool (&ok)[RPT]) {
#pragma unroll
    for (int i = 0; i < RPT; ++i) {
        uint32_t w, m;
        if (ok[i]) ok[i] = filter_slot(sp.filt_kind, sp.filt_bits, sp.filt_key_min, k[i], w, m) &&
                           (sp.filt[w] & m) == m;
    }
#pragma unroll
    for (int i = 0; i < RPT / 4; ++i) {
        const int64_t r = c0 + 4 * ((int64_t)i * kSliceBlock + threadIdx.x);
        if (r < r1)
            sp.keep[r >> 2] = (uint8_t)((ok[4 * i] ? 1u : 0u) | (ok[4 * i + 1] ? 2u : 0u) | (ok[4 * i + 2] ? 4u : 0u) |
                                        (ok[4 * i + 3] ? 8u : 0u));
    }
}

// The scatter pass's rows after a pre-filter: which of the thread's rows the
// count pass kept, and their keys (0 for the others).
template <int RPT>
__device__ __forceinline__ void slice_load_kept(const SliceParams& sp, int64_t c0, int64_t r1, int32_t (&k)[RPT],
                                                bool (&ok)[RPT]) {
    const int32_t* key = sp.cols[sp.key_col];
#pragma unroll
    for (int i = 0; i < RPT / 4; ++i) {
        const int64_t r = c0 + 4 * ((int64_t)i * kSliceBlock + threadIdx.x);
        const uint32_t kb = r < r1 ? sp.keep[r >> 2] : 0u;
        int32_t x[4] = {0, 0, 0, 0};
        if (kb) slice_load4(key, r, r1, x);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            ok[4 * i + j] = ((kb >> j) & 1u) != 0u;
            k[4 * i + j] = ok[4 * i + j] ? x[j] : 0;
        }
    }
}

// Count pass: block b's passing rows per partition, into hist[q * grid + b].
// Lanes count into four interleaved copies of the histogram (by lane mod 4),
// so fewer lanes of one LDS atomic instruction hit the same counter.
__global__ void __launch_bounds__(kSliceBlock) slice_count_kernel(SliceParams sp) {
    __shared__ uint32_t lh[4 << SDB_MAX_SLICE_BITS];
    const uint32_t P = 1u << sp.bits;
    for (uint32_t q = threadIdx.x; q < 4u * P; q += blockDim.x) lh[q] = 0u;
    __syncthreads();
    uint32_t* mine = lh + (threadIdx.x & 3u);
    const int64_t r0 = (int64_t)blockIdx.x * sp.rows_per_block;
    const int64_t r1 = min(sp.n, r0 + sp.rows_per_block);
    for (int64_t c0 = r0; c0 < r1; c0 += kSliceChunk) {
        int32_t k[kSliceRowsPerThread];
        bool ok[kSliceRowsPerThread];
        slice_load_keys<kSliceRowsPerThread>(sp, c0, r1, k, ok);
        if (sp.filt) slice_prefilter<kSliceRowsPerThread>(sp, c0, r1, k, ok);
#pragma unroll
        for (int i = 0; i < kSliceRowsPerThread; ++i)
            if (ok[i]) atomicAdd(&mine[4u * slice_of(k[i], sp.bits)], 1u);
    }
    __syncthreads();
    for (uint32_t q = threadIdx.x; q < P; q += blockDim.x)
        sp.hist[(uint64_t)q * gridDim.x + blockIdx.x] = lh[4u * q] + lh[4u * q + 1u] + lh[4u * q + 2u] + lh[4u * q + 3u];
}

// Exclusive scan of n values by the whole block (blockDim.x a multiple of
// 64, at most 1024): out[i] = carry + sum of in[0..i); in and out distinct.
// Every thread must call it; returns the sum of in[0..n).
__device__ uint32_t block_scan_any(const uint32_t* in, uint32_t* out, uint32_t n, uint32_t carry,
                                   uint32_t* wtmp) {
    const uint32_t lane = threadIdx.x & 63u, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
    const uint32_t per = (n + blockDim.x - 1u) / blockDim.x;
    const uint32_t b0 = threadIdx.x * per;
    uint32_t loc = 0;
    for (uint32_t k = 0; k < per; ++k)
        if (b0 + k < n) loc += in[b0 + k];
    uint32_t x = loc;
    for (uint32_t off = 1; off < 64u; off <<= 1) {
        const uint32_t y = __shfl_up(x, off, 64);
        if (lane >= off) x += y;
    }
    if (lane == 63u) wtmp[wave] = x;
    __syncthreads();
    uint32_t before = 0, total = 0;
    for (uint32_t w = 0; w < nw; ++w) {
        const uint32_t t = wtmp[w];
        if (w < wave) before += t;
        total += t;
    }
    uint32_t run = carry + before + x - loc;
    for (uint32_t k = 0; k < per; ++k)
        if (b0 + k < n) {
            out[b0 + k] = run;
            run += in[b0 + k];
        }
    __syncthreads();
    return total;
}

// Scatter pass: block b reads its rows again, RPT * kSliceBlock at a time,
// sorts each chunk's passing rows by partition in LDS (counting sort) and
// writes every partition's run of keys and values (TWO: both operands of a
// two-column aggregate, in chunks half as long so they fit LDS) after the ones
// block b wrote before (hist holds block b's first offset within each
// partition). With a pre-filter the passing rows are the ones the count pass
// kept, read from its per-group bytes instead of testing the predicates again.
template <int RPT, bool TWO>
__global__ void __launch_bounds__(kSliceBlock) slice_scatter_kernel(SliceParams sp) {
    constexpr int CHUNK = RPT * kSliceBlock;
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    __shared__ uint32_t wtmp[kSliceBlock / 64];
    int32_t* skey = reinterpret_cast<int32_t*>(smem);
    int32_t* sval = skey + CHUNK;
    int32_t* sval2 = sval + CHUNK;            // TWO only
    const uint32_t P = 1u << sp.bits;
    uint32_t* lcnt = reinterpret_cast<uint32_t*>(sval + (TWO ? 2 : 1) * CHUNK);
    uint32_t* lstart = lcnt + P;
    uint32_t* lcur = lstart + P;
    for (uint32_t q = threadIdx.x; q < P; q += blockDim.x) {
        lcur[q] = sp.part_start[q] + sp.hist[(uint64_t)q * gridDim.x + blockIdx.x];
        lcnt[q] = 0u;
    }
    __syncthreads();
    const int64_t r0 = (int64_t)blockIdx.x * sp.rows_per_block;
    const int64_t r1 = min(sp.n, r0 + sp.rows_per_block);
    const int32_t* val = sp.cols[sp.val_col];
    const int32_t* val2 = sp.cols[TWO ? sp.val2_col : sp.val_col];
    for (int64_t c0 = r0; c0 < r1; c0 += CHUNK) {
        int32_t k[RPT], v[RPT], v2[RPT];
        bool ok[RPT];
        uint32_t rk[RPT];
        if (sp.keep) slice_load_kept<RPT>(sp, c0, r1, k, ok);
        else slice_load_keys<RPT>(sp, c0, r1, k, ok);
#pragma unroll
        for (int i = 0; i < RPT / 4; ++i) {
            const int64_t r = c0 + 4 * ((int64_t)i * kSliceBlock + threadIdx.x);
            int32_t x[4] = {0, 0, 0, 0}, y[4] = {0, 0, 0, 0};
            const bool any = ok[4 * i] || ok[4 * i + 1] || ok[4 * i + 2] || ok[4 * i + 3];
            if (any) slice_load4(val, r, r1, x);
            if (TWO && any) slice_load4(val2, r, r1, y);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                v[4 * i + j] = x[j];
                v2[4 * i + j] = y[j];
            }
        }
#pragma unroll
        for (int i = 0; i < RPT; ++i) {
            rk[i] = 0u;
            if (ok[i]) rk[i] = atomicAdd(&lcnt[slice_of(k[i], sp.bits)], 1u);
        }
        __syncthreads();
        const uint32_t cn = block_scan_any(lcnt, lstart, P, 0u, wtmp);
#pragma unroll
        for (int i = 0; i < RPT; ++i)
            if (ok[i]) {
                const uint32_t pos = lstart[slice_of(k[i], sp.bits)] + rk[i];
                skey[pos] = k[i];
                sval[pos] = v[i];
                if (TWO) sval2[pos] = v2[i];
            }
        __syncthreads();
        for (uint32_t i = threadIdx.x; i < cn; i += blockDim.x) {
            const int32_t key = skey[i];
            const uint32_t q = slice_of(key, sp.bits);
            const uint64_t dest = (uint64_t)lcur[q] + (i - lstart[q]);
            if (dest < (uint64_t)sp.n) {   // always: both passes count the same rows
                sp.out_key[dest] = key;
                sp.out_val[dest] = sval[i];
                if (TWO) sp.out_val2[dest] = sval2[i];
            }
        }
        __syncthreads();
        for (uint32_t q = threadIdx.x; q < P; q += blockDim.x) {
            lcur[q] += lcnt[q];
            lcnt[q] = 0u;
        }
        __syncthreads();
    }
}

// The tile order of the fused launch over the partitioned rows. Loop index t
// runs on block t mod grid, which the dispatcher places on XCD t mod 8 (the
// grids here are multiples of 8); giving XCD x only the tiles whose first row
// lies in a partition q with q mod 8 == x means each XCD's L2 holds the table
// slices of its own partitions, and each slice is probed by one XCD's 32 CUs
// for eight times as long, so the blocks drift apart by fewer slices.
// One thread: the rank of each partition's first tile among its XCD's tiles.
__global__ void slice_tile_base_kernel(SliceParams sp) {
    if (blockIdx.x != 0 || threadIdx.x != 0) return;
    const uint32_t P = 1u << sp.bits;
    const uint64_t T = (uint64_t)sp.tile_rows;
    uint64_t run[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (uint32_t q = 0; q < P; ++q) {
        const uint64_t a = ((uint64_t)sp.part_start[q] + T - 1) / T;
        const uint64_t b = ((uint64_t)sp.part_start[q + 1] + T - 1) / T;
        sp.tile_base[q] = (uint32_t)run[q & 7u];
        run[q & 7u] += b - a;
    }
}

// One thread per tile j (first row j * tile_rows below the passing-row count):
// its partition q (binary search of the partition starts), then its slot
// 8 * rank + (q mod 8) in the map (filled with -1 before).
__global__ void __launch_bounds__(256) slice_tile_map_kernel(SliceParams sp) {
    const uint32_t P = 1u << sp.bits;
    const uint64_t T = (uint64_t)sp.tile_rows;
    const uint64_t total = sp.part_start[P];
    const uint64_t n_phys = (total + T - 1) / T;
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t j = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; j < n_phys; j += stride) {
        const uint64_t row = j * T;
        uint32_t lo = 0, hi = P;   // last partition whose start is <= row
        while (hi - lo > 1u) {
            const uint32_t mid = (lo + hi) >> 1;
            if ((uint64_t)sp.part_start[mid] <= row) lo = mid;
            else hi = mid;
        }
        const uint64_t first = ((uint64_t)sp.part_start[lo] + T - 1) / T;
        const uint64_t v = 8u * ((uint64_t)sp.tile_base[lo] + (j - first)) + (lo & 7u);
        if (v < (uint64_t)sp.n_vtiles) sp.tile_map[v] = (int32_t)j;
    }
}

// rows per thread of the scatter chunk: half as many with two value columns
constexpr int kSliceRowsPerThreadTwo = kSliceRowsPerThread / 2;

size_t slice_scatter_lds_bytes(uint32_t n_parts, bool two) {
    const size_t chunk = (size_t)kSliceBlock * (two ? kSliceRowsPerThreadTwo : kSliceRowsPerThread);
    return chunk * 4u * (two ? 3u : 2u) + (size_t)n_parts * 12u;
}

hipError_t launch_slice_partition(const SliceParams& sp, int grid, hipStream_t s) {
    if (sp.bits < 1 || sp.bits > SDB_MAX_SLICE_BITS || grid < 1) return hipErrorInvalidValue;
    const uint32_t P = 1u << sp.bits;
    hipLaunchKernelGGL(slice_count_kernel, dim3(grid), dim3(kSliceBlock), 0, s, sp);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    PartParams pp;
    std::memset(&pp, 0, sizeof pp);
    pp.n_parts = P;
    pp.n_regions = (uint32_t)grid;
    pp.part_hist = sp.hist;
    pp.part_count = sp.part_count;
    pp.part_start = sp.part_start;
    pp.chunk_start = sp.chunk_start;
    hipLaunchKernelGGL(part_offsets_kernel, dim3(P), dim3(256), 0, s, pp);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(part_scan_kernel, dim3(1), dim3(1024), 0, s, pp);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (sp.val2_col >= 0)
        hipLaunchKernelGGL((slice_scatter_kernel<kSliceRowsPerThreadTwo, true>), dim3(grid), dim3(kSliceBlock),
                           slice_scatter_lds_bytes(P, true), s, sp);
    else
        hipLaunchKernelGGL((slice_scatter_kernel<kSliceRowsPerThread, false>), dim3(grid), dim3(kSliceBlock),
                           slice_scatter_lds_bytes(P, false), s, sp);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (sp.tile_map) {
        e = launch_fill_u32(reinterpret_cast<uint32_t*>(sp.tile_map), (uint64_t)sp.n_vtiles, 0xFFFFFFFFu, s);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(slice_tile_base_kernel, dim3(1), dim3(64), 0, s, sp);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        const uint64_t phys = (uint64_t)sp.n_vtiles / 8u;
        const int g = (int)std::min<uint64_t>(1024u, std::max<uint64_t>(1u, (phys + 255u) / 256u));
        hipLaunchKernelGGL(slice_tile_map_kernel, dim3(g), dim3(256), 0, s, sp);
    }
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// finalize: order-preserving compaction of the group table
// ---------------------------------------------------------------------------

__device__ __forceinline__ bool group_present(const FinalizeParams& fp, uint64_t g) {
    if (g >= fp.n_groups) return false;
    return fp.scalar ? true : fp.counts[g] > 0;
}

__global__ void __launch_bounds__(kFinBlock) fin_count_kernel(FinalizeParams fp) {
    __shared__ unsigned int wsum[kFinBlock / 64];
    const uint64_t base = (uint64_t)blockIdx.x * kFinGroupsPerBlock;
    unsigned int c = 0;
    for (int k = 0; k < kFinPerThread; ++k) c += group_present(fp, base + (uint64_t)k * kFinBlock + threadIdx.x);
    for (int off = 32; off > 0; off >>= 1) c += __shfl_xor(c, off, 64);
    if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = c;
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned int t = 0;
        for (int w = 0; w < kFinBlock / 64; ++w) t += wsum[w];
        fp.block_off[blockIdx.x] = t;
    }
}

// One block turns the per-block counts into exclusive offsets and writes the total.
__global__ void __launch_bounds__(1024) fin_scan_kernel(FinalizeParams fp) {
    __shared__ long long buf[1024];
    __shared__ long long carry;
    if (threadIdx.x == 0) carry = 0;
    __syncthreads();
    for (int64_t base = 0; base < fp.n_blocks; base += 1024) {
        const int64_t i = base + threadIdx.x;
        const long long v = i < fp.n_blocks ? fp.block_off[i] : 0;
        buf[threadIdx.x] = v;
        __syncthreads();
        for (int off = 1; off < 1024; off <<= 1) {       // Hillis-Steele inclusive scan
            const long long add = threadIdx.x >= (unsigned)off ? buf[threadIdx.x - off] : 0;
            __syncthreads();
            buf[threadIdx.x] += add;
            __syncthreads();
        }
        const long long incl = buf[threadIdx.x];
        if (i < fp.n_blocks) fp.block_off[i] = carry + incl - v;
        __syncthreads();
        if (threadIdx.x == 1023) carry += incl;
        __syncthreads();
    }
    if (threadIdx.x == 0) fp.out_n[0] = carry;
}

__global__ void __launch_bounds__(kFinBlock) fin_scatter_kernel(FinalizeParams fp) {
    __shared__ unsigned int wcnt[kFinBlock / 64];
    __shared__ long long run;
    if (threadIdx.x == 0) run = fp.block_off[blockIdx.x];
    __syncthreads();
    const uint64_t base = (uint64_t)blockIdx.x * kFinGroupsPerBlock;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    for (int k = 0; k < kFinPerThread; ++k) {
        const uint64_t g = base + (uint64_t)k * kFinBlock + threadIdx.x;
        const bool present = group_present(fp, g);
        const unsigned long long m = __ballot(present);
        const unsigned int before_in_wave = __popcll(m & ((1ull << lane) - 1ull));
        if (lane == 0) wcnt[wave] = __popcll(m);
        __syncthreads();
        unsigned int before = before_in_wave;
        unsigned int total = 0;
        for (int w = 0; w < kFinBlock / 64; ++w) {
            if (w < wave) before += wcnt[w];
            total += wcnt[w];
        }
        if (present) {
            const long long o = run + before;
            for (int q = 0; q < fp.n_keys; ++q)
                fp.out_keys[o * fp.n_keys + q] =
                    (int32_t)(((uint32_t)g / fp.stride[q]) % fp.radix[q]) + fp.key_min[q];
            fp.out_sums[o] = fp.sums[g];
            fp.out_counts[o] = fp.counts[g];
        }
        __syncthreads();
        if (threadIdx.x == 0) run += total;
        __syncthreads();
    }
}

hipError_t launch_finalize(const FinalizeParams& fp, hipStream_t s) {
    hipLaunchKernelGGL(fin_count_kernel, dim3((unsigned)fp.n_blocks), dim3(kFinBlock), 0, s, fp);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(fin_scan_kernel, dim3(1), dim3(1024), 0, s, fp);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(fin_scatter_kernel, dim3((unsigned)fp.n_blocks), dim3(kFinBlock), 0, s, fp);
    return hipGetLastError();
}

// ---- fixed device scratch for sdb_run_star_query_noalloc ------------------
//
// Callers that cannot allocate device memory (code under stream capture,
// serving loops, harnesses that forbid hipMalloc) run a query with this
// file-scope array as its run scratch. Every device the library runs on holds
// its own copy from the code object's load until the process ends. In host
// code the array's name is only a host-side stand-in: its device address comes
// from hipGetSymbolAddress, taken once per device with that device current.

static __device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

hipError_t noalloc_scratch(void** out) {
    static std::mutex mu;
    static void* per_device[kNoallocMaxDevices] = {};
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kNoallocMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!per_device[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p || ((uintptr_t)p & 255u) != 0) return hipErrorInvalidSymbol;
        per_device[dev] = p;
    }
    *out = per_device[dev];
    return hipSuccess;
}

}  // namespace sdb
