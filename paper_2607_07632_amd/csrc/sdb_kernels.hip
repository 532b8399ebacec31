// Device kernels of libsdb for CDNA4 (gfx950, wave64).
//
//  * dimension build: statistics pass, direct-mapped packed map scatter, and
//    open-addressing insert with 64-bit compare-and-swap (Section 3.3);
//  * plan sampling: each stage evaluated on its own over a strided fact sample;
//  * the fused probe-filter-aggregate pass (Sections 3.2, 4.2, 4.3);
//  * group-table compaction.
//
// The fused pass is a grid-stride persistent loop. A lane owns IPT items per
// iteration; an item is W consecutive fact rows (W = 4: one 128-bit load per
// column per item). Stages run in plan order; a stage loads its column only
// for items that still hold a live row, and the whole wave leaves the stage
// list as soon as no lane has a live row (wave-wide vote). Probes keep the
// group id in a register; the terminal is a register accumulator, an LDS
// group table, or global 64-bit atomics.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <climits>
#include <mutex>

#include "sdb_internal.h"

namespace sdb {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef unsigned int v4u __attribute__((ext_vector_type(4)));
typedef unsigned long long u64x2 __attribute__((ext_vector_type(2)));
typedef u64x2 __attribute__((aligned(8))) u64x2_a8;   // two adjacent 8-byte slots

// ---------------------------------------------------------------------------
// small helpers
// ---------------------------------------------------------------------------

__device__ __forceinline__ bool range_pass(const RangeTest& t, int32_t x) {
    return ((uint32_t)(x - t.lo) <= t.span) != (t.negate != 0);
}

__device__ __forceinline__ unsigned long long wave_sum_u64(unsigned long long v) {
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

__device__ __forceinline__ int32_t wave_min_i32(int32_t v) {
    for (int off = 32; off > 0; off >>= 1) v = min(v, __shfl_xor(v, off, 64));
    return v;
}

__device__ __forceinline__ int32_t wave_max_i32(int32_t v) {
    for (int off = 32; off > 0; off >>= 1) v = max(v, __shfl_xor(v, off, 64));
    return v;
}

// Loads the W rows of item `item` of a fact column (non-temporal: fact data is
// streamed once and should not evict the dimension maps and group tables).
template <int W>
__device__ __forceinline__ void load_item(const int32_t* col, int64_t item, int32_t (&x)[W]) {
    if constexpr (W == 4) {
        v4i v = __builtin_nontemporal_load(reinterpret_cast<const v4i*>(col) + item);
        x[0] = v.x;
        x[1] = v.y;
        x[2] = v.z;
        x[3] = v.w;
    } else {
        x[0] = __builtin_nontemporal_load(col + item);
    }
}

__device__ __forceinline__ uint32_t load_dense_code(const StageDev& S, uint32_t idx) {
    if (S.width == 1) return static_cast<const uint8_t*>(S.map)[idx];
    if (S.width == 2) return static_cast<const uint16_t*>(S.map)[idx];
    return static_cast<const uint32_t*>(S.map)[idx];
}

__device__ __forceinline__ uint32_t hash_slot(const StageDev& S, int32_t k) {
    return ((uint32_t)k * 0x9E3779B1u) >> S.hshift & S.hmask;
}

// Resolves a hash probe whose first slot value is `slot`; returns the code or
// the sentinel. Linear probing; at most nslots slots are inspected.
__device__ __forceinline__ uint32_t hash_resolve(const StageDev& S, int32_t k, uint32_t h,
                                                 unsigned long long slot) {
    const unsigned long long* tab = static_cast<const unsigned long long*>(S.map);
    for (uint32_t it = 0; it < S.nslots; ++it) {
        const uint32_t hi = (uint32_t)(slot >> 32);
        if (hi == 0u) return S.sentinel;                       // empty slot: key absent
        if ((int32_t)(uint32_t)slot == k) return hi - 1u;      // a filtered row holds 0xFFFFFFFF: the sentinel
        h = (h + 1u) & S.hmask;
        slot = tab[h];
    }
    return S.sentinel;
}

__device__ __forceinline__ uint32_t code_contribution(const StageDev& S, uint32_t c) {
    uint32_t g = 0;
    for (int k = 0; k < S.n_gk; ++k) {
        uint32_t q = c;
        if (S.gk_div[k] != 1u) q /= S.gk_div[k];
        if (S.gk_radix[k] != 0u) q %= S.gk_radix[k];
        g += q * S.gk_stride[k];
    }
    return g;
}

// One stage for a single row (plan sampling).
__device__ __forceinline__ bool stage_pass_one(const StageDev& S, int32_t x) {
    if (S.kind == ST_PRED) return range_pass(S.test, x);
    if (S.kind == ST_DENSE) {
        const uint32_t idx = (uint32_t)(x - S.kmin);
        return idx < S.nslots && load_dense_code(S, idx) < S.sentinel;
    }
    const uint32_t h = hash_slot(S, x);
    const unsigned long long* tab = static_cast<const unsigned long long*>(S.map);
    return hash_resolve(S, x, h, tab[h]) < S.sentinel;
}

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

__global__ void stats_init_kernel(BuildBatch kernel_args) {
    (void)kernel_args;
    const BuildBatch& bb = *(const BuildBatch*)__builtin_amdgcn_kernarg_segment_ptr();
    if (blockIdx.x == 0 && threadIdx.x < (uint32_t)bb.n) {
        DimStats* st = bb.bp[threadIdx.x].stats;
        st->kmin = INT_MAX;
        st->kmax = INT_MIN;
        st->npass = 0ull;
        for (int p = 0; p < SDB_MAX_PAYLOADS; ++p) {
            st->pmin[p] = INT_MAX;
            st->pmax[p] = INT_MIN;
        }
        st->dup = 0u;
        st->occupied = 0ull;
        st->pkmin = INT_MAX;
        st->pkmax = INT_MIN;
    }
}

// Key range over all rows; pass count and payload ranges over passing rows.
constexpr int kStatsRows = 16;

// Each block reduces in registers and LDS and then adds its result with one
// set of atomics, so the atomics stay few however large the dimension.
__global__ void __launch_bounds__(256) dim_stats_kernel(BuildBatch kernel_args) {
    SDB_BATCH_TABLE;
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
    // kStatsRows rows per thread per step, each column's loads issued together
    constexpr int U = kStatsRows;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x * U;
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
        DimStats* st = bp.stats;
        if (kmin != INT_MAX) atomicMin(&st->kmin, kmin);
        if (kmax != INT_MIN) atomicMax(&st->kmax, kmax);
        if (npass) {
            atomicAdd(&st->npass, npass);
            atomicMin(&st->pkmin, pkmin);
            atomicMax(&st->pkmax, pkmax);
            for (int p = 0; p < bp.n_payloads; ++p) {
                atomicMin(&st->pmin[p], pmin[p]);
                atomicMax(&st->pmax[p], pmax[p]);
            }
        }
    }
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
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < bp.n; i += stride) {
        const uint32_t idx = (uint32_t)(bp.key[i] - bp.kmin);
        if ((uint64_t)idx >= bp.nslots) {          // cannot happen: kmin/kmax cover all keys
            atomicOr(&bp.stats->dup, 4u);
            continue;
        }
        const uint32_t c = dim_row_passes(bp, i) ? dim_row_code(bp, i) : bp.sentinel;
        if (bp.width == 1) static_cast<uint8_t*>(bp.map)[idx] = (uint8_t)c;
        else if (bp.width == 2) static_cast<uint16_t*>(bp.map)[idx] = (uint16_t)c;
        else static_cast<uint32_t*>(bp.map)[idx] = c;
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

// Open addressing, linear probing, 8-byte slots {key, code + 1 | 0xFFFFFFFF}.
__global__ void __launch_bounds__(256) hash_insert_kernel(BuildBatch kernel_args) {
    SDB_BATCH_TABLE;
    if (bp.dense) return;
    unsigned long long* tab = static_cast<unsigned long long*>(bp.map);
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < bp.n; i += stride) {
        const int32_t k = bp.key[i];
        const uint32_t enc = dim_row_passes(bp, i) ? dim_row_code(bp, i) + 1u : 0xFFFFFFFFu;
        const unsigned long long slot = ((unsigned long long)enc << 32) | (uint32_t)k;
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

static int build_grid(int64_t n) {
    int64_t g = (n + 255) / 256;
    if (g > 2048) g = 2048;
    if (g < 1) g = 1;
    return (int)g;
}

hipError_t launch_build_stats(const BuildBatch& bb, hipStream_t s) {
    if (bb.n <= 0) return hipSuccess;
    hipLaunchKernelGGL(stats_init_kernel, dim3(1), dim3(64), 0, s, bb);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    int64_t n_max = 0;
    for (int d = 0; d < bb.n; ++d) n_max = std::max<int64_t>(n_max, bb.bp[d].n);
    if (n_max == 0) return hipSuccess;
    // few blocks per table: every block ends with one set of atomics on the same words
    int g = build_grid((n_max + kStatsRows - 1) / kStatsRows);
    if (g > 256) g = 256;
    hipLaunchKernelGGL(dim_stats_kernel, dim3(g, bb.n), dim3(256), 0, s, bb);
    return hipGetLastError();
}

hipError_t launch_build_tables(const BuildBatch& bb, hipStream_t s) {
    if (bb.n <= 0) return hipSuccess;
    uint64_t words = 0, n_words32 = 0;
    int64_t n_dense = 0, n_hash = 0;
    for (int d = 0; d < bb.n; ++d) {
        const BuildParams& bp = bb.bp[d];
        words = std::max<uint64_t>(words, bp.fill_words);
        if (bp.dense) {
            n_dense = std::max<int64_t>(n_dense, bp.n);
            n_words32 = std::max<uint64_t>(n_words32, (bp.nslots + 31) / 32);
        } else {
            n_hash = std::max<int64_t>(n_hash, bp.n);
        }
    }
    if (words > 0) {
        hipLaunchKernelGGL(fill_table_kernel, dim3(fill_grid(words), bb.n), dim3(256), 0, s, bb);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (n_dense > 0) {
        hipLaunchKernelGGL(dense_scatter_kernel, dim3(build_grid(n_dense), bb.n), dim3(256), 0, s, bb);
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

__global__ void __launch_bounds__(256) sample_kernel(FusedParams kernel_args, int64_t step, int64_t n_sample,
                                                     unsigned long long* pass_counts) {
    (void)kernel_args;
    const FusedParams& p = *(const FusedParams*)__builtin_amdgcn_kernarg_segment_ptr();
    __shared__ unsigned int cnt[kMaxStages];
    if (threadIdx.x < kMaxStages) cnt[threadIdx.x] = 0u;
    __syncthreads();
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    // every lane runs the same number of iterations so the wave-wide votes below are complete
    const int64_t n_iter = (n_sample + stride - 1) / stride;
    for (int64_t it = 0; it < n_iter; ++it) {
        const int64_t k = it * stride + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
        const bool valid = k < n_sample;
        const int64_t row = valid ? k * step : 0;
        for (int s = 0; s < p.nstages; ++s) {
            const StageDev& S = p.st[s];
            bool pass = false;
            if (valid) pass = stage_pass_one(S, p.cols[S.col][row]);
            const unsigned long long m = __ballot(pass);
            if ((threadIdx.x & 63) == 0 && m) atomicAdd(&cnt[s], (unsigned int)__popcll(m));
        }
    }
    __syncthreads();
    if (threadIdx.x < p.nstages && cnt[threadIdx.x])
        atomicAdd(&pass_counts[threadIdx.x], (unsigned long long)cnt[threadIdx.x]);
}

hipError_t launch_sample(const FusedParams& p, int64_t step, int64_t n_sample,
                         unsigned long long* pass_counts, hipStream_t s) {
    hipLaunchKernelGGL(fill_u64_kernel, dim3(1), dim3(64), 0, s, pass_counts, (uint64_t)kMaxStages);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || n_sample == 0 || p.nstages == 0) return e;
    int64_t g = (n_sample + 255) / 256;
    if (g > 256) g = 256;
    hipLaunchKernelGGL(sample_kernel, dim3((int)g), dim3(256), 0, s, p, step, n_sample, pass_counts);
    return hipGetLastError();
}

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
        ts.lfill = reinterpret_cast<uint32_t*>(lds);
        ts.lhist = ts.lfill + 1;
        for (uint32_t i = threadIdx.x; i < 1u + p.n_parts; i += blockDim.x) ts.lfill[i] = 0u;
        // rings: every wave's 8-byte entries (values, or {group id, value}),
        // then (64-bit values) every wave's group ids
        const uint32_t wave = threadIdx.x >> 6;
        const uint32_t vbytes = p.rec_wide ? 8u : 4u;
        ts.ring_val = lds + p.ring_off + (size_t)wave * kRing * 8u;
        ts.ring_gid = reinterpret_cast<uint32_t*>(lds + p.ring_off + (blockDim.x >> 6) * kRing * 8u) +
                      (size_t)wave * kRing;
        ts.rgid = p.rec_gid + (uint64_t)blockIdx.x * p.part_cap;
        ts.rval = static_cast<unsigned char*>(p.rec_val) + (uint64_t)blockIdx.x * p.part_cap * vbytes;
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
        if (threadIdx.x == 0) p.region_count[blockIdx.x] = min(*ts.lfill, p.part_cap);
        // this block's column of the partition x block histogram
        for (uint32_t q = threadIdx.x; q < p.n_parts; q += blockDim.x)
            p.part_hist[(uint64_t)q * gridDim.x + blockIdx.x] = ts.lhist[q];
    }
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

template <int W, int IPT, int TERM, bool EG, int LB = kMaxBlock, int UNR = 0>
static const void* fused_fn() {
    return reinterpret_cast<const void*>(&star_fused_kernel<W, IPT, TERM, EG, LB, UNR>);
}

// Instances: 4-row or 1-row items, 1/2/4 items per lane, every terminal;
// eager column loads for 4-row items with 1 or 2 items per lane; blocks of
// kBigBlock threads for 4-row items with 1 or 2 items per lane; the stage
// loop written out kUnrollStages times for 4-row items, 2 items per lane,
// blocks of kMaxBlock or kBigBlock and no eager loads.
static const void* pick_fused(int vector, int ipt, int terminal, int eager, int block, int unroll) {
    if (unroll) {
        if (!vector || ipt != 2 || eager > 0) return nullptr;
#define SDB_PICK_UNR(LBv)                                                                           \
    if (block == LBv) {                                                                             \
        if (terminal == TERM_SCALAR) return fused_fn<4, 2, TERM_SCALAR, false, LBv, kUnrollStages>(); \
        if (terminal == TERM_LDS) return fused_fn<4, 2, TERM_LDS, false, LBv, kUnrollStages>();       \
        if (terminal == TERM_GLOBAL) return fused_fn<4, 2, TERM_GLOBAL, false, LBv, kUnrollStages>(); \
        if (terminal == TERM_PART) return fused_fn<4, 2, TERM_PART, false, LBv, kUnrollStages>();     \
    }
        SDB_PICK_UNR(kMaxBlock)
        SDB_PICK_UNR(kBigBlock)
#undef SDB_PICK_UNR
        return nullptr;
    }
#define SDB_PICK(Wv, I, EGv, LBv)                                                        \
    if (ipt == I) {                                                                      \
        if (terminal == TERM_SCALAR) return fused_fn<Wv, I, TERM_SCALAR, EGv, LBv>();    \
        if (terminal == TERM_LDS) return fused_fn<Wv, I, TERM_LDS, EGv, LBv>();          \
        if (terminal == TERM_GLOBAL) return fused_fn<Wv, I, TERM_GLOBAL, EGv, LBv>();    \
        if (terminal == TERM_PART) return fused_fn<Wv, I, TERM_PART, EGv, LBv>();        \
    }
    if (block == kBigBlock) {
        if (!vector || eager > 0) return nullptr;
        SDB_PICK(4, 1, false, kBigBlock)
        SDB_PICK(4, 2, false, kBigBlock)
        return nullptr;
    }
    if (block > kMaxBlock) return nullptr;
    if (eager > 0) {
        if (!vector) return nullptr;
        SDB_PICK(4, 1, true, kMaxBlock)
        SDB_PICK(4, 2, true, kMaxBlock)
    } else if (vector) {
        SDB_PICK(4, 1, false, kMaxBlock)
        SDB_PICK(4, 2, false, kMaxBlock)
        SDB_PICK(4, 4, false, kMaxBlock)
    } else {
        SDB_PICK(1, 1, false, kMaxBlock)
        SDB_PICK(1, 2, false, kMaxBlock)
        SDB_PICK(1, 4, false, kMaxBlock)
    }
#undef SDB_PICK
    return nullptr;
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
__device__ __forceinline__ void slice_load_keys(const SliceParams& sp, int64_t c0, int64_t r1,
                                                int32_t (&k)[kSliceRowsPerThread],
                                                bool (&ok)[kSliceRowsPerThread]) {
    constexpr int G = kSliceRowsPerThread / 4;
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
        slice_load_keys(sp, c0, r1, k, ok);
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

// Scatter pass: block b reads its rows again, kSliceChunk at a time, sorts
// each chunk's passing rows by partition in LDS (counting sort) and writes
// every partition's run of keys and values after the ones block b wrote
// before (hist holds block b's first offset within each partition).
__global__ void __launch_bounds__(kSliceBlock) slice_scatter_kernel(SliceParams sp) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    __shared__ uint32_t wtmp[kSliceBlock / 64];
    int32_t* skey = reinterpret_cast<int32_t*>(smem);
    int32_t* sval = skey + kSliceChunk;
    const uint32_t P = 1u << sp.bits;
    uint32_t* lcnt = reinterpret_cast<uint32_t*>(sval + kSliceChunk);
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
    for (int64_t c0 = r0; c0 < r1; c0 += kSliceChunk) {
        int32_t k[kSliceRowsPerThread], v[kSliceRowsPerThread];
        bool ok[kSliceRowsPerThread];
        uint32_t rk[kSliceRowsPerThread];
        slice_load_keys(sp, c0, r1, k, ok);
#pragma unroll
        for (int i = 0; i < kSliceRowsPerThread / 4; ++i) {
            const int64_t r = c0 + 4 * ((int64_t)i * kSliceBlock + threadIdx.x);
            int32_t x[4] = {0, 0, 0, 0};
            if (ok[4 * i] || ok[4 * i + 1] || ok[4 * i + 2] || ok[4 * i + 3]) slice_load4(val, r, r1, x);
#pragma unroll
            for (int j = 0; j < 4; ++j) v[4 * i + j] = x[j];
        }
#pragma unroll
        for (int i = 0; i < kSliceRowsPerThread; ++i) {
            rk[i] = 0u;
            if (ok[i]) rk[i] = atomicAdd(&lcnt[slice_of(k[i], sp.bits)], 1u);
        }
        __syncthreads();
        const uint32_t cn = block_scan_any(lcnt, lstart, P, 0u, wtmp);
#pragma unroll
        for (int i = 0; i < kSliceRowsPerThread; ++i)
            if (ok[i]) {
                const uint32_t pos = lstart[slice_of(k[i], sp.bits)] + rk[i];
                skey[pos] = k[i];
                sval[pos] = v[i];
            }
        __syncthreads();
        for (uint32_t i = threadIdx.x; i < cn; i += blockDim.x) {
            const int32_t key = skey[i];
            const uint32_t q = slice_of(key, sp.bits);
            const uint64_t dest = (uint64_t)lcur[q] + (i - lstart[q]);
            if (dest < (uint64_t)sp.n) {   // always: both passes count the same rows
                sp.out_key[dest] = key;
                sp.out_val[dest] = sval[i];
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

size_t slice_scatter_lds_bytes(uint32_t n_parts) {
    return (size_t)kSliceChunk * 8u + (size_t)n_parts * 12u;
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
    hipLaunchKernelGGL(slice_scatter_kernel, dim3(grid), dim3(kSliceBlock), slice_scatter_lds_bytes(P), s, sp);
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
