// Device helpers shared by the kernels of libsdb (gfx950, wave64): vector
// types, predicate tests, wave reductions, non-temporal fact-column loads and
// the single-row lookups of dense maps and open-addressing hash tables.
#pragma once

#include <hip/hip_runtime.h>

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

}  // namespace sdb
