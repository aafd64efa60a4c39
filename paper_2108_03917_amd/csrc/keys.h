// Device helpers for packed lattice keys and the open-addressing hash table.
//
// The hash map of Sec. "Permutohedral Lattice" (key = vertex coordinates c_v)
// is a linear-probing table of 64-bit packed keys with a parallel array of
// vertex indices.  A slot is claimed with a 64-bit compare-and-swap from 0
// (empty) to the key; the claiming thread later writes the vertex index.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"

// 64-bit finaliser of MurmurHash3 (Appleby): a bijective mixer, so distinct
// keys never collide before the mask is applied.
__device__ __forceinline__ uint64_t key_mix(uint64_t k) {
    k ^= k >> 33;
    k *= 0xff51afd7ed558ccdull;
    k ^= k >> 33;
    k *= 0xc4ceb9fe1a85ec53ull;
    k ^= k >> 33;
    return k;
}

// Pack c_0..c_{D-1} (+ batch id for D <= 3).  Returns false when a
// coordinate falls outside [-KEY_MAX, KEY_MAX].
template <int D>
__device__ __forceinline__ bool pack_key(const int *c, uint32_t batch, uint64_t &key) {
    uint64_t k = 0;
    bool ok = true;
#pragma unroll
    for (int i = 0; i < D; ++i) {
        int v = c[i];
        ok = ok && (v >= -KEY_MAX) && (v <= KEY_MAX);
        k |= (uint64_t)(uint32_t)(v + KEY_BIAS) << (16 * i);
    }
    if (D <= 3) k |= (uint64_t)batch << 48;
    key = k;
    return ok;
}

template <int D>
__device__ __forceinline__ void unpack_key(uint64_t key, int *c, uint32_t &batch) {
#pragma unroll
    for (int i = 0; i < D; ++i) c[i] = (int)((key >> (16 * i)) & 0xffffu) - KEY_BIAS;
    batch = (D <= 3) ? (uint32_t)(key >> 48) : 0u;
}

// Insert `key`; returns its slot, or -1 when every slot was probed.
// `is_new` is true for the one thread whose CAS claimed the slot.
__device__ __forceinline__ int hash_insert(uint64_t *tkeys, uint32_t mask, uint64_t key, bool &is_new) {
    uint32_t h = (uint32_t)key_mix(key) & mask;
    is_new = false;
    for (uint32_t probe = 0; probe <= mask; ++probe) {
        uint64_t cur = __hip_atomic_load(tkeys + h, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (cur == key) return (int)h;
        if (cur == 0) {
            unsigned long long old = atomicCAS((unsigned long long *)(tkeys + h), 0ull,
                                               (unsigned long long)key);
            if (old == 0ull) {
                is_new = true;
                return (int)h;
            }
            if (old == (unsigned long long)key) return (int)h;
        }
        h = (h + 1) & mask;
    }
    return -1;
}

// Look up `key` in a table that no thread is writing; returns the vertex
// index or -1 when the key is absent.
__device__ __forceinline__ int hash_find(const uint64_t *__restrict__ tkeys, const int32_t *__restrict__ tvals,
                                         uint32_t mask, uint64_t key) {
    uint32_t h = (uint32_t)key_mix(key) & mask;
    for (uint32_t probe = 0; probe <= mask; ++probe) {
        uint64_t cur = tkeys[h];
        if (cur == key) return tvals[h];
        if (cur == 0) return -1;
        h = (h + 1) & mask;
    }
    return -1;
}
