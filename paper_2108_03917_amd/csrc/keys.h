// Device helpers for packed lattice keys and the open-addressing hash table.
//
// The hash map of Sec. "Permutohedral Lattice" (key = vertex coordinates c_v)
// is a linear-probing table of 16-byte entries {packed key, number of
// (point, simplex vertex) pairs that hit the key, vertex index}: one 16-byte
// load answers a lookup, and the splat's per-vertex point lists are sized
// from the counts.  A slot is claimed with a 64-bit compare-and-swap of the
// key from 0 (empty) to the key.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"

struct __attribute__((aligned(16))) HEntry {
    unsigned long long key;  // 0 = empty
    int32_t count;           // pairs (p, k) whose vertex k has this key; after the numbering,
                             // the offset of the vertex's pair list (the count is then in vinfo)
    int32_t vid;             // vertex index (written by the numbering)
};
static_assert(sizeof(HEntry) == 16, "hash entry is 16 bytes");

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

// Home slot of a key: the low bits of its mixed value.
__device__ __forceinline__ uint32_t home_slot(uint64_t key, uint32_t mask) { return (uint32_t)key_mix(key) & mask; }

// Whether hash slot h holds a vertex: bit h of the occupancy bitmap.
__device__ __forceinline__ bool slot_taken(const uint32_t *__restrict__ occ, uint32_t h) {
    return (occ[h >> 5] >> (h & 31)) & 1u;
}

// Mark slot h occupied (once per vertex, by the numbering; no returned value
// to wait for).
__device__ __forceinline__ void mark_taken(uint32_t *occ, uint32_t h) { atomicOr(occ + (h >> 5), 1u << (h & 31)); }

// Look up N keys of a table that no thread is writing, all probes of one
// round in flight together.  `want[k]` false skips key k.  Returns the vertex
// index per key, -1 when absent.  Each probe first reads the slot's
// occupancy bit (a bitmap of cap / 8 bytes, which stays in L2): an empty
// slot ends the search without fetching the table's line, which is what most
// lookups of absent neighbours come down to.
template <int N>
__device__ __forceinline__ void hash_find_all(const HEntry *__restrict__ tab, const uint32_t *__restrict__ occ,
                                              uint32_t mask, const uint64_t *key, const bool *want, int *out) {
    uint32_t h[N];
    bool pending[N];
#pragma unroll
    for (int k = 0; k < N; ++k) {
        h[k] = want[k] ? home_slot(key[k], mask) : 0u;
        pending[k] = want[k];
        out[k] = -1;
    }
    for (uint32_t probe = 0; probe <= mask; ++probe) {
        bool taken[N];
#pragma unroll
        for (int k = 0; k < N; ++k) taken[k] = pending[k] && slot_taken(occ, h[k]);
        HEntry e[N];
#pragma unroll
        for (int k = 0; k < N; ++k)
            if (taken[k]) e[k] = tab[h[k]];
        bool any = false;
#pragma unroll
        for (int k = 0; k < N; ++k) {
            if (!pending[k]) continue;
            if (!taken[k]) {
                pending[k] = false;
            } else if (e[k].key == key[k]) {
                out[k] = e[k].vid;
                pending[k] = false;
            } else {
                h[k] = (h[k] + 1) & mask;
                any = true;
            }
        }
        if (!any) return;
    }
}
