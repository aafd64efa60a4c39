// Splat: elevation onto H_d, enclosing simplex, barycentric weights, hash
// insertion of the d+1 vertex keys (Sec. "Permutohedral Lattice"), and the
// barycentric accumulation of Eq. (splat).
//
// Kernel sequence of one lattice_splat (all on the lattice's stream):
//   k_clear_table   empty the table: the slots the last splat occupied (its
//                   vertices' slots) when they are few, else all of it (and
//                   always all of it on the first splat or after a failed
//                   launch); zero V, the pair count and the status
//   k_insert        one thread per point: elevate, round, rank, wrap, weights,
//                   keys; CAS-insert of the d+1 keys (runs of equal keys in
//                   neighbouring lanes are inserted once), a rank for every
//                   (point, vertex) pair from the slot's counter
//   k_scan_count/assign  vertex indices (in order of creation) and pair-list ranges
//   k_fill          per pair: slot -> vertex index, (p, b_pk) into the list
//   k_gather_parts  the parts (kPart pairs) of long pair lists, as partial rows
//   k_gather        per vertex: x_v = sum b_pv f_p and w_v = sum b_pv
//                   (optionally x_v / w_v), each row written once; a long
//                   list's row is the sum of its part rows
#include "internal.h"
#include "keys.h"

namespace {

constexpr int kBlock = 256;


struct ElevParams {
    float f[LATTICE_MAX_D];
    float inv;
};

// Elevation x = alpha E (g / sigma) with the per-axis factors folded in:
// s_j = g_{j-1} f_j;  x_j = (s_{j+1} + .. + s_d) - j s_j;  x_0 = s_1 + .. + s_d.
// The running sum goes from j = d down to 1.  Every product and sum is rounded
// on its own (no contraction), so the host oracle can take the same integer
// decisions from the same fp32 values.
template <int D>
__device__ __forceinline__ void elevate(const float *g, const ElevParams &ep, float *x) {
#pragma clang fp contract(off)
    float S = 0.f;
#pragma unroll
    for (int j = D; j >= 1; --j) {
        const float s = g[j - 1] * ep.f[j - 1];
        const float t = (float)j * s;
        x[j] = S - t;
        S = S + s;
    }
    x[0] = S;
}

constexpr int kInsertBlock = 64;  // one wavefront per workgroup: small clouds still spread over every CU

// Elevation, enclosing simplex, barycentric weights and the d+1 vertex keys
// of point p (Sec. "Permutohedral Lattice"); shared by both insert kernels.
// Inactive points (p >= m) get zero keys and weights.
template <int D>
__device__ __forceinline__ void point_keys(const float *__restrict__ pos, const int32_t *__restrict__ batch, int64_t p,
                                           bool active, const ElevParams &ep, uint64_t *key, float *b, int &status) {
#pragma clang fp contract(off)
    constexpr int DP1 = D + 1;
#pragma unroll
    for (int k = 0; k < DP1; ++k) {
        key[k] = 0;
        b[k] = 0.f;
    }

    if (active) {
        float g[D];
#pragma unroll
        for (int j = 0; j < D; ++j) g[j] = pos[p * D + j];
        float x[DP1];
        elevate<D>(g, ep, x);

        // Remainder-0 point: r_i = (d+1) * round_half_even(x_i * fl(1/(d+1))).
        int r[DP1];
        float dl[DP1];
        bool finite = true;
#pragma unroll
        for (int i = 0; i < DP1; ++i) {
            const float q = rintf(x[i] * ep.inv);
            const bool ok = fabsf(q) < 1.0e7f;  // false for NaN and inf too
            finite = finite && ok;
            r[i] = ok ? (int)q * DP1 : 0;
            dl[i] = x[i] - (float)r[i];
        }
        // rank_i = #{j: dl_j > dl_i} + #{j < i: dl_j == dl_i}  (rank 0 = largest)
        int rank[DP1];
#pragma unroll
        for (int i = 0; i < DP1; ++i) {
            int rk = 0;
#pragma unroll
            for (int j = 0; j < DP1; ++j) rk += (dl[j] > dl[i]) || (j < i && dl[j] == dl[i]);
            rank[i] = rk;
        }
        // Wrap-around so that the remainder-0 point's coordinates sum to zero.
        int sum = 0;
#pragma unroll
        for (int i = 0; i < DP1; ++i) sum += r[i];
        const int s = sum / DP1;
#pragma unroll
        for (int i = 0; i < DP1; ++i) {
            int rk = rank[i] + s;
            if (rk < 0) {
                rk += DP1;
                r[i] += DP1;
            } else if (rk > D) {
                rk -= DP1;
                r[i] -= DP1;
            }
            rank[i] = rk;
        }
        // Barycentric weights: z_q = delta of rank q, delta_i = (x_i - r_i)/(d+1);
        // b_k = z_{d-k} - z_{d+1-k} (k = 1..d), b_0 = 1 - (z_0 - z_d).
        // Evaluated in fp64 (the differences of nearly equal deltas cancel) and
        // rounded once to fp32, so every weight carries a relative error of at
        // most half an fp32 ulp.  Coordinate i adds its delta to slot d - rank_i
        // and subtracts it from slot d+1-rank_i.
        double bb[DP1 + 1];
#pragma unroll
        for (int q = 0; q <= DP1; ++q) bb[q] = 0.0;
#pragma unroll
        for (int i = 0; i < DP1; ++i) {
            const double z = ((double)x[i] - (double)r[i]) / (double)DP1;
#pragma unroll
            for (int q = 0; q <= DP1; ++q) {
                if (q == D - rank[i]) bb[q] += z;
                if (q == DP1 - rank[i]) bb[q] -= z;
            }
        }
        // slot 0 holds +z_d, slot d+1 holds -z_0
        b[0] = (float)(1.0 - ((-bb[DP1]) - bb[0]));
#pragma unroll
        for (int q = 1; q <= D; ++q) b[q] = (float)bb[q];

        uint32_t bid = 0;
        if (batch) {
            const int32_t bv = batch[p];
            if (bv < 0 || bv > 65535) status |= ST_RANGE;
            bid = (uint32_t)bv & 0xffffu;
        }
        if (!finite) status |= ST_RANGE;
        // Key of the vertex with remainder k: c_i = r_i + k - (d+1)[rank_i > d - k].
#pragma unroll
        for (int k = 0; k < DP1; ++k) {
            int c[D];
#pragma unroll
            for (int i = 0; i < D; ++i) c[i] = r[i] + k - ((rank[i] > D - k) ? DP1 : 0);
            if (!pack_key<D>(c, bid, key[k])) status |= ST_RANGE;
        }
    }
}

// Bit of a pair's slot record that marks the pair whose insertion created
// the vertex (slots are below 2^30).
constexpr int kCreator = 1 << 30;

template <int D>
__global__ __launch_bounds__(kInsertBlock) void k_insert(const float *__restrict__ pos, const int32_t *__restrict__ batch,
                                                   int64_t m, ElevParams ep, HEntry *tab, uint32_t mask,
                                                   int32_t *__restrict__ idx, int32_t *__restrict__ rank_out,
                                                   float *__restrict__ bary, int32_t *counters) {
#pragma clang fp contract(off)
    constexpr int DP1 = D + 1;
    const int64_t p = (int64_t)blockIdx.x * kInsertBlock + threadIdx.x;
    const bool active = p < m;
    const int lane = threadIdx.x & 63;

    uint64_t key[DP1];
    float b[DP1];
    int status = 0;
    point_keys<D>(pos, batch, p, active, ep, key, b, status);
    const bool ok = active && status == 0;

    // Wave-level dedup: neighbouring lanes often carry the same key (points
    // of one simplex share its vertex of remainder k).  A run of equal keys in
    // consecutive lanes is inserted and counted once, by its first lane.
    const uint64_t below_mask = (2ull << lane) - 1ull;  // lanes 0..lane (wraps to all ones at lane 63)
    uint64_t hkey[DP1];
    int head[DP1], runlen[DP1];
#pragma unroll
    for (int k = 0; k < DP1; ++k) {
        const uint64_t kk = ok ? key[k] : 0ull;
        const uint64_t prev = __shfl_up(kk, 1, 64);
        const bool is_head = (lane == 0) || (kk != prev);
        const uint64_t heads = __ballot(is_head);
        head[k] = 63 - __clzll((long long)(heads & below_mask));
        const uint64_t above = lane == 63 ? 0ull : (heads >> (lane + 1));
        runlen[k] = above ? __ffsll((long long)above) : 64 - lane;
        hkey[k] = (is_head && kk != 0ull) ? kk : 0ull;
    }

    // Head lanes claim or find their slots; the d+1 probes of one round are in
    // flight together.
    int slot[DP1];
    bool pend[DP1], created[DP1];
    uint32_t h[DP1];
#pragma unroll
    for (int k = 0; k < DP1; ++k) {
        slot[k] = -1;
        created[k] = false;
        pend[k] = hkey[k] != 0ull;
        h[k] = pend[k] ? home_slot(hkey[k], mask) : 0u;
    }
    for (uint32_t probe = 0; probe <= mask; ++probe) {
        unsigned long long old[DP1];
#pragma unroll
        for (int k = 0; k < DP1; ++k)
            if (pend[k]) old[k] = atomicCAS(&tab[h[k]].key, 0ull, (unsigned long long)hkey[k]);
        bool any = false;
#pragma unroll
        for (int k = 0; k < DP1; ++k) {
            if (!pend[k]) continue;
            if (old[k] == 0ull || old[k] == hkey[k]) {
                slot[k] = (int)h[k];
                created[k] = old[k] == 0ull;
                pend[k] = false;
            } else {
                h[k] = (h[k] + 1) & mask;
                any = true;
            }
        }
        if (!any) break;
    }
    // Each head reserves runlen places in its vertex's point list.
    int base[DP1];
#pragma unroll
    for (int k = 0; k < DP1; ++k)
        base[k] = (hkey[k] != 0ull && slot[k] >= 0) ? atomicAdd(&tab[slot[k]].count, runlen[k]) : 0;
    int rk[DP1];
#pragma unroll
    for (int k = 0; k < DP1; ++k) {
        const int sl = __shfl(slot[k], head[k], 64);
        const int bs = __shfl(base[k], head[k], 64);
        if (ok) {
            // the lane whose compare-and-swap claimed the slot marks its pair
            slot[k] = sl < 0 ? sl : (sl | (lane == head[k] && created[k] ? kCreator : 0));
            rk[k] = bs + lane - head[k];
            if (sl < 0) status |= ST_CAPACITY;
        } else {
            slot[k] = -1;
            rk[k] = -1;
        }
    }

    if (active) {
#pragma unroll
        for (int k = 0; k < DP1; ++k) {
            idx[p * DP1 + k] = slot[k];
            rank_out[p * DP1 + k] = rk[k];
            bary[p * DP1 + k] = status ? 0.f : b[k];
        }
    }
    if (status) atomicOr(counters + CNT_STATUS, status);
}

// Smallest power of two holding n keys at a load of at most 5/8.
constexpr int lds_table_slots(int n) {
    int s = 64;
    while (s * 5 < n * 8) s *= 2;
    return s;
}

// k_insert with workgroup-level dedup (for clouds whose points come in
// spatial order: the keys of NB consecutive points are merged first).
template <int D, int NB>
__global__ __launch_bounds__(NB) void k_insert_shared(const float *__restrict__ pos, const int32_t *__restrict__ batch,
                                                   int64_t m, ElevParams ep, HEntry *tab, uint32_t mask,
                                                   int32_t *__restrict__ idx, int32_t *__restrict__ rank_out,
                                                   float *__restrict__ bary, int32_t *counters) {
#pragma clang fp contract(off)
    constexpr int DP1 = D + 1;
    const int64_t p = (int64_t)blockIdx.x * NB + threadIdx.x;
    const bool active = p < m;

    uint64_t key[DP1];
    float b[DP1];
    int status = 0;
    point_keys<D>(pos, batch, p, active, ep, key, b, status);
    const bool ok = active && status == 0;

    // Workgroup-level dedup: the keys of the workgroup's points are first
    // merged in an LDS hash table (NS slots, load at most 5/8), where every
    // pair also takes its rank among the workgroup's pairs of that key.  One
    // pair per distinct key (the one that claimed the LDS slot) then claims
    // or finds the global slot and reserves all of the workgroup's places in
    // the vertex's pair list with one atomic add.  Points of a sensor sweep
    // come in spatial order, so a workgroup's points share most vertices.
    constexpr int NK = NB * DP1;
    constexpr int NS = lds_table_slots(NK);
    static_assert(NK * 8 <= NS * 5, "LDS table load");
    __shared__ unsigned long long lkey[NS];
    __shared__ int lcnt[NS];
    __shared__ int lslot[NS];
    __shared__ int lbase[NS];

    for (int i = threadIdx.x; i < NS; i += NB) {
        lkey[i] = 0ull;
        lcnt[i] = 0;
    }
    __syncthreads();

    int li[DP1], lr[DP1];
    bool lhead[DP1];
    {
        bool pend[DP1];
        uint32_t hs[DP1];
#pragma unroll
        for (int k = 0; k < DP1; ++k) {
            li[k] = -1;
            lhead[k] = false;
            pend[k] = ok;
            hs[k] = (uint32_t)key_mix(key[k]) & (NS - 1);
        }
        for (int probe = 0; probe < NS; ++probe) {
            bool any = false;
#pragma unroll
            for (int k = 0; k < DP1; ++k) {
                if (!pend[k]) continue;
                const unsigned long long old = atomicCAS(&lkey[hs[k]], 0ull, (unsigned long long)key[k]);
                if (old == 0ull || old == key[k]) {
                    li[k] = (int)hs[k];
                    lhead[k] = old == 0ull;
                    pend[k] = false;
                } else {
                    hs[k] = (hs[k] + 1) & (NS - 1);
                    any = true;
                }
            }
            if (!any) break;
        }
#pragma unroll
        for (int k = 0; k < DP1; ++k) lr[k] = li[k] >= 0 ? atomicAdd(&lcnt[li[k]], 1) : 0;
    }
    __syncthreads();

    // Distinct keys: claim or find the global slot; the d+1 probes of one
    // round are in flight together.
    {
        int slot[DP1];
        bool pend[DP1], created[DP1];
        uint32_t h[DP1];
#pragma unroll
        for (int k = 0; k < DP1; ++k) {
            slot[k] = -1;
            created[k] = false;
            pend[k] = lhead[k];
            h[k] = pend[k] ? home_slot(key[k], mask) : 0u;
        }
        for (uint32_t probe = 0; probe <= mask; ++probe) {
            unsigned long long old[DP1];
#pragma unroll
            for (int k = 0; k < DP1; ++k)
                if (pend[k]) old[k] = atomicCAS(&tab[h[k]].key, 0ull, (unsigned long long)key[k]);
            bool any = false;
#pragma unroll
            for (int k = 0; k < DP1; ++k) {
                if (!pend[k]) continue;
                if (old[k] == 0ull || old[k] == key[k]) {
                    slot[k] = (int)h[k];
                    created[k] = old[k] == 0ull;
                    pend[k] = false;
                } else {
                    h[k] = (h[k] + 1) & mask;
                    any = true;
                }
            }
            if (!any) break;
        }
#pragma unroll
        for (int k = 0; k < DP1; ++k) {
            if (!lhead[k]) continue;
            lslot[li[k]] = slot[k] < 0 ? -1 : (slot[k] | (created[k] ? kCreator : 0));
            lbase[li[k]] = slot[k] < 0 ? 0 : atomicAdd(&tab[slot[k]].count, lcnt[li[k]]);
        }
    }
    __syncthreads();

    if (active) {
#pragma unroll
        for (int k = 0; k < DP1; ++k) {
            int sl = -1, rk = -1;
            if (ok) {
                const int s = lslot[li[k]];
                // the creator flag stays with the pair that claimed the LDS slot
                sl = s < 0 ? -1 : (lhead[k] ? s : (s & (kCreator - 1)));
                rk = lbase[li[k]] + lr[k];
                if (s < 0) status |= ST_CAPACITY;
            }
            idx[p * DP1 + k] = sl;
            rank_out[p * DP1 + k] = rk;
            bary[p * DP1 + k] = status ? 0.f : b[k];
        }
    }
    if (status) atomicOr(counters + CNT_STATUS, status);
}

// Empty the hash table before a splat and zero the counters.  After a
// completed splat the occupied slots are exactly the vertices' slots (a slot
// is taken only by the pair that creates a vertex), listed in
// vslot[0 .. n), n = counters[CNT_SLOTS].  A scattered 16-byte store costs
// about a whole 128-byte line, so those n slots are emptied one by one when
// 8n < cap, and the whole table is written otherwise.  `whole` (the first
// splat, or one after a failed launch, when the table may hold keys vslot
// does not list) always writes the whole table and zeroes every counter;
// otherwise CNT_SLOTS, which every thread reads, is left for the next
// numbering to rewrite.
__global__ __launch_bounds__(kBlock) void k_clear_table(HEntry *tab, uint32_t *occ, int64_t cap,
                                                        const int32_t *__restrict__ vslot, int32_t *counters,
                                                        int whole) {
    const int64_t tid = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    uint4 *t4 = reinterpret_cast<uint4 *>(tab);
    const uint4 zero = make_uint4(0, 0, 0, 0);
    const int64_t n = whole ? cap : counters[CNT_SLOTS];
    if (whole || 8 * n >= cap) {
        for (int64_t i = tid; i < cap; i += stride) t4[i] = zero;
        for (int64_t i = tid; i < (cap + 31) / 32; i += stride) occ[i] = 0u;
    } else {
        // the listed slots and the occupancy words that hold their bits (only
        // listed slots have a bit set)
        for (int64_t i = tid; i < n; i += stride) {
            const int32_t sl = vslot[i];
            t4[sl] = zero;
            occ[sl >> 5] = 0u;
        }
    }
    if (blockIdx.x == 0 && threadIdx.x < CNT_WORDS && (whole || threadIdx.x != CNT_SLOTS)) counters[threadIdx.x] = 0;
}

// Vertex numbering and pair-list layout by a two-pass scan over the
// (point, remainder) pairs in point order, of the pairs that created their
// vertex: vertices are numbered in the order their first point appears, so
// that a spatially ordered cloud (a sensor sweep) gets spatially ordered
// vertices, and the scan reads the pair records instead of the (larger,
// mostly empty) hash table.  No same-address atomics.
//   k_scan_count   per block of `span` pairs, four sums over its creating
//                  pairs: vertices, their pairs, vertices whose pair list is
//                  longer than kPart ("split" vertices) and the part rows of
//                  those vertices
//   k_scan_assign  per block: its exclusive prefix (it sums the block sums
//                  before it), then, in pair order, every created vertex's
//                  index, key, pair-list offset and count; a split vertex
//                  also gets a split index and ceil(count / kPart) part rows
//                  (see k_gather).  The last block publishes the totals.
// A scan block covers `span` pairs, in chunks of kChunk (kPairsPerThread
// consecutive pairs per thread): span is kChunk, or a multiple of it when
// kChunk would make more than kMaxScanBlocks blocks (each block sums the
// block totals before it, a cost that grows with the square of their number:
// at 2 058 blocks, a four-frame sweep's 2.1 M pairs, two chunks per block
// made the assignment 15% faster; at 782 blocks one chunk stays faster).
constexpr int kPairsPerThread = 4;
constexpr int64_t kChunk = (int64_t)kBlock * kPairsPerThread;
constexpr int64_t kMaxScanBlocks = 1536;

__device__ __forceinline__ int wave_incl_scan(int x, int lane) {
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int y = __shfl_up(x, off, 64);
        if (lane >= off) x += y;
    }
    return x;
}

// The four scanned quantities of one hash entry.
__device__ __forceinline__ int4 entry_q(const HEntry &e) {
    const int cnt = e.count;
    const int parts = (cnt + kPart - 1) / kPart;
    return make_int4(1, cnt, parts > 1, parts > 1 ? parts : 0);
}

__device__ __forceinline__ int4 add4(int4 a, int4 b) { return make_int4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w); }

// Sum over the block (every thread gets the result).
__device__ __forceinline__ int4 block_sum4(int4 q, int4 *red) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        q.x += __shfl_xor(q.x, off, 64);
        q.y += __shfl_xor(q.y, off, 64);
        q.z += __shfl_xor(q.z, off, 64);
        q.w += __shfl_xor(q.w, off, 64);
    }
    if (lane == 0) red[wave] = q;
    __syncthreads();
    int4 t = red[0];
#pragma unroll
    for (int w = 1; w < kBlock / 64; ++w) t = add4(t, red[w]);
    __syncthreads();
    return t;
}

// The kPairsPerThread pair records of this thread in a chunk starting at
// c0 (n pairs in all): the slot of each pair that created its vertex, else -1.
__device__ __forceinline__ void load_creators(const int32_t *idx, int64_t c0, int64_t s1, int *slot) {
    const int64_t e0 = c0 + (int64_t)threadIdx.x * kPairsPerThread;
    int4 r = make_int4(-1, -1, -1, -1);
    if (e0 + kPairsPerThread <= s1) {
        r = *reinterpret_cast<const int4 *>(idx + e0);
    } else {
        if (e0 < s1) r.x = idx[e0];
        if (e0 + 1 < s1) r.y = idx[e0 + 1];
        if (e0 + 2 < s1) r.z = idx[e0 + 2];
    }
    const int v[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
    for (int i = 0; i < kPairsPerThread; ++i) slot[i] = (v[i] >= 0 && (v[i] & kCreator)) ? (v[i] & (kCreator - 1)) : -1;
}

__global__ __launch_bounds__(kBlock) void k_scan_count(const int32_t *__restrict__ idx, int64_t n, int64_t span,
                                                       const HEntry *__restrict__ tab, int4 *__restrict__ blk) {
    __shared__ int4 red[kBlock / 64];
    const int64_t s0 = (int64_t)blockIdx.x * span;
    const int64_t s1 = s0 + span < n ? s0 + span : n;
    int4 q = make_int4(0, 0, 0, 0);
    for (int64_t c0 = s0; c0 < s1; c0 += kChunk) {
        int sl[kPairsPerThread];
        load_creators(idx, c0, s1, sl);
#pragma unroll
        for (int i = 0; i < kPairsPerThread; ++i)
            if (sl[i] >= 0) q = add4(q, entry_q(tab[sl[i]]));
    }
    q = block_sum4(q, red);
    if (threadIdx.x == 0) blk[blockIdx.x] = q;
}

__global__ __launch_bounds__(kBlock) void k_scan_assign(const int32_t *__restrict__ idx, int64_t n, int64_t span,
                                                        int nb, HEntry *__restrict__ tab,
                                                        const int4 *__restrict__ blk, uint64_t *__restrict__ vkeys,
                                                        int32_t *__restrict__ vinfo, int32_t *__restrict__ split,
                                                        int32_t *__restrict__ rowmap, int2 *__restrict__ partrec,
                                                        int32_t *__restrict__ vslot,
                                                        uint32_t *occ, int32_t *counters) {
    __shared__ int4 red[kBlock / 64];
    __shared__ int4 wsum[kBlock / 64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t s0 = (int64_t)blockIdx.x * span;
    const int64_t s1 = s0 + span < n ? s0 + span : n;
    // exclusive prefix of the blocks before this one
    int4 carry = make_int4(0, 0, 0, 0);
    for (int b = threadIdx.x; b < (int)blockIdx.x; b += kBlock) carry = add4(carry, blk[b]);
    carry = block_sum4(carry, red);
    if ((int)blockIdx.x == nb - 1 && threadIdx.x == 0) {
        const int4 tot = add4(carry, blk[blockIdx.x]);
        counters[CNT_V] = tot.x;
        counters[CNT_SLOTS] = tot.x;
        counters[CNT_E] = tot.y;
        counters[CNT_SPLIT] = tot.z;
        counters[CNT_ROWS] = tot.w;
    }
    for (int64_t c0 = s0; c0 < s1; c0 += kChunk) {
        int sl[kPairsPerThread];
        load_creators(idx, c0, s1, sl);
        HEntry e[kPairsPerThread];
        int4 q[kPairsPerThread];
        int4 mine = make_int4(0, 0, 0, 0);
#pragma unroll
        for (int i = 0; i < kPairsPerThread; ++i) {
            q[i] = make_int4(0, 0, 0, 0);
            if (sl[i] >= 0) {
                e[i] = tab[sl[i]];
                q[i] = entry_q(e[i]);
            }
            mine = add4(mine, q[i]);
        }
        int4 inc;
        inc.x = wave_incl_scan(mine.x, lane);
        inc.y = wave_incl_scan(mine.y, lane);
        inc.z = wave_incl_scan(mine.z, lane);
        inc.w = wave_incl_scan(mine.w, lane);
        if (lane == 63) wsum[wave] = inc;
        __syncthreads();
        // exclusive prefix of this thread's first pair
        int4 at = carry;
        int4 chunk = make_int4(0, 0, 0, 0);
#pragma unroll
        for (int w = 0; w < kBlock / 64; ++w) {
            if (w < wave) at = add4(at, wsum[w]);
            chunk = add4(chunk, wsum[w]);
        }
        at = make_int4(at.x + inc.x - mine.x, at.y + inc.y - mine.y, at.z + inc.z - mine.z, at.w + inc.w - mine.w);
#pragma unroll
        for (int i = 0; i < kPairsPerThread; ++i) {
            if (q[i].x) {
                const int v = at.x;
                // the list offset replaces the count (read above; vinfo keeps
                // it), so the fill finds both in one load of the entry
                *reinterpret_cast<int2 *>(&tab[sl[i]].count) = make_int2(at.y, v);
                vslot[v] = sl[i];
                mark_taken(occ, sl[i]);
                vkeys[v] = e[i].key;
                vinfo[2 * v] = at.y;
                vinfo[2 * v + 1] = q[i].y;
                if (q[i].z) {
                    const int sp = at.z, row0 = at.w;
                    split[3 * sp] = v;
                    split[3 * sp + 1] = row0;
                    split[3 * sp + 2] = q[i].w;
                    for (int j = 0; j < q[i].w; ++j) {
                        rowmap[row0 + j] = sp;
                        const int left = q[i].y - j * kPart;
                        partrec[row0 + j] = make_int2(at.y + j * kPart, left < kPart ? left : kPart);
                    }
                }
            }
            at = add4(at, q[i]);
        }
        carry = add4(carry, chunk);
        __syncthreads();  // wsum is rewritten by the next chunk
    }
}

// Per pair (p, k): map the hash slot to the vertex index (rewriting the
// per-point record in place) and place (p, b_pk) at its rank in the vertex's
// pair list.
template <int D>
__global__ __launch_bounds__(kBlock) void k_fill(int64_t n, int32_t *__restrict__ idx, const int32_t *__restrict__ rank,
                                                 const float *__restrict__ bary, const HEntry *__restrict__ tab,
                                                 int32_t *__restrict__ list) {
    constexpr int DP1 = D + 1;
    constexpr int U = 2;  // pairs per thread whose loads are in flight together
    int64_t lo, hi;
    block_chunk(n, kBlock, lo, hi);
    for (int64_t e0 = lo + threadIdx.x; e0 < hi; e0 += U * kBlock) {
        int s[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t e = e0 + u * kBlock;
            s[u] = e < hi ? idx[e] : -1;
        }
        int2 ov[U];
        int r[U];
        float b[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t e = e0 + u * kBlock;
            if (s[u] >= 0) {
                ov[u] = *reinterpret_cast<const int2 *>(&tab[s[u] & (kCreator - 1)].count);  // (list offset, vertex)
                r[u] = rank[e];
                b[u] = bary[e];
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t e = e0 + u * kBlock;
            if (s[u] >= 0) {
                idx[e] = ov[u].y;
                const int64_t at = (int64_t)ov[u].x + r[u];
                const int64_t pt = e / DP1;
                *reinterpret_cast<int2 *>(list + 2 * at) =
                    make_int2(list_entry(pt, (int)(e - pt * DP1)), __float_as_int(b[u]));
            }
        }
    }
}

// Store 4 (VEC) or 1 value of a vertex row as fp32 or bf16 (nearest even).
template <bool OUT_BF16>
__device__ __forceinline__ void store4(void *values, int64_t at4, float4 a) {
    if (OUT_BF16) {
        uint2 pk;
        pk.x = bf16_bits(a.x) | (bf16_bits(a.y) << 16);
        pk.y = bf16_bits(a.z) | (bf16_bits(a.w) << 16);
        reinterpret_cast<uint2 *>(values)[at4] = pk;
    } else {
        reinterpret_cast<float4 *>(values)[at4] = a;
    }
}
template <bool OUT_BF16>
__device__ __forceinline__ void store1(void *values, int64_t at, float a) {
    if (OUT_BF16)
        reinterpret_cast<uint16_t *>(values)[at] = (uint16_t)bf16_bits(a);
    else
        reinterpret_cast<float *>(values)[at] = a;
}

__device__ __forceinline__ float4 fma4(float b, float4 y, float4 acc) {
    acc.x = fmaf(b, y.x, acc.x);
    acc.y = fmaf(b, y.y, acc.y);
    acc.z = fmaf(b, y.z, acc.z);
    acc.w = fmaf(b, y.w, acc.w);
    return acc;
}

// One block of BLK list entries q (the first n of them real) for float4
// column c (VEC) or column c: their rows are loaded together, then b f and b
// are added for the real ones.  Selects, not branches: a branch would let
// the compiler sink the loads into it and serialise them.
template <bool VEC, int BLK>
__device__ __forceinline__ void add_block(const int2 (&q)[BLK], int n, const float *__restrict__ feat, int CV, int c,
                                          float4 &acc, float &w) {
    if (VEC) {
        const float4 *f4 = reinterpret_cast<const float4 *>(feat);
        float4 y[BLK];
#pragma unroll
        for (int i = 0; i < BLK; ++i) y[i] = f4[(int64_t)list_point(q[i].x) * CV + c];
#pragma unroll
        for (int i = 0; i < BLK; ++i) {
            const bool ok = i < n;
            const float b = ok ? __int_as_float(q[i].y) : 0.f;
            const float4 t = fma4(b, y[i], acc);
            acc.x = ok ? t.x : acc.x;
            acc.y = ok ? t.y : acc.y;
            acc.z = ok ? t.z : acc.z;
            acc.w = ok ? t.w : acc.w;
            w += b;
        }
    } else {
        float y[BLK];
#pragma unroll
        for (int i = 0; i < BLK; ++i) y[i] = CV > 0 ? feat[(int64_t)list_point(q[i].x) * CV + c] : 0.f;
#pragma unroll
        for (int i = 0; i < BLK; ++i) {
            const bool ok = i < n;
            const float b = ok ? __int_as_float(q[i].y) : 0.f;
            const float t = fmaf(b, y[i], acc.x);
            acc.x = ok ? t : acc.x;
            w += b;
        }
    }
}

// The list entries [e, e + BLK) clamped to [.., e1): indices past e1 re-read
// entry e1 - 1 (and are not added).
template <int BLK>
__device__ __forceinline__ void load_block(const int2 *__restrict__ L2, int e, int e1, int2 (&q)[BLK]) {
#pragma unroll
    for (int i = 0; i < BLK; ++i) q[i] = L2[e + i < e1 ? e + i : e1 - 1];
}

// Sum b f over list entries [e0, e1) for float4 column c (VEC) or column c,
// added to acc, and the weights b added to w, in blocks of BLK entries: a
// block's list loads are all issued, then its row loads, before any is used.
template <bool VEC, int BLK>
__device__ __forceinline__ void sum_pairs(const int2 *__restrict__ L2, int e0, int e1, const float *__restrict__ feat,
                                          int CV, int c, float4 &acc, float &w) {
    for (int e = e0; e < e1; e += BLK) {
        int2 q[BLK];
        load_block<BLK>(L2, e, e1, q);
        add_block<VEC, BLK>(q, e1 - e, feat, CV, c, acc, w);
    }
}

// The same, with the next block's list loads issued together with this
// block's row loads (one round trip per block instead of two; for the
// 32-entry parts of long lists).
template <bool VEC, int BLK>
__device__ __forceinline__ void sum_pairs_ahead(const int2 *__restrict__ L2, int e0, int e1,
                                                const float *__restrict__ feat, int CV, int c, float4 &acc,
                                                float &w) {
    if (e0 >= e1) return;
    int2 q[BLK];
    load_block<BLK>(L2, e0, e1, q);
    for (int e = e0; e < e1; e += BLK) {
        int2 qn[BLK];
        load_block<BLK>(L2, e + BLK, e1, qn);  // past e1: re-reads entry e1 - 1, unused
        add_block<VEC, BLK>(q, e1 - e, feat, CV, c, acc, w);
#pragma unroll
        for (int i = 0; i < BLK; ++i) q[i] = qn[i];
    }
}

// Short lists (at most kPart pairs) for float4 columns, one column per lane
// of a group of G = 2^LG lanes (G >= CV; a lane past the last column reads
// column CV - 1 and stores nothing).  The group's lanes load a list's entries
// together, entry t by lane t mod G into its register t / G: one round trip
// for the whole list, issued a list ahead of its rows.  The rows are then
// loaded kRowBlk at a time (none past the list's end), each entry handed to
// the group by a lane shuffle, and added in list order (the order sum_pairs
// adds them in).
constexpr int kRowBlk = 8;

template <int LG>
struct ListRegs {
    static constexpr int NE = (kPart + (1 << LG) - 1) >> LG;
    int x[NE], y[NE];
};

// The entries [e0, e0 + n) of a list; n outside [1, kPart] (no list to add)
// loads entry 0, which exists whenever a list is read.
template <int LG>
__device__ __forceinline__ void load_list(const int2 *__restrict__ L2, int e0, int n, int j, ListRegs<LG> &q) {
    const bool ok = n >= 1 && n <= kPart;
#pragma unroll
    for (int r = 0; r < ListRegs<LG>::NE; ++r) {
        const int t = (r << LG) + j;
        const int2 e = L2[ok ? e0 + (t < n ? t : n - 1) : 0];  // past n: entry n - 1 again, not added
        q.x[r] = e.x;
        q.y[r] = e.y;
    }
}

template <int LG>
__device__ __forceinline__ void sum_rows(const ListRegs<LG> &q, int n, const float4 *__restrict__ f4, int CV, int cc,
                                         int gbase, float4 &acc, float &w) {
    constexpr int G = 1 << LG;
#pragma unroll
    for (int t0 = 0; t0 < kPart; t0 += kRowBlk) {
        if (t0 >= n) break;
        float4 y[kRowBlk];
        float b[kRowBlk];
#pragma unroll
        for (int i = 0; i < kRowBlk; ++i) {
            const int t = t0 + i;
            const int src = gbase + (t & (G - 1));
            const int pt = list_point(__shfl(q.x[t >> LG], src, 64));
            b[i] = __int_as_float(__shfl(q.y[t >> LG], src, 64));
            y[i] = make_float4(0.f, 0.f, 0.f, 0.f);
            if (t < n) y[i] = f4[(int64_t)pt * CV + cc];  // rows past n are not loaded
        }
#pragma unroll
        for (int i = 0; i < kRowBlk; ++i) {
            const bool ok = t0 + i < n;
            const float bb = ok ? b[i] : 0.f;
            const float4 t = fma4(bb, y[i], acc);
            acc.x = ok ? t.x : acc.x;
            acc.y = ok ? t.y : acc.y;
            acc.z = ok ? t.z : acc.z;
            acc.w = ok ? t.w : acc.w;
            w += bb;
        }
    }
}

template <bool VEC>
__device__ __forceinline__ float4 scale4(float4 a, float w, int normalize) {
    if (!normalize) return a;
    a.x = w != 0.f ? a.x / w : 0.f;
    if (VEC) {
        a.y = w != 0.f ? a.y / w : 0.f;
        a.z = w != 0.f ? a.z / w : 0.f;
        a.w = w != 0.f ? a.w / w : 0.f;
    }
    return a;
}

// Eq. (splat), pulled per vertex: x_v = sum over the vertex's pair list of
// b_pv f_p, and w_v = sum b_pv.  Work units are groups of G lanes, each lane
// owning float4 (VEC) or single column chunks.  Two kernels:
//   k_gather_parts  a list longer than kPart pairs is cut into parts of kPart
//                   pairs, one unit each, so that dense regions (thousands of
//                   points on one vertex near a LiDAR sensor) do not
//                   serialise on one group; a part writes its partial row
//                   (and partial weight) to scratch.
//   k_gather        a vertex with at most kPart pairs is one unit: its row is
//                   summed and written once (no zero fill, no float atomics);
//                   then the split vertices: their parts added in part order.
// (Combining in the last part to finish would need a device-scope release
// per part, which costs more than a launch: every XCD has its own L2.)
template <bool VEC, int LG>
__global__ __launch_bounds__(kBlock) void k_gather_parts(const int32_t *__restrict__ vinfo,
                                                         const int32_t *__restrict__ list,
                                                         const int32_t *__restrict__ split,
                                                         const int32_t *__restrict__ rowmap,
                                                         const int2 *__restrict__ partrec,
                                                         float *__restrict__ partial, float *__restrict__ pweight,
                                                         const float *__restrict__ feat, int C, int log2G,
                                                         const int32_t *counters) {
    const int64_t nrows = counters[CNT_ROWS];
    const int G = 1 << log2G;
    const int lane = threadIdx.x & 63;
    const int grp = lane >> log2G;
    const int j = lane & (G - 1);
    const int gpw = 64 >> log2G;  // groups per wave
    const int CV = VEC ? (C >> 2) : C;
    const int2 *L2 = reinterpret_cast<const int2 *>(list);
    // each XCD takes one contiguous range of parts (vertices in creation
    // order): the point rows they share meet in its L2
    const XcdShare sh = xcd_share(nrows);
    if constexpr (LG > 0) {
        // the part's record and list a step ahead of its rows
        const int gbase = lane & ~(G - 1);
        const int cc = j < CV ? j : CV - 1;
        const int64_t ustep = sh.nwaves * gpw;
        auto rec = [&](int64_t u) { return u < sh.hi ? partrec[u] : make_int2(0, 0); };
        int64_t u = sh.lo + sh.wave * gpw + grp;
        int2 r = rec(u);
        ListRegs<LG> q;
        load_list<LG>(L2, r.x, r.y, j, q);
        int2 rn = rec(u + ustep);
        for (; u - grp < sh.hi; u += ustep) {
            ListRegs<LG> qn;
            load_list<LG>(L2, rn.x, rn.y, j, qn);
            const int2 rnn = rec(u + 2 * ustep);
            if (u < sh.hi) {
                float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
                float w = 0.f;
                sum_rows<LG>(q, r.y, reinterpret_cast<const float4 *>(feat), CV, cc, gbase, acc, w);
                if (j < CV) reinterpret_cast<float4 *>(partial)[u * CV + j] = acc;
                if (j == 0) pweight[u] = w;
            }
            q = qn;
            r = rn;
            rn = rnn;
        }
        return;
    }
    for (int64_t u0 = sh.lo + sh.wave * gpw; u0 < sh.hi; u0 += sh.nwaves * gpw) {
        const int64_t u = u0 + grp;
        if (u >= sh.hi) continue;
        const int sp = rowmap[u];
        const int vv = split[3 * sp];
        const int row0 = split[3 * sp + 1];
        const int off = vinfo[2 * vv];
        const int cnt = vinfo[2 * vv + 1];
        const int part = (int)(u - row0);
        const int e0 = off + part * kPart;
        const int e1 = e0 + kPart < off + cnt ? e0 + kPart : off + cnt;
        float w = 0.f;
        for (int c = j; c < CV; c += G) {
            float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
            w = 0.f;
            sum_pairs_ahead<VEC, 4>(L2, e0, e1, feat, CV, c, acc, w);
            if (VEC)
                reinterpret_cast<float4 *>(partial)[u * CV + c] = acc;
            else
                partial[u * C + c] = acc.x;
        }
        if (j == 0) {
            if (CV == 0) {
                float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
                sum_pairs<false, 4>(L2, e0, e1, feat, 0, 0, acc, w);
            }
            pweight[u] = w;
        }
    }
}

template <bool VEC, bool OUT_BF16, int LG>
__global__ __launch_bounds__(kBlock) void k_gather(const int32_t *__restrict__ vinfo, const int32_t *__restrict__ list,
                                                   const int32_t *__restrict__ split, const float *__restrict__ partial,
                                                   const float *__restrict__ pweight, const float *__restrict__ feat,
                                                   int C, int log2G, int normalize, void *__restrict__ values,
                                                   float *__restrict__ weight, const int32_t *counters) {
    const int64_t V = counters[CNT_V];
    const int64_t ns = counters[CNT_SPLIT];
    const int G = 1 << log2G;
    const int lane = threadIdx.x & 63;
    const int grp = lane >> log2G;
    const int j = lane & (G - 1);
    const int gpw = 64 >> log2G;  // groups per wave
    const int CV = VEC ? (C >> 2) : C;
    const int2 *L2 = reinterpret_cast<const int2 *>(list);

    // Short lists, each XCD one contiguous range of vertices (in creation
    // order, so the point rows they share meet in its L2).  The list header
    // of the group's next vertex is loaded while this one is summed (two
    // header registers, so that the wait for one header is not a wait for
    // the other).  With C = 0 (weights only) lane 0 of the group sums the
    // weights alone.
    const int2 *VI = reinterpret_cast<const int2 *>(vinfo);
    const XcdShare sh = xcd_share(V);
    const int64_t vstep = sh.nwaves * gpw;
    auto header = [&](int64_t v) { return v < sh.hi ? VI[v] : make_int2(0, kPart + 1); };
    auto short_list = [&](int64_t v, int2 vi) {
        if (v >= sh.hi || vi.y > kPart) return;
        const int off = vi.x, e1 = vi.x + vi.y;
        float w = 0.f;
        for (int c = j; c < CV; c += G) {
            float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
            w = 0.f;
            sum_pairs<VEC, 4>(L2, off, e1, feat, CV, c, acc, w);
            acc = scale4<VEC>(acc, w, normalize);
            if (VEC)
                store4<OUT_BF16>(values, v * CV + c, acc);
            else
                store1<OUT_BF16>(values, v * C + c, acc.x);
        }
        if (weight && j == 0) {
            if (CV == 0) {
                float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
                sum_pairs<false, 4>(L2, off, e1, feat, 0, 0, acc, w);
            }
            weight[v] = w;
        }
    };
    if constexpr (LG > 0) {
        // the next vertex's list loaded while this one's rows are
        const int gbase = lane & ~(G - 1);
        const int cc = j < CV ? j : CV - 1;
        int64_t v = sh.lo + sh.wave * gpw + grp;
        int2 h = header(v);
        ListRegs<LG> q;
        load_list<LG>(L2, h.x, h.y, j, q);
        int2 hn = header(v + vstep);
        for (; v - grp < sh.hi; v += vstep) {
            ListRegs<LG> qn;
            load_list<LG>(L2, hn.x, hn.y, j, qn);
            const int2 hnn = header(v + 2 * vstep);
            if (v < sh.hi && h.y <= kPart) {
                float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
                float w = 0.f;
                sum_rows<LG>(q, h.y, reinterpret_cast<const float4 *>(feat), CV, cc, gbase, acc, w);
                acc = scale4<true>(acc, w, normalize);
                if (j < CV) store4<OUT_BF16>(values, v * CV + j, acc);
                if (weight && j == 0) weight[v] = w;
            }
            q = qn;
            h = hn;
            hn = hnn;
        }
    } else {
        int64_t v = sh.lo + sh.wave * gpw + grp;
        int2 ha = header(v);
        for (; v - grp < sh.hi; v += 2 * vstep) {
            const int2 hb = header(v + vstep);
            short_list(v, ha);
            if (v - grp + vstep >= sh.hi) break;
            ha = header(v + 2 * vstep);
            short_list(v + vstep, hb);
        }
    }

    // Split vertices: the part rows added in part order, four per block
    // with all loads of a block in flight (a list of thousands of pairs has
    // dozens of parts); rows past the last part re-read it and are not
    // added.  Then scaled and stored like a short list's row.
    constexpr int kB = 4;
    const XcdShare ss = xcd_share(ns);
    for (int64_t s0 = ss.lo + ss.wave * gpw; s0 < ss.hi; s0 += ss.nwaves * gpw) {
        const int64_t sp = s0 + grp;
        if (sp >= ss.hi) continue;
        const int v = split[3 * sp], row0 = split[3 * sp + 1], parts = split[3 * sp + 2];
        const int rlast = row0 + parts - 1;
        float w = 0.f;
        for (int r0 = 0; r0 < parts; r0 += kB) {
            float pw[kB];
#pragma unroll
            for (int i = 0; i < kB; ++i) pw[i] = pweight[row0 + r0 + i < rlast ? row0 + r0 + i : rlast];
#pragma unroll
            for (int i = 0; i < kB; ++i) w += r0 + i < parts ? pw[i] : 0.f;
        }
        for (int c = j; c < CV; c += G) {
            float4 t = make_float4(0.f, 0.f, 0.f, 0.f);
            for (int r0 = 0; r0 < parts; r0 += kB) {
                float4 a[kB];
#pragma unroll
                for (int i = 0; i < kB; ++i) {
                    const int64_t row = row0 + r0 + i < rlast ? row0 + r0 + i : rlast;
                    if (VEC)
                        a[i] = reinterpret_cast<const float4 *>(partial)[row * CV + c];
                    else
                        a[i] = make_float4(partial[row * C + c], 0.f, 0.f, 0.f);
                }
#pragma unroll
                for (int i = 0; i < kB; ++i) {
                    const bool ok = r0 + i < parts;
                    t.x += ok ? a[i].x : 0.f;
                    t.y += ok ? a[i].y : 0.f;
                    t.z += ok ? a[i].z : 0.f;
                    t.w += ok ? a[i].w : 0.f;
                }
            }
            t = scale4<VEC>(t, w, normalize);
            if (VEC)
                store4<OUT_BF16>(values, (int64_t)v * CV + c, t);
            else
                store1<OUT_BF16>(values, (int64_t)v * C + c, t.x);
        }
        if (weight && j == 0) weight[v] = w;
    }
}

template <int D>
__global__ __launch_bounds__(kBlock) void k_export_keys(const uint64_t *__restrict__ vkeys, const int32_t *counters,
                                                        int32_t *keys, int32_t *batch) {
    const int64_t V = counters[CNT_V];
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t v = (int64_t)blockIdx.x * kBlock + threadIdx.x; v < V; v += stride) {
        int c[D];
        uint32_t b;
        unpack_key<D>(vkeys[v], c, b);
        int s = 0;
#pragma unroll
        for (int i = 0; i < D; ++i) {
            keys[v * (D + 1) + i] = c[i];
            s += c[i];
        }
        keys[v * (D + 1) + D] = -s;
        if (batch) batch[v] = (int32_t)b;
    }
}

// fp32 -> bf16, round to nearest with ties to even; NaN stays a quiet NaN.
__global__ __launch_bounds__(kBlock) void k_to_bf16(const float *__restrict__ src, int64_t n, uint16_t *__restrict__ dst) {
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += stride) {
        dst[i] = (uint16_t)bf16_bits(src[i]);
    }
}

template <typename F>
hipError_t dispatch_d(int d, F &&f) {
    switch (d) {
        case 1: return f(std::integral_constant<int, 1>{});
        case 2: return f(std::integral_constant<int, 2>{});
        case 3: return f(std::integral_constant<int, 3>{});
        case 4: return f(std::integral_constant<int, 4>{});
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_clear_table(lattice *L) {
    const unsigned grid = grid_for(L->cap, kBlock, L->cu_count, 4);
    hipLaunchKernelGGL(k_clear_table, dim3(grid), dim3(kBlock), 0, L->stream, L->tab, L->occ, L->cap, L->vslot,
                       L->counters, L->full_clear ? 1 : 0);
    return hipGetLastError();
}

hipError_t launch_insert(lattice *L, const float *pos, const int32_t *batch, int64_t m) {
    if (m == 0) return hipSuccess;
    ElevParams ep;
    for (int i = 0; i < LATTICE_MAX_D; ++i) ep.f[i] = L->factors[i];
    ep.inv = L->inv_dp1;
    const uint32_t mask = (uint32_t)(L->cap - 1);
    // Large clouds: 256 points per workgroup merged in LDS before the global
    // table (sensor sweeps share most vertices between consecutive points;
    // measured 2.5x fewer cycles on a 4-frame sweep, a few percent more on a
    // shuffled cloud).  Small clouds: one wavefront per workgroup, so that
    // they still spread over every CU.
    const bool shared = m >= (int64_t)256 * L->cu_count;
    return dispatch_d(L->d, [&](auto dc) {
        constexpr int D = decltype(dc)::value;
        if (shared)
            hipLaunchKernelGGL((k_insert_shared<D, 256>), dim3((unsigned)((m + 255) / 256)), dim3(256), 0, L->stream,
                               pos, batch, m, ep, L->tab, mask, L->idx, L->rank, L->bary, L->counters);
        else
            hipLaunchKernelGGL(k_insert<D>, dim3((unsigned)((m + kInsertBlock - 1) / kInsertBlock)),
                               dim3(kInsertBlock), 0, L->stream, pos, batch, m, ep, L->tab, mask, L->idx, L->rank,
                               L->bary, L->counters);
        return hipGetLastError();
    });
}

static int64_t scan_span(int64_t n) {
    const int64_t per = (n + kMaxScanBlocks - 1) / kMaxScanBlocks;
    return per > kChunk ? (per + kChunk - 1) / kChunk * kChunk : kChunk;
}

int64_t scan_blocks_max() { return kMaxScanBlocks; }

hipError_t launch_number(lattice *L, int64_t m) {
    const int64_t n = m * (L->d + 1);
    if (n == 0) return hipSuccess;  // no vertices: the counters stay cleared
    const int64_t span = scan_span(n);
    const int64_t nb = (n + span - 1) / span;
    int4 *blk = reinterpret_cast<int4 *>(L->blk);
    hipLaunchKernelGGL(k_scan_count, dim3((unsigned)nb), dim3(kBlock), 0, L->stream, L->idx, n, span, L->tab, blk);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_scan_assign, dim3((unsigned)nb), dim3(kBlock), 0, L->stream, L->idx, n, span, (int)nb,
                       L->tab, blk, L->vkeys, L->vinfo, L->split, L->rowmap, reinterpret_cast<int2 *>(L->partrec),
                       L->vslot, L->occ, L->counters);
    return hipGetLastError();
}

// Bound on the part rows of one splat: a split list has cnt > kPart pairs and
// ceil(cnt / kPart) < 2 cnt / kPart parts, and the lists hold at most
// (d+1) m pairs.  The number of split vertices is below that too.
int64_t split_rows_max(const lattice *L) { return 2 * (L->d + 1) * L->max_points / kPart + 1; }

hipError_t launch_fill(lattice *L, int64_t m) {
    if (m == 0) return hipSuccess;
    const int64_t n = m * (L->d + 1);
    const unsigned grid = grid_for(n, kBlock, L->cu_count, 16);
    return dispatch_d(L->d, [&](auto dc) {
        constexpr int D = decltype(dc)::value;
        hipLaunchKernelGGL(k_fill<D>, dim3(grid), dim3(kBlock), 0, L->stream, n, L->idx, L->rank, L->bary, L->tab,
                           L->list);
        return hipGetLastError();
    });
}

template <bool OUT_BF16>
static hipError_t gather_typed(lattice *L, const float *feat, int C, int normalize, void *values, float *weight) {
    const bool vec = C > 0 && (C % 4 == 0) && ((reinterpret_cast<uintptr_t>(feat) & 15) == 0) &&
                     ((reinterpret_cast<uintptr_t>(values) & (OUT_BF16 ? 7 : 15)) == 0);
    const int lanes = vec ? C / 4 : (C > 0 ? C : 1);
    int log2G = 0;
    while ((1 << log2G) < lanes && log2G < 6) ++log2G;
    const int64_t gpw = 64 >> log2G;
    // the parts of long lists first: the second kernel adds them
    const unsigned g1 = grid_for((split_rows_max(L) + gpw - 1) / gpw * 64, kBlock, L->cu_count, 16);
    const int64_t waves = (L->max_vertices + gpw - 1) / gpw;
    const unsigned grid = grid_for(waves * 64, kBlock, L->cu_count, 16);
    // float4 columns, one per lane of a group of 4 to 64 lanes: the lists
    // are loaded by the group together
    auto launch = [&](auto vc, auto lc) -> hipError_t {
        constexpr bool VEC = decltype(vc)::value;
        constexpr int LG = decltype(lc)::value;
        hipLaunchKernelGGL((k_gather_parts<VEC, LG>), dim3(g1), dim3(kBlock), 0, L->stream, L->vinfo, L->list,
                           L->split, L->rowmap, reinterpret_cast<const int2 *>(L->partrec), L->partial, L->pweight,
                           feat, C, log2G, L->counters);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL((k_gather<VEC, OUT_BF16, LG>), dim3(grid), dim3(kBlock), 0, L->stream, L->vinfo, L->list,
                           L->split, L->partial, L->pweight, feat, C, log2G, normalize, values, weight, L->counters);
        return hipGetLastError();
    };
    using T = std::true_type;
    using F = std::false_type;
    if (!vec) return launch(F{}, std::integral_constant<int, 0>{});
    switch (lanes <= 64 ? log2G : 0) {
        case 2: return launch(T{}, std::integral_constant<int, 2>{});
        case 3: return launch(T{}, std::integral_constant<int, 3>{});
        case 4: return launch(T{}, std::integral_constant<int, 4>{});
        case 5: return launch(T{}, std::integral_constant<int, 5>{});
        case 6: return launch(T{}, std::integral_constant<int, 6>{});
        default: return launch(T{}, std::integral_constant<int, 0>{});
    }
}

hipError_t launch_gather(lattice *L, const float *feat, int C, int normalize, void *values, lattice_dtype values_dt,
                         float *weight) {
    return values_dt == LATTICE_BF16 ? gather_typed<true>(L, feat, C, normalize, values, weight)
                                     : gather_typed<false>(L, feat, C, normalize, values, weight);
}

hipError_t launch_export_keys(lattice *L, int32_t *keys, int32_t *batch) {
    const unsigned grid = grid_for(L->max_vertices, kBlock, L->cu_count, 4);
    return dispatch_d(L->d, [&](auto dc) {
        constexpr int D = decltype(dc)::value;
        hipLaunchKernelGGL(k_export_keys<D>, dim3(grid), dim3(kBlock), 0, L->stream, L->vkeys, L->counters, keys,
                           batch);
        return hipGetLastError();
    });
}

hipError_t launch_to_bf16(lattice *L, const float *src, int64_t n, uint16_t *dst) {
    if (n == 0) return hipSuccess;
    const unsigned grid = grid_for(n, kBlock, L->cu_count, 4);
    hipLaunchKernelGGL(k_to_bf16, dim3(grid), dim3(kBlock), 0, L->stream, src, n, dst);
    return hipGetLastError();
}
