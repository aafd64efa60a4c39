// Splat: elevation onto H_d, enclosing simplex, barycentric weights, hash
// insertion of the d+1 vertex keys (Sec. "Permutohedral Lattice"), and the
// barycentric accumulation of Eq. (splat).
//
// Kernel sequence of one lattice_splat (all on the lattice's stream):
//   k_clear_table   empty the hash table, zero V, the pair count and the status
//   k_insert        one thread per point: elevate, round, rank, wrap, weights,
//                   keys; CAS-insert of the d+1 keys (runs of equal keys in
//                   neighbouring lanes are inserted once), a rank for every
//                   (point, vertex) pair from the slot's counter
//   k_scan_*        vertex indices and pair-list ranges in hash-slot order
//   k_fill          per pair: slot -> vertex index, (p, b_pk) into the list
//   k_gather        per vertex: x_v = sum b_pv f_p and w_v = sum b_pv
//                   (optionally x_v / w_v), each row written once; vertices
//                   with many pairs by k_gather_heavy, a workgroup each
#include "internal.h"
#include "keys.h"

namespace {

constexpr int kBlock = 256;

// fp32 -> bf16 bits, round to nearest with ties to even (NaN stays a quiet NaN).
__device__ __forceinline__ uint32_t bf16_bits(float f) {
    const uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
    return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

// Vertices with more pairs than this are reduced by a whole workgroup.
constexpr int kHeavy = 64;

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
#pragma unroll
    for (int k = 0; k < DP1; ++k) {
        key[k] = 0;
        b[k] = 0.f;
    }
    int status = 0;

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
    bool pend[DP1];
    uint32_t h[DP1];
#pragma unroll
    for (int k = 0; k < DP1; ++k) {
        slot[k] = -1;
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
            slot[k] = sl;
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

__global__ __launch_bounds__(kBlock) void k_clear_table(HEntry *tab, int64_t cap, int32_t *counters) {
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    uint4 *t4 = reinterpret_cast<uint4 *>(tab);
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < cap; i += stride) t4[i] = make_uint4(0, 0, 0, 0);
    if (blockIdx.x == 0 && threadIdx.x < CNT_WORDS) counters[threadIdx.x] = 0;
}

// Vertex numbering and pair-list layout, in hash-slot order, by a three-phase
// scan over the table (no same-address atomics):
//   k_scan_count   per block of kScanSlots slots: occupied slots and pairs
//   k_scan_blocks  one workgroup: exclusive prefix of the block sums; V and
//                  the pair total
//   k_scan_assign  per block, in slot order: vertex index, list offset and
//                  count of every occupied slot; vertices with more than
//                  kHeavy pairs are also listed for the workgroup-per-vertex
//                  gather.
constexpr int kScanSlots = 2048;

__device__ __forceinline__ int wave_incl_scan(int x, int lane) {
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int y = __shfl_up(x, off, 64);
        if (lane >= off) x += y;
    }
    return x;
}

__global__ __launch_bounds__(kBlock) void k_scan_count(const HEntry *__restrict__ tab, int64_t cap,
                                                       int32_t *__restrict__ blk) {
    __shared__ int red[2][kBlock / 64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t s0 = (int64_t)blockIdx.x * kScanSlots;
    const int64_t s1 = s0 + kScanSlots < cap ? s0 + kScanSlots : cap;
    int occ = 0, cnt = 0;
    for (int64_t s = s0 + threadIdx.x; s < s1; s += kBlock) {
        const HEntry e = tab[s];
        occ += e.key != 0ull;
        cnt += e.count;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        occ += __shfl_xor(occ, off, 64);
        cnt += __shfl_xor(cnt, off, 64);
    }
    if (lane == 0) {
        red[0][wave] = occ;
        red[1][wave] = cnt;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        int o = 0, c = 0;
        for (int w = 0; w < kBlock / 64; ++w) {
            o += red[0][w];
            c += red[1][w];
        }
        blk[2 * blockIdx.x] = o;
        blk[2 * blockIdx.x + 1] = c;
    }
}

__global__ __launch_bounds__(1024) void k_scan_blocks(int32_t *__restrict__ blk, int nb, int32_t *counters) {
    __shared__ int wsum[2][16];
    __shared__ int carry[2];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (threadIdx.x == 0) carry[0] = carry[1] = 0;
    __syncthreads();
    for (int b0 = 0; b0 < nb; b0 += 1024) {
        const int b = b0 + threadIdx.x;
        const int o = b < nb ? blk[2 * b] : 0;
        const int c = b < nb ? blk[2 * b + 1] : 0;
        const int io = wave_incl_scan(o, lane);
        const int ic = wave_incl_scan(c, lane);
        if (lane == 63) {
            wsum[0][wave] = io;
            wsum[1][wave] = ic;
        }
        __syncthreads();
        int bo = carry[0], bc = carry[1];
        for (int w = 0; w < wave; ++w) {
            bo += wsum[0][w];
            bc += wsum[1][w];
        }
        if (b < nb) {
            blk[2 * b] = bo + io - o;
            blk[2 * b + 1] = bc + ic - c;
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            for (int w = 0; w < 16; ++w) {
                carry[0] += wsum[0][w];
                carry[1] += wsum[1][w];
            }
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        counters[CNT_V] = carry[0];
        counters[CNT_E] = carry[1];
    }
}

__global__ __launch_bounds__(kBlock) void k_scan_assign(HEntry *__restrict__ tab, int64_t cap,
                                                        const int32_t *__restrict__ blk,
                                                        uint64_t *__restrict__ vkeys, int32_t *__restrict__ vinfo,
                                                        int32_t *__restrict__ heavy, int32_t *counters) {
    __shared__ int wsum[2][kBlock / 64];
    __shared__ int carry[2];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t s0 = (int64_t)blockIdx.x * kScanSlots;
    const int64_t s1 = s0 + kScanSlots < cap ? s0 + kScanSlots : cap;
    if (threadIdx.x == 0) {
        carry[0] = blk[2 * blockIdx.x];
        carry[1] = blk[2 * blockIdx.x + 1];
    }
    __syncthreads();
    for (int64_t r = s0; r < s1; r += kBlock) {
        const int64_t s = r + threadIdx.x;
        HEntry e;
        e.key = 0ull;
        e.count = 0;
        if (s < s1) e = tab[s];
        const int o = e.key != 0ull;
        const int c = e.count;
        const int io = wave_incl_scan(o, lane);
        const int ic = wave_incl_scan(c, lane);
        if (lane == 63) {
            wsum[0][wave] = io;
            wsum[1][wave] = ic;
        }
        __syncthreads();
        int bo = carry[0], bc = carry[1];
        for (int w = 0; w < wave; ++w) {
            bo += wsum[0][w];
            bc += wsum[1][w];
        }
        if (o) {
            const int v = bo + io - 1;
            tab[s].vid = v;
            vkeys[v] = e.key;
            vinfo[2 * v] = bc + ic - c;
            vinfo[2 * v + 1] = c;
            if (c > kHeavy) heavy[atomicAdd(counters + CNT_H, 1)] = v;
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            for (int w = 0; w < kBlock / 64; ++w) {
                carry[0] += wsum[0][w];
                carry[1] += wsum[1][w];
            }
        }
        __syncthreads();
    }
}

// Per pair (p, k): map the hash slot to the vertex index (rewriting the
// per-point record in place) and place (p, b_pk) at its rank in the vertex's
// pair list.
template <int D>
__global__ __launch_bounds__(kBlock) void k_fill(int64_t n, int32_t *__restrict__ idx, const int32_t *__restrict__ rank,
                                                 const float *__restrict__ bary, const HEntry *__restrict__ tab,
                                                 const int32_t *__restrict__ vinfo, int32_t *__restrict__ list) {
    constexpr int DP1 = D + 1;
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x; e < n; e += stride) {
        const int s = idx[e];
        if (s < 0) continue;
        const int v = tab[s].vid;
        idx[e] = v;
        const int64_t at = (int64_t)vinfo[2 * v] + rank[e];
        list[2 * at] = (int32_t)(e / DP1);
        list[2 * at + 1] = __float_as_int(bary[e]);
    }
}

// Eq. (splat), pulled per vertex: x_v = sum over the vertex's pair list of
// b_pv f_p, and w_v = sum b_pv.  G lanes per vertex own float4 column chunks;
// every row of `values` is written exactly once (no zero fill, no float
// atomics).  Four list entries are fetched before their feature rows are
// used, to keep several row gathers in flight per lane.
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

template <bool VEC, bool OUT_BF16>
__global__ __launch_bounds__(kBlock) void k_gather(const int32_t *__restrict__ vinfo, const int32_t *__restrict__ list,
                                                   const float *__restrict__ feat, int C, int log2G, int normalize,
                                                   void *__restrict__ values, float *__restrict__ weight,
                                                   const int32_t *counters) {
    const int64_t V = counters[CNT_V];
    const int G = 1 << log2G;
    const int lane = threadIdx.x & 63;
    const int grp = lane >> log2G;
    const int j = lane & (G - 1);
    const int vpw = 64 >> log2G;
    const int64_t wave = ((int64_t)blockIdx.x * kBlock + threadIdx.x) >> 6;
    const int64_t nwaves = ((int64_t)gridDim.x * kBlock) >> 6;
    const int CV = VEC ? (C >> 2) : C;  // columns in units of float4 (VEC) or float
    for (int64_t v0 = wave * vpw; v0 < V; v0 += nwaves * vpw) {
        const int64_t v = v0 + grp;
        if (v >= V) continue;
        const int off = vinfo[2 * v];
        const int cnt = vinfo[2 * v + 1];
        if (cnt > kHeavy) continue;  // reduced by k_gather_heavy
        const int2 *L2 = reinterpret_cast<const int2 *>(list) + off;
        float w = 0.f;
        for (int e = 0; e < cnt; ++e) w += __int_as_float(L2[e].y);
        for (int c = j; c < CV; c += G) {
            if (VEC) {
                const float4 *f4 = reinterpret_cast<const float4 *>(feat);
                float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
                int e = 0;
                for (; e + 4 <= cnt; e += 4) {
                    const int2 q0 = L2[e], q1 = L2[e + 1], q2 = L2[e + 2], q3 = L2[e + 3];
                    const float4 y0 = f4[(int64_t)q0.x * CV + c], y1 = f4[(int64_t)q1.x * CV + c];
                    const float4 y2 = f4[(int64_t)q2.x * CV + c], y3 = f4[(int64_t)q3.x * CV + c];
                    const float b0 = __int_as_float(q0.y), b1 = __int_as_float(q1.y);
                    const float b2 = __int_as_float(q2.y), b3 = __int_as_float(q3.y);
                    acc.x = fmaf(b0, y0.x, acc.x); acc.y = fmaf(b0, y0.y, acc.y);
                    acc.z = fmaf(b0, y0.z, acc.z); acc.w = fmaf(b0, y0.w, acc.w);
                    acc.x = fmaf(b1, y1.x, acc.x); acc.y = fmaf(b1, y1.y, acc.y);
                    acc.z = fmaf(b1, y1.z, acc.z); acc.w = fmaf(b1, y1.w, acc.w);
                    acc.x = fmaf(b2, y2.x, acc.x); acc.y = fmaf(b2, y2.y, acc.y);
                    acc.z = fmaf(b2, y2.z, acc.z); acc.w = fmaf(b2, y2.w, acc.w);
                    acc.x = fmaf(b3, y3.x, acc.x); acc.y = fmaf(b3, y3.y, acc.y);
                    acc.z = fmaf(b3, y3.z, acc.z); acc.w = fmaf(b3, y3.w, acc.w);
                }
                for (; e < cnt; ++e) {
                    const int2 q = L2[e];
                    const float4 y = f4[(int64_t)q.x * CV + c];
                    const float bq = __int_as_float(q.y);
                    acc.x = fmaf(bq, y.x, acc.x); acc.y = fmaf(bq, y.y, acc.y);
                    acc.z = fmaf(bq, y.z, acc.z); acc.w = fmaf(bq, y.w, acc.w);
                }
                if (normalize) {
                    acc.x = w != 0.f ? acc.x / w : 0.f;
                    acc.y = w != 0.f ? acc.y / w : 0.f;
                    acc.z = w != 0.f ? acc.z / w : 0.f;
                    acc.w = w != 0.f ? acc.w / w : 0.f;
                }
                store4<OUT_BF16>(values, v * CV + c, acc);
            } else {
                float acc = 0.f;
                for (int e = 0; e < cnt; ++e) {
                    const int2 q = L2[e];
                    acc = fmaf(__int_as_float(q.y), feat[(int64_t)q.x * C + c], acc);
                }
                if (normalize) acc = w != 0.f ? acc / w : 0.f;
                store1<OUT_BF16>(values, v * C + c, acc);
            }
        }
        if (weight && j == 0) weight[v] = w;
    }
}

// Vertices with more than kHeavy pairs (dense regions, e.g. near a LiDAR
// sensor): one workgroup of kHeavyBlock threads per vertex.  Groups of G
// lanes (one float4 or float column each) take the pairs in a strided order,
// partial sums meet in LDS, and the first group writes the row.
// Deterministic for a given list order.
constexpr int kHeavyBlock = 1024;

template <bool VEC, bool OUT_BF16>
__global__ __launch_bounds__(kHeavyBlock) void k_gather_heavy(const int32_t *__restrict__ heavy,
                                                              const int32_t *__restrict__ vinfo,
                                                              const int32_t *__restrict__ list,
                                                              const float *__restrict__ feat, int C, int log2G,
                                                              int normalize, void *__restrict__ values,
                                                              float *__restrict__ weight, const int32_t *counters) {
    __shared__ float4 red[kHeavyBlock];
    __shared__ float wred[kHeavyBlock];
    const int nheavy = counters[CNT_H];
    const int G = 1 << log2G;
    const int ngroups = kHeavyBlock >> log2G;
    const int grp = threadIdx.x >> log2G;
    const int j = threadIdx.x & (G - 1);
    const int CV = VEC ? (C >> 2) : C;
    for (int h = blockIdx.x; h < nheavy; h += gridDim.x) {
        const int v = heavy[h];
        const int off = vinfo[2 * v];
        const int cnt = vinfo[2 * v + 1];
        const int2 *L2 = reinterpret_cast<const int2 *>(list) + off;
        float w = 0.f;
        for (int e = grp; e < cnt; e += ngroups) w += __int_as_float(L2[e].y);
        wred[threadIdx.x] = w;
        __syncthreads();
        float wt = 0.f;
        for (int g = 0; g < ngroups; ++g) wt += wred[g * G];
        for (int c0 = 0; c0 < CV; c0 += G) {
            const int c = c0 + j;
            float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
            if (c < CV) {
                if (VEC) {
                    const float4 *f4 = reinterpret_cast<const float4 *>(feat);
                    int e = grp;
                    for (; e + 3 * ngroups < cnt; e += 4 * ngroups) {
                        const int2 q0 = L2[e], q1 = L2[e + ngroups], q2 = L2[e + 2 * ngroups], q3 = L2[e + 3 * ngroups];
                        const float4 y0 = f4[(int64_t)q0.x * CV + c], y1 = f4[(int64_t)q1.x * CV + c];
                        const float4 y2 = f4[(int64_t)q2.x * CV + c], y3 = f4[(int64_t)q3.x * CV + c];
                        const float b0 = __int_as_float(q0.y), b1 = __int_as_float(q1.y);
                        const float b2 = __int_as_float(q2.y), b3 = __int_as_float(q3.y);
                        acc.x = fmaf(b0, y0.x, acc.x); acc.y = fmaf(b0, y0.y, acc.y);
                        acc.z = fmaf(b0, y0.z, acc.z); acc.w = fmaf(b0, y0.w, acc.w);
                        acc.x = fmaf(b1, y1.x, acc.x); acc.y = fmaf(b1, y1.y, acc.y);
                        acc.z = fmaf(b1, y1.z, acc.z); acc.w = fmaf(b1, y1.w, acc.w);
                        acc.x = fmaf(b2, y2.x, acc.x); acc.y = fmaf(b2, y2.y, acc.y);
                        acc.z = fmaf(b2, y2.z, acc.z); acc.w = fmaf(b2, y2.w, acc.w);
                        acc.x = fmaf(b3, y3.x, acc.x); acc.y = fmaf(b3, y3.y, acc.y);
                        acc.z = fmaf(b3, y3.z, acc.z); acc.w = fmaf(b3, y3.w, acc.w);
                    }
                    for (; e < cnt; e += ngroups) {
                        const int2 q = L2[e];
                        const float4 y = f4[(int64_t)q.x * CV + c];
                        const float bq = __int_as_float(q.y);
                        acc.x = fmaf(bq, y.x, acc.x); acc.y = fmaf(bq, y.y, acc.y);
                        acc.z = fmaf(bq, y.z, acc.z); acc.w = fmaf(bq, y.w, acc.w);
                    }
                } else {
                    for (int e = grp; e < cnt; e += ngroups) {
                        const int2 q = L2[e];
                        acc.x = fmaf(__int_as_float(q.y), feat[(int64_t)q.x * C + c], acc.x);
                    }
                }
            }
            red[threadIdx.x] = acc;
            __syncthreads();
            if (grp == 0 && c < CV) {
                float4 t = make_float4(0.f, 0.f, 0.f, 0.f);
                for (int g = 0; g < ngroups; ++g) {
                    const float4 r = red[g * G + j];
                    t.x += r.x; t.y += r.y; t.z += r.z; t.w += r.w;
                }
                if (normalize) {
                    t.x = wt != 0.f ? t.x / wt : 0.f;
                    t.y = wt != 0.f ? t.y / wt : 0.f;
                    t.z = wt != 0.f ? t.z / wt : 0.f;
                    t.w = wt != 0.f ? t.w / wt : 0.f;
                }
                if (VEC)
                    store4<OUT_BF16>(values, (int64_t)v * CV + c, t);
                else
                    store1<OUT_BF16>(values, (int64_t)v * C + c, t.x);
            }
            __syncthreads();
        }
        if (weight && threadIdx.x == 0) weight[v] = wt;
        __syncthreads();
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
    hipLaunchKernelGGL(k_clear_table, dim3(grid), dim3(kBlock), 0, L->stream, L->tab, L->cap, L->counters);
    return hipGetLastError();
}

hipError_t launch_insert(lattice *L, const float *pos, const int32_t *batch, int64_t m) {
    if (m == 0) return hipSuccess;
    ElevParams ep;
    for (int i = 0; i < LATTICE_MAX_D; ++i) ep.f[i] = L->factors[i];
    ep.inv = L->inv_dp1;
    const unsigned grid = (unsigned)((m + kInsertBlock - 1) / kInsertBlock);
    const uint32_t mask = (uint32_t)(L->cap - 1);
    return dispatch_d(L->d, [&](auto dc) {
        constexpr int D = decltype(dc)::value;
        hipLaunchKernelGGL(k_insert<D>, dim3(grid), dim3(kInsertBlock), 0, L->stream, pos, batch, m, ep, L->tab, mask,
                           L->idx, L->rank, L->bary, L->counters);
        return hipGetLastError();
    });
}

int64_t scan_blocks(const lattice *L) { return (L->cap + kScanSlots - 1) / kScanSlots; }

hipError_t launch_number(lattice *L) {
    const int64_t nb = scan_blocks(L);
    hipLaunchKernelGGL(k_scan_count, dim3((unsigned)nb), dim3(kBlock), 0, L->stream, L->tab, L->cap, L->blk);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_scan_blocks, dim3(1), dim3(1024), 0, L->stream, L->blk, (int)nb, L->counters);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_scan_assign, dim3((unsigned)nb), dim3(kBlock), 0, L->stream, L->tab, L->cap, L->blk,
                       L->vkeys, L->vinfo, L->heavy, L->counters);
    return hipGetLastError();
}

hipError_t launch_fill(lattice *L, int64_t m) {
    if (m == 0) return hipSuccess;
    const int64_t n = m * (L->d + 1);
    const unsigned grid = grid_for(n, kBlock, L->cu_count, 16);
    return dispatch_d(L->d, [&](auto dc) {
        constexpr int D = decltype(dc)::value;
        hipLaunchKernelGGL(k_fill<D>, dim3(grid), dim3(kBlock), 0, L->stream, n, L->idx, L->rank, L->bary, L->tab,
                           L->vinfo, L->list);
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
    const int64_t vpw = 64 >> log2G;
    const int64_t waves = (L->max_vertices + vpw - 1) / vpw;
    const unsigned grid = grid_for(waves * 64, kBlock, L->cu_count, 16);
    if (vec)
        hipLaunchKernelGGL((k_gather<true, OUT_BF16>), dim3(grid), dim3(kBlock), 0, L->stream, L->vinfo, L->list, feat,
                           C, log2G, normalize, values, weight, L->counters);
    else
        hipLaunchKernelGGL((k_gather<false, OUT_BF16>), dim3(grid), dim3(kBlock), 0, L->stream, L->vinfo, L->list, feat,
                           C, log2G, normalize, values, weight, L->counters);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // heavy vertices: G = lanes per column group, at most 64, so that a
    // workgroup has at least 16 groups splitting each long pair list
    const unsigned hgrid = (unsigned)(L->cu_count * 2);
    if (vec)
        hipLaunchKernelGGL((k_gather_heavy<true, OUT_BF16>), dim3(hgrid), dim3(kHeavyBlock), 0, L->stream, L->heavy,
                           L->vinfo, L->list, feat, C, log2G, normalize, values, weight, L->counters);
    else
        hipLaunchKernelGGL((k_gather_heavy<false, OUT_BF16>), dim3(hgrid), dim3(kHeavyBlock), 0, L->stream, L->heavy,
                           L->vinfo, L->list, feat, C, log2G, normalize, values, weight, L->counters);
    return hipGetLastError();
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
