// Splat: elevation onto H_d, enclosing simplex, barycentric weights, hash
// insertion of the d+1 vertex keys (Sec. "Permutohedral Lattice"), and the
// barycentric accumulation of Eq. (splat).
//
// Kernel sequence of one lattice_splat (all on the lattice's stream):
//   k_clear_table   empty the hash table, zero V and the status word
//   k_insert        one thread per point: elevate, round, rank, wrap, weights,
//                   keys, CAS-insert; new vertices get indices from one atomic
//                   per wavefront (prefix sum of new-key counts over the wave)
//   k_clear_rows    zero rows 0..V-1 of values / weight (V read on device)
//   k_accumulate    G lanes per point: map slots to vertex indices, then
//                   fp32 atomic adds of b_k * f_p into the d+1 vertex rows
//   k_normalize     optional x_v / w_v
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

template <int D>
__global__ __launch_bounds__(kBlock) void k_insert(const float *__restrict__ pos, const int32_t *__restrict__ batch,
                                                   int64_t m, ElevParams ep, uint64_t *tkeys, int32_t *tvals,
                                                   uint32_t mask, int32_t *__restrict__ idx, float *__restrict__ bary,
                                                   uint64_t *__restrict__ vkeys, int32_t *counters) {
#pragma clang fp contract(off)
    constexpr int DP1 = D + 1;
    const int64_t p = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    const bool active = p < m;
    const int lane = threadIdx.x & 63;

    int slot[DP1];
    uint64_t key[DP1];
    bool isnew[DP1];
    float b[DP1];
#pragma unroll
    for (int k = 0; k < DP1; ++k) {
        slot[k] = -1;
        key[k] = 0;
        isnew[k] = false;
    }
#pragma unroll
    for (int k = 0; k < DP1; ++k) b[k] = 0.f;
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
        if (status == 0) {
#pragma unroll
            for (int k = 0; k < DP1; ++k) {
                bool nw;
                const int sl = hash_insert(tkeys, mask, key[k], nw);
                slot[k] = sl;
                isnew[k] = nw;
                if (sl < 0) status |= ST_CAPACITY;
            }
        }
    }

    // One atomic per wavefront hands out indices to the keys this wave created.
    int nnew = 0;
#pragma unroll
    for (int k = 0; k < DP1; ++k) nnew += isnew[k] ? 1 : 0;
    int incl = nnew;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int y = __shfl_up(incl, off, 64);
        if (lane >= off) incl += y;
    }
    const int total = __shfl(incl, 63, 64);
    int base = 0;
    if (lane == 63 && total > 0) base = atomicAdd(counters + CNT_V, total);
    base = __shfl(base, 63, 64);
    int v = base + incl - nnew;
#pragma unroll
    for (int k = 0; k < DP1; ++k) {
        if (isnew[k]) {
            tvals[slot[k]] = v;
            vkeys[v] = key[k];
            ++v;
        }
    }

    if (active) {
#pragma unroll
        for (int k = 0; k < DP1; ++k) {
            idx[p * DP1 + k] = slot[k];
            bary[p * DP1 + k] = status ? 0.f : b[k];
        }
    }
    if (status) atomicOr(counters + CNT_STATUS, status);
}

__global__ __launch_bounds__(kBlock) void k_clear_table(uint64_t *tkeys, int64_t cap, int32_t *counters) {
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    // cap is a power of two >= 64, so the table is a whole number of 16-byte vectors.
    uint4 *t4 = reinterpret_cast<uint4 *>(tkeys);
    const int64_t n4 = cap / 2;
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n4; i += stride) t4[i] = make_uint4(0, 0, 0, 0);
    if (blockIdx.x == 0 && threadIdx.x < CNT_WORDS) counters[threadIdx.x] = 0;
}

__global__ __launch_bounds__(kBlock) void k_clear_rows(float *values, int C, float *weight,
                                                       const int32_t *counters) {
    const int64_t V = counters[CNT_V];
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    const int64_t t0 = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (values) {
        const int64_t n = V * C;
        if ((reinterpret_cast<uintptr_t>(values) & 15) == 0) {
            float4 *v4 = reinterpret_cast<float4 *>(values);
            const int64_t n4 = n / 4;
            for (int64_t i = t0; i < n4; i += stride) v4[i] = make_float4(0.f, 0.f, 0.f, 0.f);
            for (int64_t i = n4 * 4 + t0; i < n; i += stride) values[i] = 0.f;
        } else {
            for (int64_t i = t0; i < n; i += stride) values[i] = 0.f;
        }
    }
    if (weight)
        for (int64_t i = t0; i < V; i += stride) weight[i] = 0.f;
}

// G lanes per point (G a power of two, 1..64); lane j of a group handles
// channels j, j+G, ...  The group first maps the point's d+1 hash slots to
// vertex indices (rewriting the per-point record in place), then adds
// b_k * f_p[c] into row v_k with fp32 atomics.
template <int D>
__global__ __launch_bounds__(kBlock) void k_accumulate(int64_t m, int C, int log2G, const float *__restrict__ feat,
                                                       int32_t *idx, const float *__restrict__ bary,
                                                       const int32_t *__restrict__ tvals, float *values,
                                                       float *weight) {
    constexpr int DP1 = D + 1;
    const int G = 1 << log2G;
    const int lane = threadIdx.x & 63;
    const int grp = lane >> log2G;
    const int j = lane & (G - 1);
    const int ppw = 64 >> log2G;
    const int64_t wave = ((int64_t)blockIdx.x * kBlock + threadIdx.x) >> 6;
    const int64_t nwaves = ((int64_t)gridDim.x * kBlock) >> 6;
    for (int64_t p0 = wave * ppw; p0 < m; p0 += nwaves * ppw) {
        const int64_t p = p0 + grp;
        if (p >= m) continue;
        int v[DP1];
        float b[DP1];
#pragma unroll
        for (int k = 0; k < DP1; ++k) {
            const int s = idx[p * DP1 + k];
            v[k] = s >= 0 ? tvals[s] : -1;
            b[k] = bary[p * DP1 + k];
        }
        if (j == 0) {
#pragma unroll
            for (int k = 0; k < DP1; ++k) {
                idx[p * DP1 + k] = v[k];
                if (weight && v[k] >= 0) unsafeAtomicAdd(weight + v[k], b[k]);
            }
        }
        const float *fp = feat + p * C;
        for (int c = j; c < C; c += G) {
            const float f = fp[c];
#pragma unroll
            for (int k = 0; k < DP1; ++k)
                if (v[k] >= 0) unsafeAtomicAdd(values + (int64_t)v[k] * C + c, b[k] * f);
        }
    }
}

__global__ __launch_bounds__(kBlock) void k_normalize(float *values, int C, const float *__restrict__ weight,
                                                      const int32_t *counters) {
    const int64_t V = counters[CNT_V];
    const int64_t n = V * C;
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += stride) {
        const float w = weight[i / C];
        values[i] = (w != 0.f) ? values[i] / w : 0.f;
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
        const uint32_t u = __float_as_uint(src[i]);
        uint16_t h;
        if ((u & 0x7fffffffu) > 0x7f800000u)
            h = (uint16_t)((u >> 16) | 0x40u);
        else
            h = (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
        dst[i] = h;
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
    const unsigned grid = grid_for(L->cap / 2, kBlock, L->cu_count, 4);
    hipLaunchKernelGGL(k_clear_table, dim3(grid), dim3(kBlock), 0, L->stream, L->tkeys, L->cap, L->counters);
    return hipGetLastError();
}

hipError_t launch_insert(lattice *L, const float *pos, const int32_t *batch, int64_t m) {
    if (m == 0) return hipSuccess;
    ElevParams ep;
    for (int i = 0; i < LATTICE_MAX_D; ++i) ep.f[i] = L->factors[i];
    ep.inv = L->inv_dp1;
    const unsigned grid = (unsigned)((m + kBlock - 1) / kBlock);
    const uint32_t mask = (uint32_t)(L->cap - 1);
    return dispatch_d(L->d, [&](auto dc) {
        constexpr int D = decltype(dc)::value;
        hipLaunchKernelGGL(k_insert<D>, dim3(grid), dim3(kBlock), 0, L->stream, pos, batch, m, ep, L->tkeys,
                           L->tvals, mask, L->idx, L->bary, L->vkeys, L->counters);
        return hipGetLastError();
    });
}

hipError_t launch_clear_rows(lattice *L, float *values, int C, float *weight) {
    const int64_t work = L->max_vertices * (int64_t)(C > 0 ? C : 1);
    const unsigned grid = grid_for(work / 4 + 1, kBlock, L->cu_count, 4);
    hipLaunchKernelGGL(k_clear_rows, dim3(grid), dim3(kBlock), 0, L->stream, values, C, weight, L->counters);
    return hipGetLastError();
}

hipError_t launch_accumulate(lattice *L, int64_t m, const float *feat, int C, float *values, float *weight) {
    if (m == 0) return hipSuccess;
    int log2G = 0;
    while ((1 << log2G) < C && log2G < 6) ++log2G;
    const int64_t ppw = 64 >> log2G;
    const int64_t waves = (m + ppw - 1) / ppw;
    const unsigned grid = grid_for(waves * 64, kBlock, L->cu_count, 16);
    return dispatch_d(L->d, [&](auto dc) {
        constexpr int D = decltype(dc)::value;
        hipLaunchKernelGGL(k_accumulate<D>, dim3(grid), dim3(kBlock), 0, L->stream, m, C, log2G, feat, L->idx,
                           L->bary, L->tvals, values, weight);
        return hipGetLastError();
    });
}

hipError_t launch_normalize(lattice *L, float *values, int C, const float *weight) {
    const unsigned grid = grid_for(L->max_vertices * (int64_t)C, kBlock, L->cu_count, 4);
    hipLaunchKernelGGL(k_normalize, dim3(grid), dim3(kBlock), 0, L->stream, values, C, weight, L->counters);
    return hipGetLastError();
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
