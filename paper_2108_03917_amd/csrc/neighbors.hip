// Neighbour table of the 1-hop ring (Sec. "Permutohedral Lattice": the
// 2(d+1) neighbours of a vertex are at +-[-1,..,-1,d,-1,..,-1]; Sec. "Common
// Operations": the convolution spans the 2(d+1)+1 vertices of the ring).
//
// One thread per vertex: tap 0 is the vertex itself, tap 1+j the key
// c + n_j and tap d+2+j the key c - n_j with n_j = (d+1) e_j - 1; each is
// looked up in the hash table (same batch id), -1 when not allocated.
#include "internal.h"
#include "keys.h"

namespace {

constexpr int kBlock = 256;

// One thread per (vertex, ring tap): tap 1+j looks up c + n_j, tap d+2+j
// looks up c - n_j; the thread of tap 1 also writes tap 0 (the vertex).
template <int D>
__global__ __launch_bounds__(kBlock) void k_neighbors(const uint64_t *__restrict__ vkeys,
                                                      const HEntry *__restrict__ tab,
                                                      const uint32_t *__restrict__ occ, uint32_t mask,
                                                      const int32_t *counters, int32_t *__restrict__ nbr) {
    constexpr int DP1 = D + 1;
    constexpr int R = 2 * DP1;  // ring taps
    constexpr int T = R + 1;
    const int64_t n = (int64_t)counters[CNT_V] * R;
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x; e < n; e += stride) {
        const int64_t v = e / R;
        const int tap = (int)(e - v * R);         // 0..R-1 -> row entry 1+tap
        const int j = tap < DP1 ? tap : tap - DP1;
        const bool plus = tap < DP1;
        int c[D];
        uint32_t b;
        unpack_key<D>(vkeys[v], c, b);
        // Only c_0..c_{d-1} are packed; c_d follows from the zero sum.
#pragma unroll
        for (int i = 0; i < D; ++i) {
            const int nj = (i == j ? DP1 : 0) - 1;
            c[i] = plus ? c[i] + nj : c[i] - nj;
        }
        uint64_t key;
        const bool want = pack_key<D>(c, b, key);
        int found = -1;
        hash_find_all<1>(tab, occ, mask, &key, &want, &found);
        int32_t *row = nbr + v * T;
        row[1 + tap] = found;
        if (tap == 0) row[0] = (int32_t)v;
    }
}

}  // namespace

hipError_t launch_neighbors(lattice *L) {
    const unsigned grid = grid_for(L->max_vertices * 2 * (L->d + 1), kBlock, L->cu_count, 16);
    const uint32_t mask = (uint32_t)(L->cap - 1);
    switch (L->d) {
#define NB_CASE(DD)                                                                                              \
    case DD:                                                                                                     \
        hipLaunchKernelGGL(k_neighbors<DD>, dim3(grid), dim3(kBlock), 0, L->stream, L->vkeys, L->tab, L->occ, mask, \
                           L->counters, L->nbr);                                                                 \
        return hipGetLastError();
        NB_CASE(1)
        NB_CASE(2)
        NB_CASE(3)
        NB_CASE(4)
#undef NB_CASE
        default:
            return hipErrorInvalidValue;
    }
}

// ---------------------------------------------------------------------------
// Cross-lattice tables for downsampling and upsampling (Sec. "Proposed
// Operations": Downsampling, Upsampling; the Coarsen figure).  One thread per
// (output vertex, tap), tap order as in the 1-ring (offset_0 = 0,
// offset_{1+j} = +n_j, offset_{d+2+j} = -n_j):
//   down: coarse vertex c' reads the fine vertex 2c' + offset_t;
//   up:   fine vertex u reads the coarse vertex (u + offset_t) / 2, and
//         nothing (-1) when that key has an odd coordinate (it lies inside a
//         coarse simplex).  Only c_0..c_{d-1} are packed; c_d = -sum is even
//         whenever they are.
// The lookup is in the other lattice's hash table, with the same batch id.
// ---------------------------------------------------------------------------
namespace {

template <int D, bool UP>
__global__ __launch_bounds__(kBlock) void k_cross(const uint64_t *__restrict__ vkeys, const int32_t *counters,
                                                  const HEntry *__restrict__ tab, const uint32_t *__restrict__ occ,
                                                  uint32_t mask,
                                                  int32_t *__restrict__ xnbr) {
    constexpr int DP1 = D + 1;
    constexpr int T = 2 * DP1 + 1;
    const int64_t n = (int64_t)counters[CNT_V] * T;
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x; e < n; e += stride) {
        const int64_t v = e / T;
        const int t = (int)(e - v * T);
        int c[D];
        uint32_t b;
        unpack_key<D>(vkeys[v], c, b);
        const int j = t == 0 ? -1 : (t <= DP1 ? t - 1 : t - 1 - DP1);
        const int sgn = t == 0 ? 0 : (t <= DP1 ? 1 : -1);
        bool integral = true;
#pragma unroll
        for (int i = 0; i < D; ++i) {
            const int off = sgn * ((i == j ? DP1 : 0) - 1);
            if (UP) {
                const int q = c[i] + off;
                integral = integral && (q & 1) == 0;
                c[i] = q >> 1;  // exact for even q, sign included
            } else {
                c[i] = 2 * c[i] + off;
            }
        }
        uint64_t key = 0;
        const bool want = pack_key<D>(c, b, key) && integral;
        int found = -1;
        hash_find_all<1>(tab, occ, mask, &key, &want, &found);
        xnbr[e] = found;
    }
}

}  // namespace

hipError_t launch_cross(lattice *out, const lattice *src, bool up, int32_t *xnbr) {
    const unsigned grid = grid_for(out->max_vertices * (int64_t)out->T, kBlock, out->cu_count, 16);
    const uint32_t mask = (uint32_t)(src->cap - 1);
    switch (out->d) {
#define CR_CASE(DD)                                                                                              \
    case DD:                                                                                                     \
        if (up)                                                                                                  \
            hipLaunchKernelGGL((k_cross<DD, true>), dim3(grid), dim3(kBlock), 0, out->stream, out->vkeys,        \
                               out->counters, src->tab, src->occ, mask, xnbr);                                   \
        else                                                                                                     \
            hipLaunchKernelGGL((k_cross<DD, false>), dim3(grid), dim3(kBlock), 0, out->stream, out->vkeys,       \
                               out->counters, src->tab, src->occ, mask, xnbr);                                   \
        return hipGetLastError();
        CR_CASE(1)
        CR_CASE(2)
        CR_CASE(3)
        CR_CASE(4)
#undef CR_CASE
        default:
            return hipErrorInvalidValue;
    }
}
