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

template <int D>
__global__ __launch_bounds__(kBlock) void k_neighbors(const uint64_t *__restrict__ vkeys,
                                                      const HEntry *__restrict__ tab, uint32_t mask,
                                                      const int32_t *counters, int32_t *__restrict__ nbr) {
    constexpr int DP1 = D + 1;
    constexpr int T = 2 * DP1 + 1;
    const int64_t V = counters[CNT_V];
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t v = (int64_t)blockIdx.x * kBlock + threadIdx.x; v < V; v += stride) {
        int c[D];
        uint32_t b;
        unpack_key<D>(vkeys[v], c, b);
        // Keys of the 2(d+1) ring vertices: index j for +n_j, DP1 + j for -n_j.
        uint64_t key[2 * DP1];
        bool want[2 * DP1];
#pragma unroll
        for (int j = 0; j < DP1; ++j) {
#pragma unroll
            for (int sgn = 0; sgn < 2; ++sgn) {
                // Only c_0..c_{d-1} are packed; c_d follows from the zero sum.
                int q[D];
#pragma unroll
                for (int i = 0; i < D; ++i) {
                    const int n = (i == j ? DP1 : 0) - 1;
                    q[i] = sgn == 0 ? c[i] + n : c[i] - n;
                }
                want[sgn * DP1 + j] = pack_key<D>(q, b, key[sgn * DP1 + j]);
            }
        }
        int found[2 * DP1];
        hash_find_all<2 * DP1>(tab, mask, key, want, found);
        int32_t *row = nbr + v * T;
        row[0] = (int32_t)v;
#pragma unroll
        for (int t = 0; t < 2 * DP1; ++t) row[1 + t] = found[t];
    }
}

}  // namespace

hipError_t launch_neighbors(lattice *L) {
    const unsigned grid = grid_for(L->max_vertices, kBlock, L->cu_count, 8);
    const uint32_t mask = (uint32_t)(L->cap - 1);
    switch (L->d) {
#define NB_CASE(DD)                                                                                              \
    case DD:                                                                                                     \
        hipLaunchKernelGGL(k_neighbors<DD>, dim3(grid), dim3(kBlock), 0, L->stream, L->vkeys, L->tab, mask,       \
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
