// Slice (Eq. slice): f_p = sum_{v in I_p} b_pv x_v, with the vertex indices
// and barycentric weights recorded by the last splat.
//
// G lanes per point, each lane owning float4 column chunks j, j+G, ... of the
// C channels: a row gather of the d+1 vertex rows is contiguous per group, so
// a wavefront issues 64 x 16 B coalesced reads per vertex.
#include "internal.h"

namespace {

constexpr int kBlock = 256;

template <int D, bool VEC>
__global__ __launch_bounds__(kBlock) void k_slice(int64_t m, int C, int log2G, const int32_t *__restrict__ idx,
                                                  const float *__restrict__ bary, const float *__restrict__ values,
                                                  float *__restrict__ out) {
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
            v[k] = idx[p * DP1 + k];
            b[k] = bary[p * DP1 + k];
        }
        if (VEC) {
            const int C4 = C >> 2;
            const float4 *val4 = reinterpret_cast<const float4 *>(values);
            float4 *out4 = reinterpret_cast<float4 *>(out) + p * C4;
            for (int c = j; c < C4; c += G) {
                float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
                for (int k = 0; k < DP1; ++k) {
                    if (v[k] < 0) continue;
                    const float4 y = val4[(int64_t)v[k] * C4 + c];
                    acc.x = fmaf(b[k], y.x, acc.x);
                    acc.y = fmaf(b[k], y.y, acc.y);
                    acc.z = fmaf(b[k], y.z, acc.z);
                    acc.w = fmaf(b[k], y.w, acc.w);
                }
                out4[c] = acc;
            }
        } else {
            for (int c = j; c < C; c += G) {
                float acc = 0.f;
#pragma unroll
                for (int k = 0; k < DP1; ++k)
                    if (v[k] >= 0) acc = fmaf(b[k], values[(int64_t)v[k] * C + c], acc);
                out[p * C + c] = acc;
            }
        }
    }
}

}  // namespace

hipError_t launch_slice(lattice *L, const float *values, int C, float *out) {
    const int64_t m = L->m;
    if (m == 0) return hipSuccess;
    const bool vec = (C % 4 == 0) && ((reinterpret_cast<uintptr_t>(values) & 15) == 0) &&
                     ((reinterpret_cast<uintptr_t>(out) & 15) == 0);
    const int lanes_needed = vec ? C / 4 : C;
    int log2G = 0;
    while ((1 << log2G) < lanes_needed && log2G < 6) ++log2G;
    const int64_t ppw = 64 >> log2G;
    const int64_t waves = (m + ppw - 1) / ppw;
    const unsigned grid = grid_for(waves * 64, kBlock, L->cu_count, 16);
#define SL_CASE(DD)                                                                                          \
    case DD:                                                                                                 \
        if (vec)                                                                                             \
            hipLaunchKernelGGL((k_slice<DD, true>), dim3(grid), dim3(kBlock), 0, L->stream, m, C, log2G, L->idx, \
                               L->bary, values, out);                                                        \
        else                                                                                                 \
            hipLaunchKernelGGL((k_slice<DD, false>), dim3(grid), dim3(kBlock), 0, L->stream, m, C, log2G,      \
                               L->idx, L->bary, values, out);                                                \
        return hipGetLastError();
    switch (L->d) {
        SL_CASE(1)
        SL_CASE(2)
        SL_CASE(3)
        SL_CASE(4)
        default:
            return hipErrorInvalidValue;
    }
#undef SL_CASE
}
