// Slice (Eq. slice): f_p = sum_{v in I_p} b_pv x_v, with the vertex indices
// and barycentric weights recorded by the last splat.
//
// The same gather is the gradient of the splat with respect to the point
// features (Eq. splat is x = B^T f, so df = B dx).  For the normalised
// splat x_v / w_v the vertex gradient is divided by w_v first (NORM: the
// weight b_pv becomes b_pv / w_v, and 0 where w_v = 0).
//
// G lanes per point, each lane owning float4 column chunks j, j+G, ... of the
// C channels: a row gather of the d+1 vertex rows is contiguous per group, so
// a wavefront issues 64 x 16 B coalesced reads per vertex.
#include "internal.h"

#include <hip/hip_ext.h>

namespace {

constexpr int kBlock = 256;

__device__ __forceinline__ float bf16_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }

// Load 4 consecutive channels of a vertex row stored as fp32 or bf16.
template <bool IN_BF16>
__device__ __forceinline__ float4 load4(const void *values, int64_t at4) {
    if (IN_BF16) {
        const uint2 u = reinterpret_cast<const uint2 *>(values)[at4];
        return make_float4(bf16_lo(u.x), bf16_hi(u.x), bf16_lo(u.y), bf16_hi(u.y));
    }
    return reinterpret_cast<const float4 *>(values)[at4];
}
template <bool IN_BF16>
__device__ __forceinline__ float load1(const void *values, int64_t at) {
    if (IN_BF16) return __uint_as_float((uint32_t)reinterpret_cast<const uint16_t *>(values)[at] << 16);
    return reinterpret_cast<const float *>(values)[at];
}

template <int D, bool VEC, bool IN_BF16, bool NORM>
__global__ __launch_bounds__(kBlock) void k_slice(int64_t m, int C, int log2G, const int32_t *__restrict__ idx,
                                                  const float *__restrict__ bary, const void *__restrict__ values,
                                                  const float *__restrict__ vweight, float *__restrict__ out) {
    constexpr int DP1 = D + 1;
    const int G = 1 << log2G;
    const int lane = threadIdx.x & 63;
    const int grp = lane >> log2G;
    const int j = lane & (G - 1);
    const int ppw = 64 >> log2G;
    // each XCD slices one contiguous range of points: neighbouring points
    // share their vertex rows, which then meet in that XCD's L2
    const XcdShare sh = xcd_share(m);
    for (int64_t p0 = sh.lo + sh.wave * ppw; p0 < sh.hi; p0 += sh.nwaves * ppw) {
        const int64_t p = p0 + grp;
        if (p >= sh.hi) continue;
        // A point whose insertion failed (the splat reports it) has vertex -1
        // in some slots: those read another of its rows with weight 0, and a
        // point with none reads nothing.  The d+1 row loads are unconditional
        // so that they are all in flight together (with a branch per vertex
        // the compiler issued them one round trip at a time).
        int v[DP1];
        float b[DP1];
        int fb = -1;
#pragma unroll
        for (int k = 0; k < DP1; ++k) {
            v[k] = idx[p * DP1 + k];
            b[k] = bary[p * DP1 + k];
            fb = v[k] >= 0 ? v[k] : fb;
        }
        const bool any = fb >= 0;
#pragma unroll
        for (int k = 0; k < DP1; ++k) {
            b[k] = v[k] >= 0 ? b[k] : 0.f;
            v[k] = v[k] >= 0 ? v[k] : (any ? fb : 0);
        }
        if (NORM && any) {
            float wv[DP1];
#pragma unroll
            for (int k = 0; k < DP1; ++k) wv[k] = vweight[v[k]];
#pragma unroll
            for (int k = 0; k < DP1; ++k) b[k] = wv[k] != 0.f ? b[k] / wv[k] : 0.f;
        }
        if (VEC) {
            const int C4 = C >> 2;
            float4 *out4 = reinterpret_cast<float4 *>(out) + p * C4;
            for (int c = j; c < C4; c += G) {
                float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
                if (any) {
                    float4 y[DP1];
#pragma unroll
                    for (int k = 0; k < DP1; ++k) y[k] = load4<IN_BF16>(values, (int64_t)v[k] * C4 + c);
#pragma unroll
                    for (int k = 0; k < DP1; ++k) {
                        acc.x = fmaf(b[k], y[k].x, acc.x);
                        acc.y = fmaf(b[k], y[k].y, acc.y);
                        acc.z = fmaf(b[k], y[k].z, acc.z);
                        acc.w = fmaf(b[k], y[k].w, acc.w);
                    }
                }
                out4[c] = acc;
            }
        } else {
            for (int c = j; c < C; c += G) {
                float acc = 0.f;
                if (any) {
                    float y[DP1];
#pragma unroll
                    for (int k = 0; k < DP1; ++k) y[k] = load1<IN_BF16>(values, (int64_t)v[k] * C + c);
#pragma unroll
                    for (int k = 0; k < DP1; ++k) acc = fmaf(b[k], y[k], acc);
                }
                out[p * C + c] = acc;
            }
        }
    }
}

}  // namespace

template <bool IN_BF16, bool NORM>
static hipError_t slice_typed(lattice *L, const void *values, int C, const float *vweight, float *out) {
    const int64_t m = L->m;
    if (m == 0) return hipSuccess;
    const bool vec = (C % 4 == 0) && ((reinterpret_cast<uintptr_t>(values) & (IN_BF16 ? 7 : 15)) == 0) &&
                     ((reinterpret_cast<uintptr_t>(out) & 15) == 0);
    const int lanes_needed = vec ? C / 4 : C;
    int log2G = 0;
    while ((1 << log2G) < lanes_needed && log2G < 6) ++log2G;
    const int64_t ppw = 64 >> log2G;
    const int64_t waves = (m + ppw - 1) / ppw;
    const unsigned grid = grid_for(waves * 64, kBlock, L->cu_count, 16);
#define SL_CASE(DD)                                                                                              \
    case DD:                                                                                                     \
        if (vec)                                                                                                 \
            hipExtLaunchKernelGGL((k_slice<DD, true, IN_BF16, NORM>), dim3(grid), dim3(kBlock), 0, L->stream,    \
                                  L->kt_start, L->kt_stop, 0, m, C, log2G, L->idx, L->bary, values, vweight, out); \
        else                                                                                                     \
            hipExtLaunchKernelGGL((k_slice<DD, false, IN_BF16, NORM>), dim3(grid), dim3(kBlock), 0, L->stream,   \
                                  L->kt_start, L->kt_stop, 0, m, C, log2G, L->idx, L->bary, values, vweight, out); \
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

hipError_t launch_slice(lattice *L, const void *values, lattice_dtype values_dt, int C, float *out) {
    return values_dt == LATTICE_BF16 ? slice_typed<true, false>(L, values, C, nullptr, out)
                                     : slice_typed<false, false>(L, values, C, nullptr, out);
}

hipError_t launch_splat_backward(lattice *L, const void *grad_values, lattice_dtype gv_dt, int C,
                                 const float *vweight, float *grad_feat) {
    if (vweight)
        return gv_dt == LATTICE_BF16 ? slice_typed<true, true>(L, grad_values, C, vweight, grad_feat)
                                     : slice_typed<false, true>(L, grad_values, C, vweight, grad_feat);
    return launch_slice(L, grad_values, gv_dt, C, grad_feat);
}
