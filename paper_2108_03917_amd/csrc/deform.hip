// DeformSlice (Sec. "Proposed Operations", DeformSlicing; Eq. deformSlice),
// optionally fused with the final linear classifier (Sec. "Implementation":
// the per-point high-dimensional features are never stored):
//
//   q_pk   = b_pk x_{v_pk}                                   (Gather)
//   mx_p   = max_k q_pk, per channel                         (MaxPool)
//   db_pk  = tanh(b_delta + (q_pk - mx_p) . w_delta)         (SubtractMax, Linear+Tanh)
//   f_p    = sum_k (b_pk + db_pk) x_{v_pk}                   (slice with b + db)
//   out_p  = f_p                  or   f_p W_cls^T + b_cls   (classifier)
//
// One group of G lanes per point (G the smallest power of two covering the
// row's float4 chunks, or its channels when C is not a multiple of 4): a
// lane keeps its chunks of the d+1 vertex rows in registers, so each row is
// read once; the two dot products over C (the offsets' linear layer and
// each class of the classifier) are reduced across the group with
// butterfly shuffles.  The classifier weights are read as float4 rows
// [n_cls][C] and stay in the L1/L2 (a few KB).
#include "internal.h"

namespace {

constexpr int kBlock = 256;

__device__ __forceinline__ float bf16_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }

template <bool IN_BF16>
__device__ __forceinline__ float4 row4(const void *values, int64_t at4) {
    if (IN_BF16) {
        const uint2 u = reinterpret_cast<const uint2 *>(values)[at4];
        return make_float4(bf16_lo(u.x), bf16_hi(u.x), bf16_lo(u.y), bf16_hi(u.y));
    }
    return reinterpret_cast<const float4 *>(values)[at4];
}
template <bool IN_BF16>
__device__ __forceinline__ float row1(const void *values, int64_t at) {
    if (IN_BF16) return __uint_as_float((uint32_t)reinterpret_cast<const uint16_t *>(values)[at] << 16);
    return reinterpret_cast<const float *>(values)[at];
}

// Sum over the G lanes of a group (G a power of two, groups aligned).
__device__ __forceinline__ float group_sum(float x, int G) {
    for (int off = G >> 1; off > 0; off >>= 1) x += __shfl_xor(x, off, 64);
    return x;
}

__device__ __forceinline__ float4 f4(float a) { return make_float4(a, a, a, a); }
__device__ __forceinline__ float4 mul4(float s, float4 a) { return make_float4(s * a.x, s * a.y, s * a.z, s * a.w); }
__device__ __forceinline__ float4 max4(float4 a, float4 b) {
    return make_float4(fmaxf(a.x, b.x), fmaxf(a.y, b.y), fmaxf(a.z, b.z), fmaxf(a.w, b.w));
}

// VEC: a lane's chunk i is float4 column chunk j + i G; else channel j + i G.
// CH chunks per lane: 1 (rows of at most 64 chunks) or 4 (at most 256).
template <int D, bool VEC, bool IN_BF16, bool CLS, int CH>
__global__ __launch_bounds__(kBlock) void k_deform_slice(int64_t m, int C, int log2G, const int32_t *__restrict__ idx,
                                                         const float *__restrict__ bary,
                                                         const void *__restrict__ values,
                                                         const float *__restrict__ w_delta, float b_delta,
                                                         const float *__restrict__ w_cls,
                                                         const float *__restrict__ b_cls, int n_cls,
                                                         float *__restrict__ out, float *__restrict__ delta_out) {
    constexpr int DP1 = D + 1;
    const int G = 1 << log2G;
    const int lane = threadIdx.x & 63;
    const int grp = lane >> log2G;
    const int j = lane & (G - 1);
    const int ppw = 64 >> log2G;
    const int NC = VEC ? (C >> 2) : C;  // chunks (float4 or single) per row
    const int64_t wave = ((int64_t)blockIdx.x * kBlock + threadIdx.x) >> 6;
    const int64_t nwaves = ((int64_t)gridDim.x * kBlock) >> 6;

    // the lane's slice of the offset weights
    float4 wd[CH];
#pragma unroll
    for (int i = 0; i < CH; ++i) {
        const int c = j + i * G;
        wd[i] = f4(0.f);
        if (c < NC) wd[i] = VEC ? reinterpret_cast<const float4 *>(w_delta)[c] : make_float4(w_delta[c], 0.f, 0.f, 0.f);
    }

    for (int64_t p0 = wave * ppw; p0 < m; p0 += nwaves * ppw) {
        const int64_t p = p0 + grp;
        const bool live = p < m;
        const int64_t pc = live ? p : 0;
        int v[DP1];
        float b[DP1];
#pragma unroll
        for (int k = 0; k < DP1; ++k) {
            v[k] = idx[pc * DP1 + k];
            b[k] = bary[pc * DP1 + k];
        }
        // Gather: the d+1 rows, chunk by chunk
        float4 x[DP1][CH];
#pragma unroll
        for (int k = 0; k < DP1; ++k)
#pragma unroll
            for (int i = 0; i < CH; ++i) {
                const int c = j + i * G;
                x[k][i] = f4(0.f);
                if (c < NC && v[k] >= 0)
                    x[k][i] = VEC ? row4<IN_BF16>(values, (int64_t)v[k] * NC + c)
                                  : make_float4(row1<IN_BF16>(values, (int64_t)v[k] * C + c), 0.f, 0.f, 0.f);
            }
        // MaxPool over the simplex, SubtractMax, Linear (lane partials)
        float4 mx[CH];
#pragma unroll
        for (int i = 0; i < CH; ++i) {
            mx[i] = mul4(b[0], x[0][i]);
#pragma unroll
            for (int k = 1; k < DP1; ++k) mx[i] = max4(mx[i], mul4(b[k], x[k][i]));
        }
        float db[DP1];
#pragma unroll
        for (int k = 0; k < DP1; ++k) {
            float s = 0.f;
#pragma unroll
            for (int i = 0; i < CH; ++i) {
                const float4 q = mul4(b[k], x[k][i]);
                s = fmaf(q.x - mx[i].x, wd[i].x, s);
                s = fmaf(q.y - mx[i].y, wd[i].y, s);
                s = fmaf(q.z - mx[i].z, wd[i].z, s);
                s = fmaf(q.w - mx[i].w, wd[i].w, s);
            }
            db[k] = tanhf(b_delta + group_sum(s, G));  // Tanh
        }
        // slice with the deformed weights
        float4 f[CH];
#pragma unroll
        for (int i = 0; i < CH; ++i) {
            f[i] = f4(0.f);
#pragma unroll
            for (int k = 0; k < DP1; ++k) {
                const float wk = b[k] + db[k];
                f[i].x = fmaf(wk, x[k][i].x, f[i].x);
                f[i].y = fmaf(wk, x[k][i].y, f[i].y);
                f[i].z = fmaf(wk, x[k][i].z, f[i].z);
                f[i].w = fmaf(wk, x[k][i].w, f[i].w);
            }
        }
        if (live && delta_out && j == 0) {
#pragma unroll
            for (int k = 0; k < DP1; ++k) delta_out[p * DP1 + k] = db[k];
        }
        if (!CLS) {
            if (live) {
#pragma unroll
                for (int i = 0; i < CH; ++i) {
                    const int c = j + i * G;
                    if (c < NC) {
                        if (VEC)
                            reinterpret_cast<float4 *>(out)[p * NC + c] = f[i];
                        else
                            out[p * C + c] = f[i].x;
                    }
                }
            }
        } else {
            // classifier: one group-wide dot product per class; the lane
            // j == cls mod G keeps the classes it writes
            for (int cls0 = 0; cls0 < n_cls; cls0 += G) {
                float mine = 0.f;
                const int nc = n_cls - cls0 < G ? n_cls - cls0 : G;
                for (int t = 0; t < nc; ++t) {
                    const int cls = cls0 + t;
                    float s = 0.f;
#pragma unroll
                    for (int i = 0; i < CH; ++i) {
                        const int c = j + i * G;
                        if (c < NC) {
                            if (VEC) {
                                const float4 wc = reinterpret_cast<const float4 *>(w_cls)[(int64_t)cls * NC + c];
                                s = fmaf(f[i].x, wc.x, s);
                                s = fmaf(f[i].y, wc.y, s);
                                s = fmaf(f[i].z, wc.z, s);
                                s = fmaf(f[i].w, wc.w, s);
                            } else {
                                s = fmaf(f[i].x, w_cls[(int64_t)cls * C + c], s);
                            }
                        }
                    }
                    s = group_sum(s, G);
                    if (j == t) mine = s;
                }
                if (live && j < nc) out[p * n_cls + cls0 + j] = mine + (b_cls ? b_cls[cls0 + j] : 0.f);
            }
        }
    }
}

template <int D, bool IN_BF16, int CH>
hipError_t launch_d(lattice *L, bool vec, int log2G, unsigned grid, const void *values, int C, const float *w_delta,
                    float b_delta, const float *w_cls, const float *b_cls, int n_cls, float *out, float *delta) {
#define DS_LAUNCH(VV, CC)                                                                                         \
    hipLaunchKernelGGL((k_deform_slice<D, VV, IN_BF16, CC, CH>), dim3(grid), dim3(kBlock), 0, L->stream, L->m, C, \
                       log2G, L->idx, L->bary, values, w_delta, b_delta, w_cls, b_cls, n_cls, out, delta)
    if (vec) {
        if (w_cls)
            DS_LAUNCH(true, true);
        else
            DS_LAUNCH(true, false);
    } else {
        if (w_cls)
            DS_LAUNCH(false, true);
        else
            DS_LAUNCH(false, false);
    }
#undef DS_LAUNCH
    return hipGetLastError();
}

template <int D>
hipError_t launch_dd(lattice *L, bool bf, int ch, bool vec, int log2G, unsigned grid, const void *values, int C,
                     const float *w_delta, float b_delta, const float *w_cls, const float *b_cls, int n_cls,
                     float *out, float *delta) {
    if (bf)
        return ch == 1 ? launch_d<D, true, 1>(L, vec, log2G, grid, values, C, w_delta, b_delta, w_cls, b_cls, n_cls,
                                              out, delta)
                       : launch_d<D, true, 4>(L, vec, log2G, grid, values, C, w_delta, b_delta, w_cls, b_cls, n_cls,
                                              out, delta);
    return ch == 1 ? launch_d<D, false, 1>(L, vec, log2G, grid, values, C, w_delta, b_delta, w_cls, b_cls, n_cls, out,
                                           delta)
                   : launch_d<D, false, 4>(L, vec, log2G, grid, values, C, w_delta, b_delta, w_cls, b_cls, n_cls, out,
                                           delta);
}

// Float4 path: C a multiple of 4 and every row pointer aligned to a chunk.
bool deform_vec(const void *values, lattice_dtype values_dt, int C, const float *w_delta, const float *w_cls,
                const float *out) {
    const bool bf = values_dt == LATTICE_BF16;
    return (C % 4 == 0) && ((reinterpret_cast<uintptr_t>(values) & (bf ? 7 : 15)) == 0) &&
           ((reinterpret_cast<uintptr_t>(w_delta) & 15) == 0) &&
           (w_cls ? ((reinterpret_cast<uintptr_t>(w_cls) & 15) == 0) : ((reinterpret_cast<uintptr_t>(out) & 15) == 0));
}

}  // namespace

int deform_max_channels(const void *values, lattice_dtype values_dt, int C, const float *w_delta, const float *w_cls,
                        const float *out) {
    return deform_vec(values, values_dt, C, w_delta, w_cls, out) ? 4 * 64 * 4 : 64 * 4;
}

hipError_t launch_deform_slice(lattice *L, const void *values, lattice_dtype values_dt, int C, const float *w_delta,
                               float b_delta, const float *w_cls, const float *b_cls, int n_cls, float *out,
                               float *delta) {
    const int64_t m = L->m;
    if (m == 0) return hipSuccess;
    const bool bf = values_dt == LATTICE_BF16;
    const bool vec = deform_vec(values, values_dt, C, w_delta, w_cls, out);
    const int lanes = vec ? C / 4 : C;
    if (lanes > 256) return hipErrorInvalidValue;
    int log2G = 0;
    while ((1 << log2G) < lanes && log2G < 6) ++log2G;
    const int ch = lanes <= 64 ? 1 : 4;
    const int64_t ppw = 64 >> log2G;
    const int64_t waves = (m + ppw - 1) / ppw;
    const unsigned grid = grid_for(waves * 64, kBlock, L->cu_count, 16);
#define DS_D(DD)                                                                                                     \
    case DD:                                                                                                         \
        return launch_dd<DD>(L, bf, ch, vec, log2G, grid, values, C, w_delta, b_delta, w_cls, b_cls, n_cls, out, delta);
    switch (L->d) {
        DS_D(1)
        DS_D(2)
        DS_D(3)
        DS_D(4)
        default:
            return hipErrorInvalidValue;
    }
#undef DS_D
}
