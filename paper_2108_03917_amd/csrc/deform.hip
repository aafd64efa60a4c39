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
// read once, and the offsets' dot product over C is reduced across the
// group.
//
// k_deform_fast (float4 rows of at most 128 channels, at most 64 classes --
// the shapes of the segmentation networks): G is a compile-time constant,
// so the group sums are DPP row operations and lane swaps, not LDS
// shuffles.  The classifier runs class-per-lane: each lane keeps one
// class's weight row in registers for the whole launch, the wave's point
// features pass through LDS, and 64 / n_cls points (at most 4) are scored
// side by side.  Every logit is one lane's sequential dot product; no
// cross-lane reduction and no re-read of the weights.
//
// k_deform_generic (any other shape): runtime G, butterfly shuffles, and the
// classifier as one group-wide dot product per class with the weights read
// as float4 rows from the L1/L2.
#include <atomic>

#include "internal.h"

#include <hip/hip_ext.h>

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
__global__ __launch_bounds__(kBlock) void k_deform_generic(int64_t m, int C, int log2G, const int32_t *__restrict__ idx,
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


// Sum over aligned groups of 2^LG lanes; every lane of a group receives the
// same bits (each step adds a value and its partner's in either order).
template <int CTRL>
__device__ __forceinline__ float add_dpp(float x) {
    return x + __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xF, 0xF, false));
}
template <int LG>
__device__ __forceinline__ float group_sum_c(float x) {
    if (LG >= 1) x = add_dpp<0xB1>(x);   // quad_perm [1,0,3,2]
    if (LG >= 2) x = add_dpp<0x4E>(x);   // quad_perm [2,3,0,1]
    if (LG >= 3) x = add_dpp<0x141>(x);  // row_half_mirror: the other quad of the 8
    if (LG >= 4) x = add_dpp<0x140>(x);  // row_mirror: the other 8 of the row
    if (LG >= 5) {                       // the other row of each 32
        const auto r = __builtin_amdgcn_permlane16_swap(__float_as_int(x), __float_as_int(x), false, false);
        x = __int_as_float(r[0]) + __int_as_float(r[1]);
    }
    if (LG >= 6) {                       // the other 32 lanes
        const auto r = __builtin_amdgcn_permlane32_swap(__float_as_int(x), __float_as_int(x), false, false);
        x = __int_as_float(r[0]) + __int_as_float(r[1]);
    }
    return x;
}

typedef float f32x4_t __attribute__((ext_vector_type(4)));

// One group of G = 2^LG lanes per point, one float4 chunk per lane
// (C <= 4G, C a multiple of 4).  NCB > 0: the classifier, n_cls <= 16 NCB,
// on fp32 MFMA: the features of 16 points are staged in LDS (rows padded to
// 4G + 4 floats, so that the 16 rows of one read fall in distinct banks),
// and one 16x16x4 step multiplies 16 points x 4 channels by 4 channels x 16
// classes.  Lane l supplies point / class l % 16 and channels
// 16t + 4(l / 16) + e at step (t, e), the same channel on both sides, so
// every channel meets its own weight once.  The weight fragments are loaded
// once per workgroup into LDS in lane order (each read is 64 consecutive
// float4), except for 128-channel rows with more than 32 classes, where they
// would not fit beside the staged rows and stay in registers.
template <int D, int LG, bool IN_BF16, int NCB>
__global__ __launch_bounds__(kBlock) void k_deform_fast(int64_t m, int C, const int32_t *__restrict__ idx,
                                                        const float *__restrict__ bary,
                                                        const void *__restrict__ values,
                                                        const float *__restrict__ w_delta, float b_delta,
                                                        const float *__restrict__ w_cls,
                                                        const float *__restrict__ b_cls, int n_cls,
                                                        float *__restrict__ out, float *__restrict__ delta_out) {
    constexpr bool CLS = NCB > 0;
    constexpr int DP1 = D + 1;
    constexpr int G = 1 << LG;
    constexpr int PPW = 64 / G;   // points per wave and round
    constexpr int S = 4 * G + 4;  // staged row stride, floats
    constexpr int T16 = G / 4;    // 16-channel steps covering 4G channels
    constexpr int WAVES = kBlock / 64;
    constexpr bool WL = CLS && !(LG == 5 && NCB == 4);  // weight fragments in LDS
    __shared__ float fbuf[CLS ? WAVES * 16 * S : 1];
    __shared__ int64_t sid[CLS ? WAVES * 16 : 1];
    __shared__ float4 wlds[WL ? NCB * T16 * 64 : 1];

    const int lane = threadIdx.x & 63;
    const int wv = threadIdx.x >> 6;
    const int grp = lane >> LG;
    const int j = lane & (G - 1);
    const int NC = C >> 2;
    const bool has = j < NC;
    const int64_t wave = ((int64_t)blockIdx.x * kBlock + threadIdx.x) >> 6;
    const int64_t nwaves = ((int64_t)gridDim.x * kBlock) >> 6;

    const float4 wd = has ? reinterpret_cast<const float4 *>(w_delta)[j] : f4(0.f);

    // classifier fragments: lane l holds class cb*16 + l%16, channels
    // 16t + 4(l/16) + 0..3 (zero past C or past n_cls)
    const int col = lane & 15;
    const int kg = lane >> 4;
    auto wfrag = [&](int cb, int t, int ln) {
        const int cls = cb * 16 + (ln & 15);
        const int ch = 16 * t + 4 * (ln >> 4);
        return (cls < n_cls && ch < C) ? *reinterpret_cast<const float4 *>(w_cls + (int64_t)cls * C + ch) : f4(0.f);
    };
    float4 wf[CLS && !WL ? NCB : 1][CLS && !WL ? T16 : 1];
    float bias[CLS ? NCB : 1];
    if (CLS) {
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) {
            const int cls = cb * 16 + col;
            bias[cb] = (cls < n_cls && b_cls) ? b_cls[cls] : 0.f;
        }
    }
    if (WL) {
        // fragment (cb, t) of lane ln at wlds[(cb T16 + t) 64 + ln]
        for (int e = threadIdx.x; e < NCB * T16 * 64; e += kBlock) wlds[e] = wfrag(e / (T16 * 64), (e / 64) % T16, e & 63);
        __syncthreads();
    } else if (CLS) {
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
            for (int t = 0; t < T16; ++t) wf[cb][t] = wfrag(cb, t, lane);
    }
    float *fb = fbuf + wv * (CLS ? 16 * S : 0);
    int64_t *sb = sid + wv * (CLS ? 16 : 0);

    auto wave_sync = [] {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    };
    auto score = [&](int nsl) {
        if (lane < 16 && lane >= nsl) sb[lane] = -1;  // unfilled slots of a last, partial batch
        wave_sync();
        f32x4_t acc[CLS ? NCB : 1];
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) acc[cb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int t = 0; t < T16; ++t) {
            const int ch = 16 * t + 4 * kg;
            float4 a = f4(0.f);
            if (ch < C) a = *reinterpret_cast<const float4 *>(fb + col * S + ch);
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) {
                const float4 w = WL ? wlds[(cb * T16 + t) * 64 + lane] : wf[WL ? 0 : cb][WL ? 0 : t];
                acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, w.x, acc[cb], 0, 0, 0);
                acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, w.y, acc[cb], 0, 0, 0);
                acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, w.z, acc[cb], 0, 0, 0);
                acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, w.w, acc[cb], 0, 0, 0);
            }
        }
        // 16x16 accumulator layout: register r of lane l holds point
        // 4 (l / 16) + r, class l % 16 of the block
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int64_t p = sb[4 * kg + r];
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) {
                const int cls = cb * 16 + col;
                if (p >= 0 && cls < n_cls) out[p * n_cls + cls] = acc[cb][r] + bias[cb];
            }
        }
        wave_sync();
    };

    int nsl = 0;
    for (int64_t p0 = wave * PPW; p0 < m; p0 += nwaves * PPW) {
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
        float4 x[DP1];
#pragma unroll
        for (int k = 0; k < DP1; ++k)
            x[k] = (has && v[k] >= 0) ? row4<IN_BF16>(values, (int64_t)v[k] * NC + j) : f4(0.f);
        float4 mx = mul4(b[0], x[0]);
#pragma unroll
        for (int k = 1; k < DP1; ++k) mx = max4(mx, mul4(b[k], x[k]));
        float db[DP1];
#pragma unroll
        for (int k = 0; k < DP1; ++k) {
            const float4 q = mul4(b[k], x[k]);
            float s = 0.f;
            s = fmaf(q.x - mx.x, wd.x, s);
            s = fmaf(q.y - mx.y, wd.y, s);
            s = fmaf(q.z - mx.z, wd.z, s);
            s = fmaf(q.w - mx.w, wd.w, s);
            db[k] = b_delta + group_sum_c<LG>(s);
        }
        if (LG >= 4) {
            // every lane of a group holds every argument: lane k of each row
            // takes the tanh of argument k, then row_newbcast:k hands it to
            // the row (a group is one or two whole rows)
            const int r = lane & 15;
            float a = db[0];
#pragma unroll
            for (int k = 1; k < DP1; ++k) a = r == k ? db[k] : a;
            const float t = tanhf(a);
            db[0] = __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(t), 0x150, 0xF, 0xF, false));
            if (DP1 > 1) db[1] = __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(t), 0x151, 0xF, 0xF, false));
            if (DP1 > 2) db[2] = __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(t), 0x152, 0xF, 0xF, false));
            if (DP1 > 3) db[3] = __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(t), 0x153, 0xF, 0xF, false));
            if (DP1 > 4) db[4] = __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(t), 0x154, 0xF, 0xF, false));
        } else {
#pragma unroll
            for (int k = 0; k < DP1; ++k) db[k] = tanhf(db[k]);
        }
        float4 f = f4(0.f);
#pragma unroll
        for (int k = 0; k < DP1; ++k) {
            const float wk = b[k] + db[k];
            f.x = fmaf(wk, x[k].x, f.x);
            f.y = fmaf(wk, x[k].y, f.y);
            f.z = fmaf(wk, x[k].z, f.z);
            f.w = fmaf(wk, x[k].w, f.w);
        }
        if (live && delta_out && j == 0) {
#pragma unroll
            for (int k = 0; k < DP1; ++k) delta_out[p * DP1 + k] = db[k];
        }
        if (!CLS) {
            if (live && has) reinterpret_cast<float4 *>(out)[p * NC + j] = f;
        } else {
            if (has) *reinterpret_cast<float4 *>(fb + (nsl + grp) * S + 4 * j) = f;
            if (j == 0) sb[nsl + grp] = live ? p : -1;
            nsl += PPW;
            if (nsl == 16) {
                score(16);
                nsl = 0;
            }
        }
    }
    if (CLS && nsl > 0) score(nsl);
}

template <int D, bool IN_BF16, int CH>
hipError_t launch_d(lattice *L, bool vec, int log2G, unsigned grid, const void *values, int C, const float *w_delta,
                    float b_delta, const float *w_cls, const float *b_cls, int n_cls, float *out, float *delta) {
#define DS_LAUNCH(VV, CC)                                                                                         \
    hipExtLaunchKernelGGL((k_deform_generic<D, VV, IN_BF16, CC, CH>), dim3(grid), dim3(kBlock), 0, L->stream,    \
                          L->kt_start, L->kt_stop, 0, L->m, C, log2G, L->idx, L->bary, values, w_delta, b_delta, \
                          w_cls, b_cls, n_cls, out, delta)
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

// The classifier kernels keep their weight fragments in registers for the
// whole launch: launch at most as many workgroups as stay resident (each
// wave then loads them once and loops over many points).
template <int D, int LG, bool IN_BF16, int NCB>
unsigned fast_grid(const lattice *L, unsigned grid) {
    if (NCB == 0) return grid;
    static std::atomic<int> per_cu{0};  // per instantiation; every device is a gfx950
    int n = per_cu.load(std::memory_order_relaxed);
    if (n == 0) {
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k_deform_fast<D, LG, IN_BF16, NCB>, kBlock, 0) !=
                hipSuccess ||
            n < 1)
            n = 1;
        per_cu.store(n, std::memory_order_relaxed);
    }
    const int64_t cap = (int64_t)n * L->cu_count;
    return grid < cap ? grid : (unsigned)cap;
}

template <int D, int LG, bool IN_BF16, int NCB>
hipError_t launch_fast1(lattice *L, unsigned grid, const void *values, int C, const float *w_delta, float b_delta,
                        const float *w_cls, const float *b_cls, int n_cls, float *out, float *delta) {
    hipExtLaunchKernelGGL((k_deform_fast<D, LG, IN_BF16, NCB>), dim3(fast_grid<D, LG, IN_BF16, NCB>(L, grid)),
                          dim3(kBlock), 0, L->stream, L->kt_start, L->kt_stop, 0, L->m, C, L->idx, L->bary, values,
                          w_delta, b_delta, w_cls, b_cls, n_cls, out, delta);
    return hipGetLastError();
}

template <int D, int LG, bool IN_BF16>
hipError_t launch_fast_ncb(lattice *L, int ncb, unsigned grid, const void *values, int C, const float *w_delta,
                           float b_delta, const float *w_cls, const float *b_cls, int n_cls, float *out,
                           float *delta) {
    switch (ncb) {
        case 0: return launch_fast1<D, LG, IN_BF16, 0>(L, grid, values, C, w_delta, b_delta, w_cls, b_cls, n_cls, out, delta);
        case 1: return launch_fast1<D, LG, IN_BF16, 1>(L, grid, values, C, w_delta, b_delta, w_cls, b_cls, n_cls, out, delta);
        case 2: return launch_fast1<D, LG, IN_BF16, 2>(L, grid, values, C, w_delta, b_delta, w_cls, b_cls, n_cls, out, delta);
        case 4: return launch_fast1<D, LG, IN_BF16, 4>(L, grid, values, C, w_delta, b_delta, w_cls, b_cls, n_cls, out, delta);
        default: return hipErrorInvalidValue;
    }
}

template <int D>
hipError_t launch_fast(lattice *L, bool bf, int lg, int ncb, unsigned grid, const void *values, int C,
                       const float *w_delta, float b_delta, const float *w_cls, const float *b_cls, int n_cls,
                       float *out, float *delta) {
#define DF_LG(LGV)                                                                                                  \
    case LGV:                                                                                                       \
        return bf ? launch_fast_ncb<D, LGV, true>(L, ncb, grid, values, C, w_delta, b_delta, w_cls, b_cls, n_cls, out, \
                                                  delta)                                                            \
                  : launch_fast_ncb<D, LGV, false>(L, ncb, grid, values, C, w_delta, b_delta, w_cls, b_cls, n_cls,   \
                                                   out, delta);
    switch (lg) {
        DF_LG(2)
        DF_LG(3)
        DF_LG(4)
        DF_LG(5)
        default: return hipErrorInvalidValue;
    }
#undef DF_LG
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
    if (vec && lanes <= 32 && (!w_cls || n_cls <= 64)) {
        int lg = 2;
        while ((1 << lg) < lanes) ++lg;
        const int64_t ppw = 64 >> lg;
        const unsigned grid = grid_for(((m + ppw - 1) / ppw) * 64, kBlock, L->cu_count, 16);
        const int ncb = !w_cls ? 0 : n_cls <= 16 ? 1 : n_cls <= 32 ? 2 : 4;
        switch (L->d) {
            case 1: return launch_fast<1>(L, bf, lg, ncb, grid, values, C, w_delta, b_delta, w_cls, b_cls, n_cls, out, delta);
            case 2: return launch_fast<2>(L, bf, lg, ncb, grid, values, C, w_delta, b_delta, w_cls, b_cls, n_cls, out, delta);
            case 3: return launch_fast<3>(L, bf, lg, ncb, grid, values, C, w_delta, b_delta, w_cls, b_cls, n_cls, out, delta);
            case 4: return launch_fast<4>(L, bf, lg, ncb, grid, values, C, w_delta, b_delta, w_cls, b_cls, n_cls, out, delta);
            default: return hipErrorInvalidValue;
        }
    }
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
