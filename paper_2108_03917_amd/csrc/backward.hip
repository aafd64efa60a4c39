// Backward passes of the lattice operations (Sec. "Implementation": the
// network is trained end to end, so each operation needs the gradient of a
// loss with respect to its inputs).  Every forward here is linear in the
// quantity differentiated, so each gradient is the transposed map:
//
//   slice  f_p = sum_k b_pk y_{v_k}      ->  dy_v = sum_{(p,k): v_k = v} b_pk df_p
//          (Eq. splat applied to df: the splat's pair-list gather, splat.hip)
//   splat  x_v = sum_p b_pv f_p          ->  df_p = sum_k b_pk dx_{v_k}
//          (Eq. slice applied to dx: the slice kernel, slice.hip; the
//          normalised splat divides dx_v by w_v first)
//   conv   y_v = sum_t x_{nbr(v,t)} W_t^T
//          dx_u = sum over (v, t) with nbr(v,t) = u of g_v W_t
//          dW_t = sum_v g_v^T x_{nbr(v,t)}
//
// Input gradient.  The 1-hop ring is symmetric (Sec. "Permutohedral
// Lattice": the neighbours sit at +-n_j): tap 1+j of v is u exactly when tap
// d+2+j of u is v, and tap 0 is the vertex itself.  So dx_u = sum_s
// g_{nbr(u,s)} W_{flip(s)}, a forward convolution of g with the weights
// W'[i][s][o] = W[o][flip(s)][i].  k_flip_weights builds W' and the forward
// conv kernels (conv.hip) run it: no scatter, no atomics.
//
// Weight gradient.  For each tap, dW_t [C_out x C_in] is a product whose
// reduction runs over the V vertices: A = g^T (rows of g, contiguous) and
// B = the gathered rows x_{nbr(v,t)}.  k_conv_wgrad gives each workgroup one
// tap, one 64 x 64 tile of (output, input) channels and one chunk of the
// vertices (chunk c of nch covers rows [c V / nch, (c+1) V / nch), V read on
// the device).  Per step of 32 vertices it stages the 32 g rows and the 32
// gathered x rows in LDS as fp32 and four wavefronts each accumulate a
// 32 x 32 block with v_mfma_f32_32x32x2f32 (K = the vertex index).  Each
// chunk writes its tile to a partial buffer; k_wgrad_reduce adds the nch
// partials in a fixed order, so the result does not depend on scheduling.
// The bias gradient (sum_v g_v) is summed from the same g rows by the
// workgroups of tap 0 and the first input tile.
#include "internal.h"

namespace {

typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kBlock = 256;
constexpr int kTile = 64;   // output and input channels per tile
constexpr int kStep = 32;   // vertices per K step
constexpr int kRowsPer = kStep / (kBlock / 16);  // rows each loader thread stages per step
constexpr int kWgPerCu = 4;  // weight-gradient workgroups per CU the chunk count aims at
// (32-row steps at four workgroups per CU measured best over 64 and 128 rows
// at two to eight workgroups per CU, on 64x64, 64x128 and 128x128 shapes)

// fp32 -> bf16 -> fp32, round to nearest with ties to even (NaN stays NaN).
__device__ __forceinline__ float round_bf16(float f) {
    const uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return __uint_as_float(u | 0x00400000u);
    return __uint_as_float((u + 0x7fffu + ((u >> 16) & 1u)) & 0xffff0000u);
}

// LDS tile [kStep][kTile] fp32.  Column c of an odd row sits at c ^ 32: the
// two 32-lane halves of an MFMA operand read (rows k and k+1, same columns)
// then fall on different banks.
__device__ __forceinline__ int swz(int k, int c) { return k * kTile + (c ^ ((k & 1) << 5)); }

// Four consecutive channels [c, c+4) of row `row` (fp32 or bf16 storage),
// zero past C.  VEC: C % 4 == 0 and the rows are 16-byte (fp32) or 8-byte
// (bf16) aligned.
template <bool BF16, bool VEC>
__device__ __forceinline__ float4 load4(const void *base, int64_t row, int C, int c) {
    float4 r = make_float4(0.f, 0.f, 0.f, 0.f);
    if (VEC) {
        if (c >= C) return r;
        if (BF16) {
            const uint2 u = *reinterpret_cast<const uint2 *>(reinterpret_cast<const uint16_t *>(base) + row * C + c);
            r.x = __uint_as_float(u.x << 16);
            r.y = __uint_as_float(u.x & 0xffff0000u);
            r.z = __uint_as_float(u.y << 16);
            r.w = __uint_as_float(u.y & 0xffff0000u);
        } else {
            r = *reinterpret_cast<const float4 *>(reinterpret_cast<const float *>(base) + row * C + c);
        }
        return r;
    }
    float v[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        v[e] = 0.f;
        if (c + e < C) {
            if (BF16)
                v[e] = __uint_as_float((uint32_t)reinterpret_cast<const uint16_t *>(base)[row * C + c + e] << 16);
            else
                v[e] = reinterpret_cast<const float *>(base)[row * C + c + e];
        }
    }
    return make_float4(v[0], v[1], v[2], v[3]);
}

template <bool G_BF16, bool X_BF16, bool ROUND, bool VEC>
__global__ __launch_bounds__(kBlock) void k_conv_wgrad(const void *__restrict__ g, int C_out,
                                                       const void *__restrict__ x, int C_in, int T,
                                                       const int32_t *__restrict__ nbr,
                                                       const int32_t *__restrict__ counters, int nch,
                                                       float *__restrict__ partial, float *__restrict__ pbias) {
    __shared__ float gs[kStep * kTile];
    __shared__ float xs[kStep * kTile];
    __shared__ float bred[kBlock / 16][kTile];

    const int64_t V = counters[CNT_V];
    const int chunk = blockIdx.x;
    const int t = blockIdx.y;
    const int tiles_i = (C_in + kTile - 1) / kTile;
    const int o0 = (blockIdx.z / tiles_i) * kTile;
    const int i0 = (blockIdx.z % tiles_i) * kTile;
    const int64_t lo = V * chunk / nch;
    const int64_t hi = V * (chunk + 1) / nch;
    const bool do_bias = pbias != nullptr && t == 0 && i0 == 0;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int h = lane >> 5;            // MFMA K index of this lane
    const int ow = (wave >> 1) * 32;    // this wave's 32 x 32 block
    const int iw = (wave & 1) * 32;
    // Loader mapping: thread owns channel chunk c4 (4 channels) of rows
    // r0, r0+16, r0+32, ... of the step.
    const int c4 = (tid & 15) * 4;
    const int r0 = tid >> 4;

    f32x16_t acc;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = 0.f;
    float bsum[4] = {0.f, 0.f, 0.f, 0.f};

    // The neighbour indices of a step are loaded one step before its rows,
    // so that a row gather never waits on its own index load.
    float4 ga[kRowsPer], xa[kRowsPer];
    int32_t ua[kRowsPer];
    auto load_index = [&](int64_t k0) {
#pragma unroll
        for (int j = 0; j < kRowsPer; ++j) {
            const int64_t v = k0 + r0 + 16 * j;
            ua[j] = v < hi ? nbr[v * T + t] : -1;
        }
    };
    auto load_step = [&](int64_t k0) {
#pragma unroll
        for (int j = 0; j < kRowsPer; ++j) {
            const int64_t v = k0 + r0 + 16 * j;
            ga[j] = make_float4(0.f, 0.f, 0.f, 0.f);
            xa[j] = make_float4(0.f, 0.f, 0.f, 0.f);
            if (v < hi) ga[j] = load4<G_BF16, VEC>(g, v, C_out, o0 + c4);
            if (ua[j] >= 0) xa[j] = load4<X_BF16, VEC>(x, ua[j], C_in, i0 + c4);
        }
    };
    if (lo < hi) {
        load_index(lo);
        load_step(lo);
        load_index(lo + kStep);
    }
    for (int64_t k0 = lo; k0 < hi; k0 += kStep) {
        // registers -> LDS (rounded to bf16 for a bf16 computation)
#pragma unroll
        for (int j = 0; j < kRowsPer; ++j) {
            const int k = r0 + 16 * j;
            float4 a = ga[j], b = xa[j];
            if (do_bias) {
                bsum[0] += a.x;
                bsum[1] += a.y;
                bsum[2] += a.z;
                bsum[3] += a.w;
            }
            // (rows stored as bf16 are already rounded)
            if (ROUND && !G_BF16) a = make_float4(round_bf16(a.x), round_bf16(a.y), round_bf16(a.z), round_bf16(a.w));
            if (ROUND && !X_BF16) b = make_float4(round_bf16(b.x), round_bf16(b.y), round_bf16(b.z), round_bf16(b.w));
            *reinterpret_cast<float4 *>(&gs[swz(k, c4)]) = a;
            *reinterpret_cast<float4 *>(&xs[swz(k, c4)]) = b;
        }
        __syncthreads();
        if (k0 + kStep < hi) {  // next step's loads in flight during the MFMAs
            load_step(k0 + kStep);
            load_index(k0 + 2 * kStep);
        }
#pragma unroll 8
        for (int s = 0; s < kStep / 2; ++s) {
            const int k = 2 * s + h;
            const float a = gs[swz(k, ow + (lane & 31))];
            const float b = xs[swz(k, iw + (lane & 31))];
            acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc, 0, 0, 0);
        }
        __syncthreads();
    }

    // Partial tile of this chunk: register r of lane l holds row
    // 8 (r / 4) + 4 (l / 32) + r % 4 (output channel), column l % 32 (input channel).
    const int64_t tapstride = C_in;
    float *dst = partial + (int64_t)chunk * C_out * T * C_in;
    const int ic = i0 + iw + (lane & 31);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int oc = o0 + ow + 8 * (r >> 2) + 4 * h + (r & 3);
        if (oc < C_out && ic < C_in) dst[((int64_t)oc * T + t) * tapstride + ic] = acc[r];
    }
    if (do_bias) {
#pragma unroll
        for (int e = 0; e < 4; ++e) bred[r0][c4 + e] = bsum[e];
        __syncthreads();
        if (tid < kTile) {
            float s = 0.f;
            for (int q = 0; q < kBlock / 16; ++q) s += bred[q][tid];
            if (o0 + tid < C_out) pbias[(int64_t)chunk * C_out + o0 + tid] = s;
        }
    }
}

// The bf16 computation on bf16 MFMA (v_mfma_f32_32x32x16_bf16): lane l
// supplies A[l % 32][8 (l / 32) + 0..7] and B[8 (l / 32) + 0..7][l % 32],
// eight consecutive K = vertex values per lane.  So the step's rows are
// staged transposed in LDS, channel-major with the 32 vertices of the step
// contiguous (row stride kTRow bytes): each thread loads two consecutive
// rows of four channels, packs the two bf16 values of each channel into one
// word and stores it at [channel][vertex pair].  Products of bf16 values are
// exact in fp32 and the sums are fp32, as in the fp32-MFMA kernel.
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kTStep = 32;   // vertices per step (two MFMA K-steps of 16)
constexpr int kTRow = 80;    // LDS bytes per channel row: 32 bf16 + 16 bytes of padding

// Four consecutive channels [c, c+4) of row `row` as bf16 bits (rounded to
// nearest even from fp32 storage), zero past C; C % 4 == 0 and aligned rows.
template <bool BF16>
__device__ __forceinline__ uint2 load4_bf16(const void *base, int64_t row, int C, int c) {
    if (c >= C) return make_uint2(0u, 0u);
    if (BF16) return *reinterpret_cast<const uint2 *>(reinterpret_cast<const uint16_t *>(base) + row * C + c);
    const float4 f = *reinterpret_cast<const float4 *>(reinterpret_cast<const float *>(base) + row * C + c);
    return make_uint2(bf16_bits(f.x) | (bf16_bits(f.y) << 16), bf16_bits(f.z) | (bf16_bits(f.w) << 16));
}

template <bool G_BF16, bool X_BF16>
__global__ __launch_bounds__(kBlock) void k_conv_wgrad_bf16(const void *__restrict__ g, int C_out,
                                                            const void *__restrict__ x, int C_in, int T,
                                                            const int32_t *__restrict__ nbr,
                                                            const int32_t *__restrict__ counters, int nch,
                                                            float *__restrict__ partial, float *__restrict__ pbias) {
    __shared__ __attribute__((aligned(16))) char gs[kTile * kTRow];
    __shared__ __attribute__((aligned(16))) char xs[kTile * kTRow];
    __shared__ float bred[kBlock / 16][kTile];

    const int64_t V = counters[CNT_V];
    const int chunk = blockIdx.x;
    const int t = blockIdx.y;
    const int tiles_i = (C_in + kTile - 1) / kTile;
    const int o0 = (blockIdx.z / tiles_i) * kTile;
    const int i0 = (blockIdx.z % tiles_i) * kTile;
    const int64_t lo = V * chunk / nch;
    const int64_t hi = V * (chunk + 1) / nch;
    const bool do_bias = pbias != nullptr && t == 0 && i0 == 0;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int h = lane >> 5;
    const int ow = (wave >> 1) * 32;
    const int iw = (wave & 1) * 32;
    // Loader mapping: channel chunk c4 (4 channels), rows 2 rp and 2 rp + 1 of the step.
    const int c4 = (tid & 15) * 4;
    const int rp = tid >> 4;

    f32x16_t acc;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = 0.f;
    float bsum[4] = {0.f, 0.f, 0.f, 0.f};

    uint2 ga[2], xa[2];
    int32_t ua[2];
    auto load_index = [&](int64_t k0) {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int64_t v = k0 + 2 * rp + j;
            ua[j] = v < hi ? nbr[v * T + t] : -1;
        }
    };
    auto load_step = [&](int64_t k0) {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int64_t v = k0 + 2 * rp + j;
            ga[j] = v < hi ? load4_bf16<G_BF16>(g, v, C_out, o0 + c4) : make_uint2(0u, 0u);
            xa[j] = ua[j] >= 0 ? load4_bf16<X_BF16>(x, ua[j], C_in, i0 + c4) : make_uint2(0u, 0u);
        }
    };
    // the bias sums the output gradient as stored (fp32 rows unrounded)
    auto add_bias = [&](int64_t k0) {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int64_t v = k0 + 2 * rp + j;
            if (v >= hi || o0 + c4 >= C_out) continue;
            if (G_BF16) {
                const uint2 u = ga[j];
                bsum[0] += __uint_as_float(u.x << 16);
                bsum[1] += __uint_as_float(u.x & 0xffff0000u);
                bsum[2] += __uint_as_float(u.y << 16);
                bsum[3] += __uint_as_float(u.y & 0xffff0000u);
            } else {
                const float4 f =
                    *reinterpret_cast<const float4 *>(reinterpret_cast<const float *>(g) + v * C_out + o0 + c4);
                bsum[0] += f.x;
                bsum[1] += f.y;
                bsum[2] += f.z;
                bsum[3] += f.w;
            }
        }
    };
    if (lo < hi) {
        load_index(lo);
        load_step(lo);
        load_index(lo + kTStep);
    }
    for (int64_t k0 = lo; k0 < hi; k0 += kTStep) {
        if (do_bias) add_bias(k0);
        // registers -> LDS: word e of a thread = channel c4 + e of rows 2 rp, 2 rp + 1
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int sh = (e & 1) * 16;
            const uint32_t gw = ((((e < 2) ? ga[0].x : ga[0].y) >> sh) & 0xffffu) |
                                ((((e < 2) ? ga[1].x : ga[1].y) >> sh) << 16);
            const uint32_t xw = ((((e < 2) ? xa[0].x : xa[0].y) >> sh) & 0xffffu) |
                                ((((e < 2) ? xa[1].x : xa[1].y) >> sh) << 16);
            *reinterpret_cast<uint32_t *>(gs + (c4 + e) * kTRow + 4 * rp) = gw;
            *reinterpret_cast<uint32_t *>(xs + (c4 + e) * kTRow + 4 * rp) = xw;
        }
        __syncthreads();
        if (k0 + kTStep < hi) {
            load_step(k0 + kTStep);
            load_index(k0 + 2 * kTStep);
        }
#pragma unroll
        for (int s = 0; s < kTStep / 16; ++s) {
            const u32x4_t a = *reinterpret_cast<const u32x4_t *>(gs + (ow + (lane & 31)) * kTRow + 32 * s + 16 * h);
            const u32x4_t b = *reinterpret_cast<const u32x4_t *>(xs + (iw + (lane & 31)) * kTRow + 32 * s + 16 * h);
            acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                          __builtin_bit_cast(bf16x8_t, b), acc, 0, 0, 0);
        }
        __syncthreads();
    }

    float *dst = partial + (int64_t)chunk * C_out * T * C_in;
    const int ic = i0 + iw + (lane & 31);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int oc = o0 + ow + 8 * (r >> 2) + 4 * h + (r & 3);
        if (oc < C_out && ic < C_in) dst[((int64_t)oc * T + t) * C_in + ic] = acc[r];
    }
    if (do_bias) {
        // threads tid and tid + 16 k (k = 0..15) share channel chunk c4
#pragma unroll
        for (int e = 0; e < 4; ++e) bred[rp][c4 + e] = bsum[e];
        __syncthreads();
        if (tid < kTile) {
            float sacc = 0.f;
            for (int q = 0; q < kBlock / 16; ++q) sacc += bred[q][tid];
            if (o0 + tid < C_out) pbias[(int64_t)chunk * C_out + o0 + tid] = sacc;
        }
    }
}

// out[j] = sum over the nch chunk partials part[c][j], in a fixed order:
// a workgroup owns 64 consecutive outputs; its four wavefronts sum the
// chunks c = g, g+4, g+8, ... (g = wavefront) with four loads in flight, and
// the four group sums are added in group order.
constexpr int kRedCols = 64;
__global__ __launch_bounds__(kBlock) void k_wgrad_reduce(const float *__restrict__ part, int nch, int64_t n,
                                                         float *__restrict__ out) {
    __shared__ float red[kBlock / kRedCols][kRedCols];
    const int g = threadIdx.x / kRedCols;
    const int64_t j = (int64_t)blockIdx.x * kRedCols + (threadIdx.x % kRedCols);
    float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
    if (j < n) {
        constexpr int G = kBlock / kRedCols;
        int c = g;
        for (; c + 3 * G < nch; c += 4 * G) {
            s0 += part[(int64_t)c * n + j];
            s1 += part[(int64_t)(c + G) * n + j];
            s2 += part[(int64_t)(c + 2 * G) * n + j];
            s3 += part[(int64_t)(c + 3 * G) * n + j];
        }
        for (; c < nch; c += G) s0 += part[(int64_t)c * n + j];
    }
    red[g][threadIdx.x % kRedCols] = (s0 + s1) + (s2 + s3);
    __syncthreads();
    if (g == 0 && j < n) {
        float t = 0.f;
        for (int q = 0; q < kBlock / kRedCols; ++q) t += red[q][threadIdx.x];
        out[j] = t;
    }
}

// W'[i][s][o] = W[o][flip(s)][i]; flip(0) = 0, flip(1+j) = d+2+j, flip(d+2+j) = 1+j.
template <typename E>
__global__ __launch_bounds__(kBlock) void k_flip_weights(const E *__restrict__ w, int C_out, int T, int C_in,
                                                         E *__restrict__ wt) {
    const int64_t n = (int64_t)C_out * T * C_in;
    const int half = (T - 1) / 2;  // d + 1
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t q = (int64_t)blockIdx.x * kBlock + threadIdx.x; q < n; q += stride) {
        // q indexes W' [C_in][T][C_out]
        const int o = (int)(q % C_out);
        const int s = (int)((q / C_out) % T);
        const int i = (int)(q / ((int64_t)C_out * T));
        const int fs = s == 0 ? 0 : (s <= half ? s + half : s - half);
        wt[q] = w[((int64_t)o * T + fs) * C_in + i];
    }
}

}  // namespace

// Number of vertex chunks of the weight gradient: about kWgPerCu workgroups
// per CU over all taps and tiles, a multiple of 8 (the chunk's workgroups of
// every tap then share one XCD's L2), and no more chunks than steps of 64
// rows in the largest lattice.
int wgrad_chunks(const lattice *L, int C_in, int C_out) {
    const int64_t tiles = (int64_t)((C_out + kTile - 1) / kTile) * ((C_in + kTile - 1) / kTile) * L->T;
    int64_t nch = (kWgPerCu * (int64_t)L->cu_count + tiles - 1) / tiles;
    nch = (nch + 7) / 8 * 8;
    const int64_t steps = (L->max_vertices + kStep - 1) / kStep;
    if (nch > steps) nch = steps;
    if (nch < 1) nch = 1;
    if (nch > 1024) nch = 1024;
    return (int)nch;
}

hipError_t launch_conv_wgrad(lattice *L, const void *g, lattice_dtype g_dt, int C_out, const void *x,
                             lattice_dtype x_dt, int C_in, lattice_dtype dt, int nch, float *partial,
                             float *pbias, float *grad_w, float *grad_bias) {
    const bool gb = g_dt == LATTICE_BF16, xb = x_dt == LATTICE_BF16, rnd = dt == LATTICE_BF16;
    const bool vec = C_out % 4 == 0 && C_in % 4 == 0 && (reinterpret_cast<uintptr_t>(g) & (gb ? 7 : 15)) == 0 &&
                     (reinterpret_cast<uintptr_t>(x) & (xb ? 7 : 15)) == 0;
    const dim3 grid((unsigned)nch, (unsigned)L->T,
                    (unsigned)(((C_out + kTile - 1) / kTile) * ((C_in + kTile - 1) / kTile)));
    if (rnd && vec) {
        // bf16 computation on bf16 MFMA
        if (gb && xb)
            hipLaunchKernelGGL((k_conv_wgrad_bf16<true, true>), grid, dim3(kBlock), 0, L->stream, g, C_out, x, C_in,
                               L->T, L->nbr, L->counters, nch, partial, grad_bias ? pbias : nullptr);
        else if (gb)
            hipLaunchKernelGGL((k_conv_wgrad_bf16<true, false>), grid, dim3(kBlock), 0, L->stream, g, C_out, x, C_in,
                               L->T, L->nbr, L->counters, nch, partial, grad_bias ? pbias : nullptr);
        else if (xb)
            hipLaunchKernelGGL((k_conv_wgrad_bf16<false, true>), grid, dim3(kBlock), 0, L->stream, g, C_out, x, C_in,
                               L->T, L->nbr, L->counters, nch, partial, grad_bias ? pbias : nullptr);
        else
            hipLaunchKernelGGL((k_conv_wgrad_bf16<false, false>), grid, dim3(kBlock), 0, L->stream, g, C_out, x,
                               C_in, L->T, L->nbr, L->counters, nch, partial, grad_bias ? pbias : nullptr);
    } else {
#define WG(GB, XB, RN, VC)                                                                                      \
    hipLaunchKernelGGL((k_conv_wgrad<GB, XB, RN, VC>), grid, dim3(kBlock), 0, L->stream, g, C_out, x, C_in, L->T, \
                       L->nbr, L->counters, nch, partial, grad_bias ? pbias : nullptr)
#define WG_V(GB, XB, RN) \
    if (vec)             \
        WG(GB, XB, RN, true); \
    else                 \
        WG(GB, XB, RN, false)
    if (gb) {
        if (xb) { WG_V(true, true, true); }
        else if (rnd) { WG_V(true, false, true); }
        else { WG_V(true, false, false); }
    } else {
        if (xb) { if (rnd) { WG_V(false, true, true); } else { WG_V(false, true, false); } }
        else if (rnd) { WG_V(false, false, true); }
        else { WG_V(false, false, false); }
    }
#undef WG_V
#undef WG
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (grad_w) {
        const int64_t n = (int64_t)C_out * L->T * C_in;
        hipLaunchKernelGGL(k_wgrad_reduce, dim3((unsigned)((n + kRedCols - 1) / kRedCols)), dim3(kBlock), 0,
                           L->stream, partial, nch, n, grad_w);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (grad_bias) {
        hipLaunchKernelGGL(k_wgrad_reduce, dim3((unsigned)((C_out + kRedCols - 1) / kRedCols)), dim3(kBlock), 0,
                           L->stream, pbias, nch, (int64_t)C_out, grad_bias);
        e = hipGetLastError();
    }
    return e;
}

hipError_t launch_flip_weights(lattice *L, const void *w, bool bf16, int C_out, int C_in, void *wt) {
    const int64_t n = (int64_t)C_out * L->T * C_in;
    const unsigned grid = grid_for(n, kBlock, L->cu_count, 2);
    if (bf16)
        hipLaunchKernelGGL(k_flip_weights<uint16_t>, dim3(grid), dim3(kBlock), 0, L->stream,
                           reinterpret_cast<const uint16_t *>(w), C_out, L->T, C_in, reinterpret_cast<uint16_t *>(wt));
    else
        hipLaunchKernelGGL(k_flip_weights<float>, dim3(grid), dim3(kBlock), 0, L->stream,
                           reinterpret_cast<const float *>(w), C_out, L->T, C_in, reinterpret_cast<float *>(wt));
    return hipGetLastError();
}
