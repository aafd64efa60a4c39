// Backward of DeformSlice and its fused classifier (Sec. "Proposed
// Operations", DeformSlicing, Eq. deformSlice; Sec. "Implementation": the
// network is trained end to end).  With the forward
//
//   q_pk  = b_pk x_k,  mx_p = max_k q_pk,  db_pk = tanh(b_delta + (q_pk - mx_p) . w_delta),
//   f_p   = sum_k (b_pk + db_pk) x_k,  out_p = f_p  or  f_p W_cls^T + b_cls
//
// (x_k the row of vertex v_pk) and g_p = dL/dout_p, the gradients are
//
//   gf_p      = g_p W_cls  (or g_p)             dW_cls = sum_p g_p^T f_p,  db_cls = sum_p g_p
//   darg_pk   = (gf_p . x_k) (1 - db_pk^2)      S_p = sum_k darg_pk
//   dw_delta  = sum_pk darg_pk (q_pk - mx_p)    db_delta = sum_pk darg_pk
//   dx_pk[c]  = (b_pk + db_pk) gf_p[c] + b_pk w_delta[c] (darg_pk - [k = k*_pc] S_p)
//   dX_v      = sum of dx_pk over the pairs (p, k) with v_pk = v
//
// where k*_pc is the vertex that wins the max of channel c (the first of
// equal maxima of the float32 products b x, as the forward computes them).
//
//   k_dfb_points   one wavefront per point, lane = channel (CH chunks of 64):
//                  recomputes the forward, writes gf_p and k*_p (one byte per
//                  channel), the pair coefficients (b + db, b darg, b S) and,
//                  with the classifier, f_p; accumulates dw_delta and db_delta
//                  per wavefront (written as partials at the end).
//   k_dfb_gather   one wavefront per vertex over its pair list (the splat's
//                  lists: no atomics), lane = channel.
//   k_dfb_cls      dW_cls and db_cls partials per chunk of points.
//   k_dfb_reduce   every partial added in a fixed order: the results do not
//                  depend on scheduling.
#include "internal.h"

namespace {

constexpr int kBlock = 256;

__device__ __forceinline__ float wave_sum_f(float x) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off, 64);
    return x;
}

template <bool IN_BF16>
__device__ __forceinline__ float value_at(const void *values, int64_t at) {
    if (IN_BF16) return __uint_as_float((uint32_t)reinterpret_cast<const uint16_t *>(values)[at] << 16);
    return reinterpret_cast<const float *>(values)[at];
}

// Scratch carved out of one buffer (offsets in bytes, each 256-aligned).
struct DfbLayout {
    int64_t gf, am, coef, f, pw, pb, pc, pbc, total;
};

__host__ __device__ inline int64_t align256(int64_t x) { return (x + 255) / 256 * 256; }

inline DfbLayout dfb_layout(int64_t m, int C, int dp1, int n_cls, int nwaves, int nch) {
    DfbLayout l;
    int64_t at = 0;
    l.gf = at;   at += align256(m * C * 4);
    l.am = at;   at += align256(m * C);
    l.coef = at; at += align256(m * dp1 * 3 * 4);
    l.f = at;    at += n_cls > 0 ? align256(m * C * 4) : 0;
    l.pw = at;   at += align256((int64_t)nwaves * C * 4);
    l.pb = at;   at += align256((int64_t)nwaves * 4);
    l.pc = at;   at += n_cls > 0 ? align256((int64_t)nch * n_cls * C * 4) : 0;
    l.pbc = at;  at += n_cls > 0 ? align256((int64_t)nch * n_cls * 4) : 0;
    l.total = at;
    return l;
}

template <int D, bool IN_BF16, bool CLS, int CH>
__global__ __launch_bounds__(kBlock) void k_dfb_points(int64_t m, int C, const int32_t *__restrict__ idx,
                                                       const float *__restrict__ bary, const void *__restrict__ values,
                                                       const float *__restrict__ w_delta, float b_delta,
                                                       const float *__restrict__ w_cls, int n_cls,
                                                       const float *__restrict__ grad_out, float *__restrict__ gf_out,
                                                       uint8_t *__restrict__ am_out, float *__restrict__ coef,
                                                       float *__restrict__ f_out, float *__restrict__ part_w,
                                                       float *__restrict__ part_b) {
    constexpr int DP1 = D + 1;
    const int lane = threadIdx.x & 63;
    const int64_t wave = ((int64_t)blockIdx.x * kBlock + threadIdx.x) >> 6;
    const int64_t nwaves = ((int64_t)gridDim.x * kBlock) >> 6;

    float wd[CH], acc_w[CH];
#pragma unroll
    for (int i = 0; i < CH; ++i) {
        const int c = lane + 64 * i;
        wd[i] = c < C ? w_delta[c] : 0.f;
        acc_w[i] = 0.f;
    }
    float acc_b = 0.f;

    for (int64_t p = wave; p < m; p += nwaves) {
        int v[DP1];
        float b[DP1];
#pragma unroll
        for (int k = 0; k < DP1; ++k) {
            v[k] = idx[p * DP1 + k];
            b[k] = bary[p * DP1 + k];
        }
        float x[DP1][CH];
#pragma unroll
        for (int k = 0; k < DP1; ++k)
#pragma unroll
            for (int i = 0; i < CH; ++i) {
                const int c = lane + 64 * i;
                x[k][i] = (c < C && v[k] >= 0) ? value_at<IN_BF16>(values, (int64_t)v[k] * C + c) : 0.f;
            }
        // MaxPool with the winning vertex (first of equal maxima)
        float mx[CH];
        int am[CH];
#pragma unroll
        for (int i = 0; i < CH; ++i) {
            mx[i] = b[0] * x[0][i];
            am[i] = 0;
#pragma unroll
            for (int k = 1; k < DP1; ++k) {
                const float q = b[k] * x[k][i];
                if (q > mx[i]) {
                    mx[i] = q;
                    am[i] = k;
                }
            }
        }
        // the offsets, as the forward computes them
        float db[DP1];
#pragma unroll
        for (int k = 0; k < DP1; ++k) {
            float s = 0.f;
#pragma unroll
            for (int i = 0; i < CH; ++i) s = fmaf(b[k] * x[k][i] - mx[i], wd[i], s);
            db[k] = tanhf(b_delta + wave_sum_f(s));
        }
        // gf = g W_cls (classifier) or g
        float gf[CH];
#pragma unroll
        for (int i = 0; i < CH; ++i) {
            const int c = lane + 64 * i;
            gf[i] = 0.f;
            if (!CLS && c < C) gf[i] = grad_out[p * C + c];
        }
        if (CLS) {
            for (int cls = 0; cls < n_cls; ++cls) {
                const float g = grad_out[p * n_cls + cls];
#pragma unroll
                for (int i = 0; i < CH; ++i) {
                    const int c = lane + 64 * i;
                    if (c < C) gf[i] = fmaf(g, w_cls[(int64_t)cls * C + c], gf[i]);
                }
            }
        }
        // Tanh backward, and S
        float darg[DP1];
        float S = 0.f;
#pragma unroll
        for (int k = 0; k < DP1; ++k) {
            float s = 0.f;
#pragma unroll
            for (int i = 0; i < CH; ++i) s = fmaf(gf[i], x[k][i], s);
            darg[k] = wave_sum_f(s) * (1.f - db[k] * db[k]);
            S += darg[k];
        }
        // Linear backward, accumulated per lane channel
#pragma unroll
        for (int i = 0; i < CH; ++i)
#pragma unroll
            for (int k = 0; k < DP1; ++k) acc_w[i] = fmaf(darg[k], b[k] * x[k][i] - mx[i], acc_w[i]);
        acc_b += S;
        // per-point records for the vertex gather and the classifier
#pragma unroll
        for (int i = 0; i < CH; ++i) {
            const int c = lane + 64 * i;
            if (c < C) {
                gf_out[p * C + c] = gf[i];
                am_out[p * C + c] = (uint8_t)am[i];
                if (CLS) {
                    float f = 0.f;
#pragma unroll
                    for (int k = 0; k < DP1; ++k) f = fmaf(b[k] + db[k], x[k][i], f);
                    f_out[p * C + c] = f;
                }
            }
        }
#pragma unroll
        for (int k = 0; k < DP1; ++k)
            if (lane == k) {
                coef[(p * DP1 + k) * 3 + 0] = b[k] + db[k];
                coef[(p * DP1 + k) * 3 + 1] = b[k] * darg[k];
                coef[(p * DP1 + k) * 3 + 2] = b[k] * S;
            }
    }
#pragma unroll
    for (int i = 0; i < CH; ++i) {
        const int c = lane + 64 * i;
        if (c < C) part_w[wave * C + c] = acc_w[i];
    }
    if (lane == 0) part_b[wave] = acc_b;
}

// dX_v over v's pair list: for pair (p, b) the slot k of v in p's simplex,
// then dx_pk.  Four entries' loads are issued together.
template <int D, int CH, bool OUT_BF16>
__global__ __launch_bounds__(kBlock) void k_dfb_gather(const int32_t *__restrict__ counters, int C,
                                                       const int32_t *__restrict__ vinfo,
                                                       const int32_t *__restrict__ list,
                                                       const int32_t *__restrict__ idx, const float *__restrict__ coef,
                                                       const float *__restrict__ gf, const uint8_t *__restrict__ am,
                                                       const float *__restrict__ w_delta, void *__restrict__ out) {
    constexpr int DP1 = D + 1;
    constexpr int U = 4;
    const int lane = threadIdx.x & 63;
    const int64_t V = counters[CNT_V];
    float wd[CH];
#pragma unroll
    for (int i = 0; i < CH; ++i) {
        const int c = lane + 64 * i;
        wd[i] = c < C ? w_delta[c] : 0.f;
    }
    const XcdShare sh = xcd_share(V);
    for (int64_t v = sh.lo + sh.wave; v < sh.hi; v += sh.nwaves) {
        const int64_t off = vinfo[2 * v];
        const int cnt = vinfo[2 * v + 1];
        float acc[CH], accw[CH];
#pragma unroll
        for (int i = 0; i < CH; ++i) acc[i] = accw[i] = 0.f;
        for (int e0 = 0; e0 < cnt; e0 += U) {
            int64_t p[U];
            int k[U];
            bool ok[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                ok[u] = e0 + u < cnt;
                p[u] = ok[u] ? list[2 * (off + e0 + u)] : 0;
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                k[u] = 0;
#pragma unroll
                for (int j = 0; j < DP1; ++j)
                    if (idx[p[u] * DP1 + j] == (int32_t)v) k[u] = j;
            }
            float al[U], be[U], ga[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const float *cf = coef + (p[u] * DP1 + k[u]) * 3;
                al[u] = ok[u] ? cf[0] : 0.f;
                be[u] = ok[u] ? cf[1] : 0.f;
                ga[u] = ok[u] ? cf[2] : 0.f;
            }
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int i = 0; i < CH; ++i) {
                    const int c = lane + 64 * i;
                    if (c < C) {
                        const float g = gf[p[u] * C + c];
                        const bool win = am[p[u] * C + c] == k[u];
                        acc[i] = fmaf(al[u], g, acc[i]);
                        accw[i] += win ? be[u] - ga[u] : be[u];
                    }
                }
        }
#pragma unroll
        for (int i = 0; i < CH; ++i) {
            const int c = lane + 64 * i;
            if (c < C) {
                const float r = fmaf(wd[i], accw[i], acc[i]);
                if (OUT_BF16)
                    reinterpret_cast<uint16_t *>(out)[v * C + c] = (uint16_t)bf16_bits(r);
                else
                    reinterpret_cast<float *>(out)[v * C + c] = r;
            }
        }
    }
}

// Classifier gradients, chunk `blockIdx.y` of the points and classes
// 4 blockIdx.x .. +3: each thread owns channels c = threadIdx.x + 256 i.
__global__ __launch_bounds__(kBlock) void k_dfb_cls(int64_t m, int C, int n_cls, int nch,
                                                    const float *__restrict__ grad_out, const float *__restrict__ f,
                                                    float *__restrict__ part_c, float *__restrict__ part_bc) {
    const int cls0 = blockIdx.x * 4;
    const int ch = blockIdx.y;
    const int64_t p0 = m * ch / nch, p1 = m * (ch + 1) / nch;
    for (int c = threadIdx.x; c < C; c += kBlock) {
        float acc[4] = {0.f, 0.f, 0.f, 0.f};
        for (int64_t p = p0; p < p1; ++p) {
            const float fv = f[p * C + c];
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (cls0 + j < n_cls) acc[j] = fmaf(grad_out[p * n_cls + cls0 + j], fv, acc[j]);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (cls0 + j < n_cls) part_c[((int64_t)ch * n_cls + cls0 + j) * C + c] = acc[j];
    }
    if (threadIdx.x < 4 && cls0 + (int)threadIdx.x < n_cls) {
        const int cls = cls0 + threadIdx.x;
        float s = 0.f;
        for (int64_t p = p0; p < p1; ++p) s += grad_out[p * n_cls + cls];
        part_bc[(int64_t)ch * n_cls + cls] = s;
    }
}

// out[j] = sum over r < rows of part[r * n + j], in order of r.
__global__ __launch_bounds__(kBlock) void k_dfb_reduce(const float *__restrict__ part, int64_t rows, int64_t n,
                                                       float *__restrict__ out) {
    const int64_t j = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (j >= n) return;
    float s = 0.f;
    for (int64_t r = 0; r < rows; ++r) s += part[r * n + j];
    out[j] = s;
}

template <int D, bool IN_BF16, bool CLS>
hipError_t launch_points_ch(lattice *L, int ch, unsigned grid, const void *values, int C, const float *w_delta,
                            float b_delta, const float *w_cls, int n_cls, const float *grad_out, float *gf,
                            uint8_t *am, float *coef, float *f, float *pw, float *pb) {
    auto go = [&](auto kern) {
        hipLaunchKernelGGL(kern, dim3(grid), dim3(kBlock), 0, L->stream, L->m, C, L->idx, L->bary, values, w_delta,
                           b_delta, w_cls, n_cls, grad_out, gf, am, coef, f, pw, pb);
        return hipGetLastError();
    };
    switch (ch) {
        case 1: return go(k_dfb_points<D, IN_BF16, CLS, 1>);
        case 2: return go(k_dfb_points<D, IN_BF16, CLS, 2>);
        case 4: return go(k_dfb_points<D, IN_BF16, CLS, 4>);
        case 8: return go(k_dfb_points<D, IN_BF16, CLS, 8>);
        default: return go(k_dfb_points<D, IN_BF16, CLS, 16>);
    }
}

template <int D>
hipError_t launch_gather_ch(lattice *L, int ch, bool out_bf16, int C, const float *coef, const float *gf,
                            const uint8_t *am, const float *w_delta, void *out) {
    const int64_t waves = L->max_vertices;
    int64_t grid = (waves + 3) / 4;
    const int64_t cap = (int64_t)L->cu_count * 8;
    if (grid > cap) grid = cap;
    grid = (grid + 7) / 8 * 8;  // whole XCD groups: each XCD takes one range of vertices
    auto go = [&](auto kern) {
        hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(kBlock), 0, L->stream, L->counters, C, L->vinfo, L->list,
                           L->idx, coef, gf, am, w_delta, out);
        return hipGetLastError();
    };
#define DFB_G(CHV)                                                                        \
    case CHV:                                                                             \
        return out_bf16 ? go(k_dfb_gather<D, CHV, true>) : go(k_dfb_gather<D, CHV, false>);
    switch (ch) {
        DFB_G(1)
        DFB_G(2)
        DFB_G(4)
        DFB_G(8)
        default:
            return out_bf16 ? go(k_dfb_gather<D, 16, true>) : go(k_dfb_gather<D, 16, false>);
    }
#undef DFB_G
}

template <int D>
hipError_t run_d(lattice *L, const void *values, bool in_bf16, int C, const float *w_delta, float b_delta,
                 const float *w_cls, int n_cls, const float *grad_out, void *grad_values, bool out_bf16,
                 float *grad_w_delta, float *grad_b_delta, float *grad_w_cls, float *grad_b_cls, char *scratch,
                 int nwaves, int nch) {
    const int ch = C <= 64 ? 1 : C <= 128 ? 2 : C <= 256 ? 4 : C <= 512 ? 8 : 16;
    const DfbLayout l = dfb_layout(L->m, C, D + 1, w_cls ? n_cls : 0, nwaves, nch);
    float *gf = reinterpret_cast<float *>(scratch + l.gf);
    uint8_t *am = reinterpret_cast<uint8_t *>(scratch + l.am);
    float *coef = reinterpret_cast<float *>(scratch + l.coef);
    float *f = w_cls ? reinterpret_cast<float *>(scratch + l.f) : nullptr;
    float *pw = reinterpret_cast<float *>(scratch + l.pw);
    float *pb = reinterpret_cast<float *>(scratch + l.pb);
    const unsigned grid = (unsigned)(nwaves / 4);
    hipError_t e;
    if (w_cls)
        e = in_bf16 ? launch_points_ch<D, true, true>(L, ch, grid, values, C, w_delta, b_delta, w_cls, n_cls, grad_out,
                                                      gf, am, coef, f, pw, pb)
                    : launch_points_ch<D, false, true>(L, ch, grid, values, C, w_delta, b_delta, w_cls, n_cls,
                                                       grad_out, gf, am, coef, f, pw, pb);
    else
        e = in_bf16 ? launch_points_ch<D, true, false>(L, ch, grid, values, C, w_delta, b_delta, w_cls, 0, grad_out,
                                                       gf, am, coef, f, pw, pb)
                    : launch_points_ch<D, false, false>(L, ch, grid, values, C, w_delta, b_delta, w_cls, 0, grad_out,
                                                        gf, am, coef, f, pw, pb);
    if (e != hipSuccess) return e;
    if (grad_values && (e = launch_gather_ch<D>(L, ch, out_bf16, C, coef, gf, am, w_delta, grad_values)) != hipSuccess)
        return e;
    if (grad_w_delta) {
        hipLaunchKernelGGL(k_dfb_reduce, dim3((C + kBlock - 1) / kBlock), dim3(kBlock), 0, L->stream, pw,
                           (int64_t)nwaves, (int64_t)C, grad_w_delta);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (grad_b_delta) {
        hipLaunchKernelGGL(k_dfb_reduce, dim3(1), dim3(kBlock), 0, L->stream, pb, (int64_t)nwaves, (int64_t)1,
                           grad_b_delta);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (w_cls && (grad_w_cls || grad_b_cls)) {
        float *pc = reinterpret_cast<float *>(scratch + l.pc);
        float *pbc = reinterpret_cast<float *>(scratch + l.pbc);
        hipLaunchKernelGGL(k_dfb_cls, dim3((unsigned)((n_cls + 3) / 4), (unsigned)nch), dim3(kBlock), 0, L->stream,
                           L->m, C, n_cls, nch, grad_out, f, pc, pbc);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if (grad_w_cls) {
            const int64_t n = (int64_t)n_cls * C;
            hipLaunchKernelGGL(k_dfb_reduce, dim3((unsigned)((n + kBlock - 1) / kBlock)), dim3(kBlock), 0, L->stream,
                               pc, (int64_t)nch, n, grad_w_cls);
            if ((e = hipGetLastError()) != hipSuccess) return e;
        }
        if (grad_b_cls) {
            hipLaunchKernelGGL(k_dfb_reduce, dim3((unsigned)((n_cls + kBlock - 1) / kBlock)), dim3(kBlock), 0,
                               L->stream, pbc, (int64_t)nch, (int64_t)n_cls, grad_b_cls);
            if ((e = hipGetLastError()) != hipSuccess) return e;
        }
    }
    return hipSuccess;
}

}  // namespace

// Wavefronts of the point kernel and point chunks of the classifier kernel.
void deform_backward_shape(const lattice *L, int *nwaves, int *nch) {
    *nwaves = L->cu_count * 4 * 4;  // four workgroups of four wavefronts per CU
    int64_t c = L->m / 1024;
    if (c < 1) c = 1;
    if (c > 256) c = 256;
    *nch = (int)c;
}

int64_t deform_backward_scratch_bytes(const lattice *L, int C, int n_cls) {
    int nwaves, nch;
    deform_backward_shape(L, &nwaves, &nch);
    return dfb_layout(L->m, C, L->d + 1, n_cls, nwaves, nch).total;
}

hipError_t launch_deform_backward(lattice *L, const void *values, lattice_dtype values_dt, int C,
                                  const float *w_delta, float b_delta, const float *w_cls, int n_cls,
                                  const float *grad_out, void *grad_values, lattice_dtype grad_dt,
                                  float *grad_w_delta, float *grad_b_delta, float *grad_w_cls, float *grad_b_cls,
                                  void *scratch) {
    int nwaves, nch;
    deform_backward_shape(L, &nwaves, &nch);
    const bool in_bf16 = values_dt == LATTICE_BF16, out_bf16 = grad_dt == LATTICE_BF16;
    char *s = reinterpret_cast<char *>(scratch);
    switch (L->d) {
#define DFB_D(DD)                                                                                              \
    case DD:                                                                                                   \
        return run_d<DD>(L, values, in_bf16, C, w_delta, b_delta, w_cls, n_cls, grad_out, grad_values, out_bf16, \
                         grad_w_delta, grad_b_delta, grad_w_cls, grad_b_cls, s, nwaves, nch);
        DFB_D(1)
        DFB_D(2)
        DFB_D(3)
        DFB_D(4)
#undef DFB_D
        default:
            return hipErrorInvalidValue;
    }
}
