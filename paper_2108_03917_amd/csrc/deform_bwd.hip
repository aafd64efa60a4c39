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
//   k_dfb_cls      dW_cls and db_cls partials per chunk of 256 points, on
//                  fp32 MFMA: a wavefront per chunk and tile of 32 classes x
//                  32 channels, the chunk's g and f rows as the operands.
//   rowsum         every partial added in a fixed order: the results do not
//                  depend on scheduling.
#include "internal.h"
#include "rowsum.h"

namespace {

constexpr int kBlock = 256;
constexpr int kClsLdsFloats = 4096;  // classifier weights staged in LDS up to 16 KB (occupancy kept)
constexpr int kDxRows1 = 8;          // list entries whose gf and am rows are loaded together, C <= 64

// N wavefront sums at once (each step of the N butterflies issued together).
template <int N>
__device__ __forceinline__ void wave_sum_n(float *x) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        float y[N];
#pragma unroll
        for (int k = 0; k < N; ++k) y[k] = __shfl_xor(x[k], off, 64);
#pragma unroll
        for (int k = 0; k < N; ++k) x[k] += y[k];
    }
}

template <bool IN_BF16>
__device__ __forceinline__ float value_at(const void *values, int64_t at) {
    if (IN_BF16) return __uint_as_float((uint32_t)reinterpret_cast<const uint16_t *>(values)[at] << 16);
    return reinterpret_cast<const float *>(values)[at];
}

// Scratch carved out of one buffer (offsets in bytes, each 256-aligned).
struct DfbLayout {
    int64_t gf, am, coef, f, pw, pb, pc, pbc, tmp, part, total;
};

__host__ __device__ inline int64_t align256(int64_t x) { return (x + 255) / 256 * 256; }

inline DfbLayout dfb_layout(int64_t m, int C, int dp1, int n_cls, int nwaves, int nch, int64_t part_rows) {
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
    // the row sums' chunk sums, for the largest of the four reductions
    int64_t t = rowsum::scratch_floats(nwaves, C);
    if (n_cls > 0 && rowsum::scratch_floats(nch, (int64_t)n_cls * C) > t) t = rowsum::scratch_floats(nch, (int64_t)n_cls * C);
    l.tmp = at;  at += align256(t * 4);
    l.part = at; at += align256(part_rows * 2 * C * 4);  // the long lists' part rows: acc, accw
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
    // the classifier's weights in LDS when they fit (wcs = 1), else read
    // from global memory
    extern __shared__ float wcs_lds[];
    const bool wcs = CLS && (int64_t)n_cls * C <= kClsLdsFloats;
    if (wcs) {
        for (int64_t i = threadIdx.x; i < (int64_t)n_cls * C; i += kBlock) wcs_lds[i] = w_cls[i];
        __syncthreads();
    }
    const float *wc = wcs ? wcs_lds : w_cls;

    // the next point's record is loaded while this point is processed
    int vn[DP1];
    float bn[DP1];
    auto load_record = [&](int64_t p) {
        const int64_t q = p < m ? p : 0;
#pragma unroll
        for (int k = 0; k < DP1; ++k) {
            vn[k] = idx[q * DP1 + k];
            bn[k] = bary[q * DP1 + k];
        }
    };
    if (wave < m) load_record(wave);
    for (int64_t p = wave; p < m; p += nwaves) {
        int v[DP1];
        float b[DP1];
#pragma unroll
        for (int k = 0; k < DP1; ++k) {
            v[k] = vn[k];
            b[k] = bn[k];
        }
        // the point's logit gradient, lane cls holding g[cls] (64 at a time)
        float gl = 0.f;
        if (CLS && lane < n_cls) gl = grad_out[p * n_cls + lane];
        float x[DP1][CH];
#pragma unroll
        for (int k = 0; k < DP1; ++k)
#pragma unroll
            for (int i = 0; i < CH; ++i) {
                const int c = lane + 64 * i;
                x[k][i] = (c < C && v[k] >= 0) ? value_at<IN_BF16>(values, (int64_t)v[k] * C + c) : 0.f;
            }
        load_record(p + nwaves);
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
            db[k] = s;
        }
        wave_sum_n<DP1>(db);  // the d+1 reductions interleaved
#pragma unroll
        for (int k = 0; k < DP1; ++k) db[k] = tanhf(b_delta + db[k]);
        // gf = g W_cls (classifier) or g
        float gf[CH];
#pragma unroll
        for (int i = 0; i < CH; ++i) {
            const int c = lane + 64 * i;
            gf[i] = 0.f;
            if (!CLS && c < C) gf[i] = grad_out[p * C + c];
        }
        if (CLS) {
            for (int c0 = 0; c0 < n_cls; c0 += 64) {
                if (c0 > 0) gl = lane + c0 < n_cls ? grad_out[p * n_cls + c0 + lane] : 0.f;
                const int nb = n_cls - c0 < 64 ? n_cls - c0 : 64;
                for (int t = 0; t < nb; ++t) {
                    const float g = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, gl), t));
#pragma unroll
                    for (int i = 0; i < CH; ++i) {
                        const int c = lane + 64 * i;
                        if (c < C) gf[i] = fmaf(g, wc[(int64_t)(c0 + t) * C + c], gf[i]);
                    }
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
            darg[k] = s;
        }
        wave_sum_n<DP1>(darg);
#pragma unroll
        for (int k = 0; k < DP1; ++k) {
            darg[k] *= 1.f - db[k] * db[k];
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

// Over the pair-list entries of a vertex (n of them, 1 <= n <= kPart), each
// giving a point p and the vertex's slot k in p's simplex, the two sums whose
// combination is dX_v: acc = sum alpha_pk gf_p and accw = sum (beta_pk -
// [k = k*_pc] gamma_pk), with dX_v = acc + w_delta accw.  Lane t holds entry
// t (`x`, from dx_entry) and its three coefficients (dx_coef); the rows of
// gf and am are loaded several entries at a time (dx_rows), each entry's
// values read from its lane, and added in list order.  The kernels load a
// list's entries two lists ahead and its coefficients one list ahead.
__device__ __forceinline__ int dx_entry(const int32_t *__restrict__ list, int64_t e0, int n, int lane) {
    const bool ok = n >= 1 && n <= kPart;  // otherwise entry 0, which exists whenever a list is read
    return list[2 * (ok ? e0 + (lane < n ? lane : n - 1) : 0)];
}

struct DxCoef {
    float al, be, ga;
};

// The coefficients of a list of n entries; n outside [1, kPart] (a header
// past the range, whose entry 0 may predate this splat) loads nothing.
template <int D>
__device__ __forceinline__ DxCoef dx_coef(int x, int n, const float *__restrict__ coef) {
    if (n < 1 || n > kPart) return DxCoef{0.f, 0.f, 0.f};
    const float *cf = coef + ((int64_t)list_point(x) * (D + 1) + list_slot(x)) * 3;
    return DxCoef{cf[0], cf[1], cf[2]};
}

template <int CH>
constexpr int dx_block() { return CH == 1 ? kDxRows1 : CH >= 8 ? 1 : 8 / CH; }

template <int CH>
__device__ __forceinline__ void dx_rows(int x, DxCoef q, int n, int C, const float *__restrict__ gf,
                                        const uint8_t *__restrict__ am, float *acc, float *accw) {
    constexpr int NB = dx_block<CH>();  // entries whose rows are in flight together
    const int lane = threadIdx.x & 63;
    const int pl = list_point(x), kl = list_slot(x);
#pragma unroll
    for (int i = 0; i < CH; ++i) acc[i] = accw[i] = 0.f;
    for (int t0 = 0; t0 < n; t0 += NB) {
        int ps[NB], ks[NB];
        float al[NB], be[NB], ga[NB];
#pragma unroll
        for (int u = 0; u < NB; ++u) {
            const int t = t0 + u;  // below 2 kPart; lanes past n hold entry n - 1
            ps[u] = __builtin_amdgcn_readlane(pl, t);
            ks[u] = __builtin_amdgcn_readlane(kl, t);
            al[u] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(q.al), t));
            be[u] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(q.be), t));
            ga[u] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(q.ga), t));
        }
        // rows past n are not loaded (a wave-uniform branch)
        float g[NB][CH];
        int a[NB][CH];
#pragma unroll
        for (int u = 0; u < NB; ++u)
#pragma unroll
            for (int i = 0; i < CH; ++i) {
                const int c = lane + 64 * i;
                g[u][i] = 0.f;
                a[u][i] = 0;
                if (t0 + u < n && c < C) {
                    g[u][i] = gf[(int64_t)ps[u] * C + c];
                    a[u][i] = am[(int64_t)ps[u] * C + c];
                }
            }
#pragma unroll
        for (int u = 0; u < NB; ++u) {
            if (t0 + u >= n) break;
#pragma unroll
            for (int i = 0; i < CH; ++i) {
                acc[i] = fmaf(al[u], g[u][i], acc[i]);
                accw[i] += a[u][i] == ks[u] ? be[u] - ga[u] : be[u];
            }
        }
    }
}

// The parts of long pair lists (the splat's split lists: more than kPart
// entries, cut into parts of kPart): one wavefront per part row, writing its
// acc and accw to part row u of `partial` [rows][2 C].
template <int D, int CH>
__global__ __launch_bounds__(kBlock) void k_dfb_parts(const int32_t *__restrict__ counters, int C,
                                                      const int32_t *__restrict__ list,
                                                      const int2 *__restrict__ partrec, const float *__restrict__ coef,
                                                      const float *__restrict__ gf, const uint8_t *__restrict__ am,
                                                      float *__restrict__ partial) {
    const int lane = threadIdx.x & 63;
    const int64_t nrows = counters[CNT_ROWS];
    const XcdShare sh = xcd_share(nrows);
    const int64_t st = sh.nwaves;
    auto rec = [&](int64_t u) { return u < sh.hi ? partrec[u] : make_int2(0, 0); };
    int64_t u = sh.lo + sh.wave;
    int2 r0 = rec(u);
    int x0 = dx_entry(list, r0.x, r0.y, lane);
    int2 r1 = rec(u + st);
    DxCoef q0 = dx_coef<D>(x0, r0.y, coef);
    int x1 = dx_entry(list, r1.x, r1.y, lane);
    int2 r2 = rec(u + 2 * st);
    for (; u < sh.hi; u += st) {
        const DxCoef q1 = dx_coef<D>(x1, r1.y, coef);
        const int x2 = dx_entry(list, r2.x, r2.y, lane);
        const int2 r3 = rec(u + 3 * st);
        float acc[CH], accw[CH];
        dx_rows<CH>(x0, q0, r0.y, C, gf, am, acc, accw);
        float *o = partial + u * 2 * C;
#pragma unroll
        for (int i = 0; i < CH; ++i) {
            const int c = lane + 64 * i;
            if (c < C) {
                o[c] = acc[i];
                o[C + c] = accw[i];
            }
        }
        r0 = r1;
        x0 = x1;
        q0 = q1;
        r1 = r2;
        x1 = x2;
        r2 = r3;
    }
}

// dX_v: a vertex with at most kPart entries over its list, a split vertex
// by adding its part rows in part order; one wavefront per vertex, lane =
// channel.
template <int D, int CH, bool OUT_BF16>
__global__ __launch_bounds__(kBlock) void k_dfb_gather(const int32_t *__restrict__ counters, int C,
                                                       const int32_t *__restrict__ vinfo,
                                                       const int32_t *__restrict__ list,
                                                       const int32_t *__restrict__ split,
                                                       const float *__restrict__ coef,
                                                       const float *__restrict__ gf, const uint8_t *__restrict__ am,
                                                       const float *__restrict__ partial,
                                                       const float *__restrict__ w_delta, void *__restrict__ out) {
    const int lane = threadIdx.x & 63;
    const int64_t V = counters[CNT_V];
    const int64_t ns = counters[CNT_SPLIT];
    float wd[CH];
#pragma unroll
    for (int i = 0; i < CH; ++i) {
        const int c = lane + 64 * i;
        wd[i] = c < C ? w_delta[c] : 0.f;
    }
    auto store = [&](int64_t v, const float *acc, const float *accw) {
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
    };
    // short lists: headers three vertices ahead, entries two, coefficients one
    const XcdShare sh = xcd_share(V);
    const int64_t st = sh.nwaves;
    const int2 *VI = reinterpret_cast<const int2 *>(vinfo);
    auto header = [&](int64_t v) { return v < sh.hi ? VI[v] : make_int2(0, 0); };
    int64_t v = sh.lo + sh.wave;
    int2 h0 = header(v);
    int x0 = dx_entry(list, h0.x, h0.y, lane);
    int2 h1 = header(v + st);
    DxCoef q0 = dx_coef<D>(x0, h0.y, coef);
    int x1 = dx_entry(list, h1.x, h1.y, lane);
    int2 h2 = header(v + 2 * st);
    for (; v < sh.hi; v += st) {
        const DxCoef q1 = dx_coef<D>(x1, h1.y, coef);
        const int x2 = dx_entry(list, h2.x, h2.y, lane);
        const int2 h3 = header(v + 3 * st);
        if (h0.y <= kPart) {  // a split vertex: below
            float acc[CH], accw[CH];
            dx_rows<CH>(x0, q0, h0.y, C, gf, am, acc, accw);
            store(v, acc, accw);
        }
        h0 = h1;
        x0 = x1;
        q0 = q1;
        h1 = h2;
        x1 = x2;
        h2 = h3;
    }
    const XcdShare ss = xcd_share(ns);
    for (int64_t sp = ss.lo + ss.wave; sp < ss.hi; sp += ss.nwaves) {
        const int v = split[3 * sp], row0 = split[3 * sp + 1], parts = split[3 * sp + 2];
        float acc[CH], accw[CH];
#pragma unroll
        for (int i = 0; i < CH; ++i) acc[i] = accw[i] = 0.f;
        for (int u = 0; u < parts; ++u) {
            const float *o = partial + ((int64_t)row0 + u) * 2 * C;
#pragma unroll
            for (int i = 0; i < CH; ++i) {
                const int c = lane + 64 * i;
                if (c < C) {
                    acc[i] += o[c];
                    accw[i] += o[C + c];
                }
            }
        }
        store(v, acc, accw);
    }
}

// Classifier gradients: dW_cls [n_cls][C] = sum_p g_p^T f_p and db_cls =
// sum_p g_p, as partial sums over chunks of kClsChunk points, on fp32 MFMA.
// One wavefront per chunk and tile of 32 classes x 32 channels (blockIdx.y):
// v_mfma_f32_32x32x2f32 with A = the chunk's g rows transposed (32 classes x
// 2 points: lane l holds class l mod 32 of point l / 32 of the pair) and B
// = their f rows (2 points x 32 channels).  The tiles with c0 = 0 also sum
// each class's g values (db_cls).  Classes past n_cls, channels past C and
// points past m are zeros.
constexpr int kClsChunk = 256;
constexpr int kClsSteps = 8;  // point pairs whose loads are in flight together
typedef float f32x16c_t __attribute__((ext_vector_type(16)));

__global__ __launch_bounds__(kBlock) void k_dfb_cls(int64_t m, int nch, int C, int n_cls,
                                                    const float *__restrict__ grad_out, const float *__restrict__ f,
                                                    float *__restrict__ part_c, float *__restrict__ part_bc) {
    const int lane = threadIdx.x & 63;
    const int64_t chunk = (int64_t)blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6);
    if (chunk >= nch) return;  // a whole wavefront; the kernel has no barrier
    const int ntc = (C + 31) / 32;
    const int k0 = (int)(blockIdx.y / ntc) * 32, c0 = (int)(blockIdx.y % ntc) * 32;
    const int row = lane & 31, half = lane >> 5;
    const int kA = k0 + row, cB = c0 + row;
    const bool okA = kA < n_cls, okB = cB < C;
    const int64_t p0 = chunk * kClsChunk;
    const int64_t p1 = p0 + kClsChunk < m ? p0 + kClsChunk : m;
    f32x16c_t acc;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = 0.f;
    float sb = 0.f;
    for (int64_t q = p0; q < p1; q += 2 * kClsSteps) {
        float a[kClsSteps], b[kClsSteps];
#pragma unroll
        for (int s = 0; s < kClsSteps; ++s) {
            const int64_t p = q + 2 * s + half;
            const bool okp = p < p1;
            a[s] = okp && okA ? grad_out[p * n_cls + kA] : 0.f;
            b[s] = okp && okB ? f[p * C + cB] : 0.f;
        }
#pragma unroll
        for (int s = 0; s < kClsSteps; ++s) {
            acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[s], b[s], acc, 0, 0, 0);
            sb += a[s];
        }
    }
    // D: lane l holds channel l mod 32, in register r the class 8 (r / 4) + 4 (l / 32) + r mod 4
    float *o = part_c + chunk * n_cls * C;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int k = k0 + 8 * (r >> 2) + 4 * half + (r & 3);
        if (k < n_cls && okB) o[(int64_t)k * C + cB] = acc[r];
    }
    if (c0 == 0) {
        sb += __shfl_xor(sb, 32, 64);
        if (half == 0 && okA) part_bc[chunk * n_cls + kA] = sb;
    }
}

// The same per-point work for C a multiple of 4 up to 256 (the segmentation
// networks' widths): a group of G = 2^LG lanes per point, lane j holding the
// float4 chunk j of each row, 64 / G points per wavefront side by side; the
// dot products over C are group sums (d+1 of them interleaved).  The
// per-channel sums of dw_delta are added across the groups at the end.
template <bool IN_BF16>
__device__ __forceinline__ float4 row4(const void *values, int64_t at4) {
    if (IN_BF16) {
        const uint2 u = reinterpret_cast<const uint2 *>(values)[at4];
        return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                           __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u));
    }
    return reinterpret_cast<const float4 *>(values)[at4];
}

template <int LG, int N>
__device__ __forceinline__ void group_sum_n(float *x) {
#pragma unroll
    for (int off = (1 << LG) >> 1; off > 0; off >>= 1) {
        float y[N];
#pragma unroll
        for (int k = 0; k < N; ++k) y[k] = __shfl_xor(x[k], off, 64);
#pragma unroll
        for (int k = 0; k < N; ++k) x[k] += y[k];
    }
}

constexpr int kGl = 4;  // registers of g classes loaded ahead, per lane

template <int D, int LG, bool IN_BF16, bool CLS>
__global__ __launch_bounds__(kBlock) void k_dfb_points_g(int64_t m, int C, const int32_t *__restrict__ idx,
                                                         const float *__restrict__ bary,
                                                         const void *__restrict__ values,
                                                         const float *__restrict__ w_delta, float b_delta,
                                                         const float *__restrict__ w_cls, int n_cls,
                                                         const float *__restrict__ grad_out,
                                                         float *__restrict__ gf_out, uint8_t *__restrict__ am_out,
                                                         float *__restrict__ coef, float *__restrict__ f_out,
                                                         float *__restrict__ part_w, float *__restrict__ part_b) {
    constexpr int DP1 = D + 1;
    constexpr int G = 1 << LG;
    constexpr int PPW = 64 / G;
    const int lane = threadIdx.x & 63;
    const int grp = lane >> LG, j = lane & (G - 1);
    const int NC = C >> 2;
    const bool has = j < NC;
    const int64_t wave = ((int64_t)blockIdx.x * kBlock + threadIdx.x) >> 6;
    const int64_t nwaves = ((int64_t)gridDim.x * kBlock) >> 6;
    extern __shared__ float wcs_lds[];
    const bool wcs = CLS && (int64_t)n_cls * C <= kClsLdsFloats;
    if (wcs) {
        for (int64_t i = threadIdx.x; i < (int64_t)n_cls * C; i += kBlock) wcs_lds[i] = w_cls[i];
        __syncthreads();
    }
    const float *wc = wcs ? wcs_lds : w_cls;
    const float4 wd = has ? reinterpret_cast<const float4 *>(w_delta)[j] : make_float4(0.f, 0.f, 0.f, 0.f);
    float4 acc_w = make_float4(0.f, 0.f, 0.f, 0.f);
    float acc_b = 0.f;
    // a point's vertex ids are loaded an iteration ahead of its rows
    int vn[DP1];
    auto load_ids = [&](int64_t p0n) {
        const int64_t pn = p0n + grp;
        const int64_t qn = pn < m ? pn : 0;
#pragma unroll
        for (int k = 0; k < DP1; ++k) vn[k] = idx[qn * DP1 + k];
    };
    load_ids(wave * PPW);
    for (int64_t p0 = wave * PPW; p0 < m; p0 += nwaves * PPW) {
        const int64_t p = p0 + grp;
        const bool live = p < m;
        const int64_t q = live ? p : 0;
        int v[DP1];
        float b[DP1];
#pragma unroll
        for (int k = 0; k < DP1; ++k) v[k] = vn[k];
        load_ids(p0 + nwaves * PPW);
#pragma unroll
        for (int k = 0; k < DP1; ++k) b[k] = live ? bary[q * DP1 + k] : 0.f;
        // the point's first kGl G classes of g, loaded with its record (lane j
        // of the group holds class i G + j in gpre[i])
        float gpre[kGl];
#pragma unroll
        for (int i = 0; i < kGl; ++i) {
            const int c = i * G + j;
            gpre[i] = (CLS && live && c < n_cls) ? grad_out[q * n_cls + c] : 0.f;
        }
        float4 x[DP1];
#pragma unroll
        for (int k = 0; k < DP1; ++k)
            x[k] = (has && live && v[k] >= 0) ? row4<IN_BF16>(values, (int64_t)v[k] * NC + j)
                                              : make_float4(0.f, 0.f, 0.f, 0.f);
        // MaxPool with the winning vertex (first of equal maxima), per channel
        float4 mx = make_float4(b[0] * x[0].x, b[0] * x[0].y, b[0] * x[0].z, b[0] * x[0].w);
        int a0 = 0, a1 = 0, a2 = 0, a3 = 0;
#pragma unroll
        for (int k = 1; k < DP1; ++k) {
            const float q0 = b[k] * x[k].x, q1 = b[k] * x[k].y, q2 = b[k] * x[k].z, q3 = b[k] * x[k].w;
            if (q0 > mx.x) { mx.x = q0; a0 = k; }
            if (q1 > mx.y) { mx.y = q1; a1 = k; }
            if (q2 > mx.z) { mx.z = q2; a2 = k; }
            if (q3 > mx.w) { mx.w = q3; a3 = k; }
        }
        // the offsets, as the forward computes them
        float db[DP1];
#pragma unroll
        for (int k = 0; k < DP1; ++k) {
            float t = 0.f;
            t = fmaf(b[k] * x[k].x - mx.x, wd.x, t);
            t = fmaf(b[k] * x[k].y - mx.y, wd.y, t);
            t = fmaf(b[k] * x[k].z - mx.z, wd.z, t);
            t = fmaf(b[k] * x[k].w - mx.w, wd.w, t);
            db[k] = t;
        }
        group_sum_n<LG, DP1>(db);
#pragma unroll
        for (int k = 0; k < DP1; ++k) db[k] = tanhf(b_delta + db[k]);
        // gf = g W_cls (classifier) or g, this lane's four channels
        float4 gf = make_float4(0.f, 0.f, 0.f, 0.f);
        if (!CLS) {
            if (has && live) gf = reinterpret_cast<const float4 *>(grad_out)[q * NC + j];
        } else {
            for (int c0 = 0; c0 < n_cls; c0 += G) {
                // lane j of the group holds the point's g[c0 + j]; class c0 + t from lane t
                const int ci = c0 >> LG;
                float gl = gpre[0];
#pragma unroll
                for (int i = 1; i < kGl; ++i) gl = ci == i ? gpre[i] : gl;
                if (ci >= kGl) gl = (live && c0 + j < n_cls) ? grad_out[q * n_cls + c0 + j] : 0.f;
                const int nb = n_cls - c0 < G ? n_cls - c0 : G;
                for (int t = 0; t < nb; ++t) {
                    const float g = __shfl(gl, (grp << LG) + t, 64);
                    if (has) {
                        const float4 w = *reinterpret_cast<const float4 *>(wc + (int64_t)(c0 + t) * C + 4 * j);
                        gf.x = fmaf(g, w.x, gf.x);
                        gf.y = fmaf(g, w.y, gf.y);
                        gf.z = fmaf(g, w.z, gf.z);
                        gf.w = fmaf(g, w.w, gf.w);
                    }
                }
            }
        }
        // Tanh backward, and S
        float darg[DP1];
#pragma unroll
        for (int k = 0; k < DP1; ++k) {
            float t = 0.f;
            t = fmaf(gf.x, x[k].x, t);
            t = fmaf(gf.y, x[k].y, t);
            t = fmaf(gf.z, x[k].z, t);
            t = fmaf(gf.w, x[k].w, t);
            darg[k] = t;
        }
        group_sum_n<LG, DP1>(darg);
        float S = 0.f;
#pragma unroll
        for (int k = 0; k < DP1; ++k) {
            darg[k] *= 1.f - db[k] * db[k];
            S += darg[k];
        }
        // Linear backward, accumulated per channel
#pragma unroll
        for (int k = 0; k < DP1; ++k) {
            acc_w.x = fmaf(darg[k], b[k] * x[k].x - mx.x, acc_w.x);
            acc_w.y = fmaf(darg[k], b[k] * x[k].y - mx.y, acc_w.y);
            acc_w.z = fmaf(darg[k], b[k] * x[k].z - mx.z, acc_w.z);
            acc_w.w = fmaf(darg[k], b[k] * x[k].w - mx.w, acc_w.w);
        }
        if (j == 0 && live) acc_b += S;
        // per-point records for the vertex gather and the classifier
        if (has && live) {
            reinterpret_cast<float4 *>(gf_out)[p * NC + j] = gf;
            reinterpret_cast<uint32_t *>(am_out)[p * NC + j] =
                (uint32_t)a0 | ((uint32_t)a1 << 8) | ((uint32_t)a2 << 16) | ((uint32_t)a3 << 24);
            if (CLS) {
                float4 f = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
                for (int k = 0; k < DP1; ++k) {
                    const float w = b[k] + db[k];
                    f.x = fmaf(w, x[k].x, f.x);
                    f.y = fmaf(w, x[k].y, f.y);
                    f.z = fmaf(w, x[k].z, f.z);
                    f.w = fmaf(w, x[k].w, f.w);
                }
                reinterpret_cast<float4 *>(f_out)[p * NC + j] = f;
            }
        }
        // slot k's coefficients from lane k mod G of the group
        if (live) {
#pragma unroll
            for (int k = 0; k < DP1; ++k)
                if ((k & (G - 1)) == j) {
                    coef[(p * DP1 + k) * 3 + 0] = b[k] + db[k];
                    coef[(p * DP1 + k) * 3 + 1] = b[k] * darg[k];
                    coef[(p * DP1 + k) * 3 + 2] = b[k] * S;
                }
        }
    }
    // the groups' per-channel sums added (lane j of every group holds chunk j)
#pragma unroll
    for (int off = G; off < 64; off <<= 1) {
        acc_w.x += __shfl_xor(acc_w.x, off, 64);
        acc_w.y += __shfl_xor(acc_w.y, off, 64);
        acc_w.z += __shfl_xor(acc_w.z, off, 64);
        acc_w.w += __shfl_xor(acc_w.w, off, 64);
    }
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) acc_b += __shfl_xor(acc_b, off, 64);
    if (grp == 0 && has) reinterpret_cast<float4 *>(part_w)[wave * NC + j] = acc_w;
    if (lane == 0) part_b[wave] = acc_b;
}

template <int D, bool IN_BF16, bool CLS>
hipError_t launch_points_ch(lattice *L, int ch, unsigned grid, const void *values, int C, const float *w_delta,
                            float b_delta, const float *w_cls, int n_cls, const float *grad_out, float *gf,
                            uint8_t *am, float *coef, float *f, float *pw, float *pb) {
    const size_t lds = (CLS && (int64_t)n_cls * C <= kClsLdsFloats) ? (size_t)n_cls * C * sizeof(float) : 0;
    auto go = [&](auto kern) {
        hipLaunchKernelGGL(kern, dim3(grid), dim3(kBlock), lds, L->stream, L->m, C, L->idx, L->bary, values, w_delta,
                           b_delta, w_cls, n_cls, grad_out, gf, am, coef, f, pw, pb);
        return hipGetLastError();
    };
    // the grouped kernel: C a multiple of 4 up to 256, rows (and, without the
    // classifier, dL/df and w_delta) aligned for their vector loads
    const bool grouped = C % 4 == 0 && C <= 256 &&
                         (reinterpret_cast<uintptr_t>(values) & (IN_BF16 ? 7 : 15)) == 0 &&
                         (reinterpret_cast<uintptr_t>(w_delta) & 15) == 0 &&
                         (CLS ? (reinterpret_cast<uintptr_t>(w_cls) & 15) == 0
                              : (reinterpret_cast<uintptr_t>(grad_out) & 15) == 0);
    if (grouped) {
        int lg = 0;
        while ((1 << lg) < C / 4) ++lg;
        switch (lg) {
            case 0: return go(k_dfb_points_g<D, 0, IN_BF16, CLS>);
            case 1: return go(k_dfb_points_g<D, 1, IN_BF16, CLS>);
            case 2: return go(k_dfb_points_g<D, 2, IN_BF16, CLS>);
            case 3: return go(k_dfb_points_g<D, 3, IN_BF16, CLS>);
            case 4: return go(k_dfb_points_g<D, 4, IN_BF16, CLS>);
            case 5: return go(k_dfb_points_g<D, 5, IN_BF16, CLS>);
            default: return go(k_dfb_points_g<D, 6, IN_BF16, CLS>);
        }
    }
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
                            const uint8_t *am, const float *w_delta, float *partial, void *out) {
    const int64_t cap = (int64_t)L->cu_count * 8;
    auto grid_of = [&](int64_t waves) {
        int64_t g = (waves + 3) / 4;
        if (g > cap) g = cap;
        return (g + 7) / 8 * 8;  // whole XCD groups: each XCD takes one range
    };
    const int64_t g_parts = grid_of(split_rows_max(L)), g_vert = grid_of(L->max_vertices);
    auto go = [&](auto parts_kern, auto kern) {
        hipLaunchKernelGGL(parts_kern, dim3((unsigned)g_parts), dim3(kBlock), 0, L->stream, L->counters, C, L->list,
                           reinterpret_cast<const int2 *>(L->partrec), coef, gf, am, partial);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(kern, dim3((unsigned)g_vert), dim3(kBlock), 0, L->stream, L->counters, C, L->vinfo, L->list,
                           L->split, coef, gf, am, partial, w_delta, out);
        return hipGetLastError();
    };
#define DFB_G(CHV)                                                                                       \
    case CHV:                                                                                            \
        return out_bf16 ? go(k_dfb_parts<D, CHV>, k_dfb_gather<D, CHV, true>)                            \
                        : go(k_dfb_parts<D, CHV>, k_dfb_gather<D, CHV, false>);
    switch (ch) {
        DFB_G(1)
        DFB_G(2)
        DFB_G(4)
        DFB_G(8)
        default:
            return out_bf16 ? go(k_dfb_parts<D, 16>, k_dfb_gather<D, 16, true>)
                            : go(k_dfb_parts<D, 16>, k_dfb_gather<D, 16, false>);
    }
#undef DFB_G
}

template <int D>
hipError_t run_d(lattice *L, const void *values, bool in_bf16, int C, const float *w_delta, float b_delta,
                 const float *w_cls, int n_cls, const float *grad_out, void *grad_values, bool out_bf16,
                 float *grad_w_delta, float *grad_b_delta, float *grad_w_cls, float *grad_b_cls, char *scratch,
                 int nwaves, int nch) {
    const int ch = C <= 64 ? 1 : C <= 128 ? 2 : C <= 256 ? 4 : C <= 512 ? 8 : 16;
    const DfbLayout l = dfb_layout(L->m, C, D + 1, w_cls ? n_cls : 0, nwaves, nch, split_rows_max(L));
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
    if (grad_values && (e = launch_gather_ch<D>(L, ch, out_bf16, C, coef, gf, am, w_delta,
                                                reinterpret_cast<float *>(scratch + l.part), grad_values)) != hipSuccess)
        return e;
    float *tmp = reinterpret_cast<float *>(scratch + l.tmp);
    if (grad_w_delta && (e = rowsum::sum(L->stream, pw, nwaves, C, tmp, grad_w_delta)) != hipSuccess) return e;
    if (grad_b_delta && (e = rowsum::sum(L->stream, pb, nwaves, 1, tmp, grad_b_delta)) != hipSuccess) return e;
    if (w_cls && (grad_w_cls || grad_b_cls)) {
        float *pc = reinterpret_cast<float *>(scratch + l.pc);
        float *pbc = reinterpret_cast<float *>(scratch + l.pbc);
        const unsigned tiles = (unsigned)(((n_cls + 31) / 32) * ((C + 31) / 32));
        hipLaunchKernelGGL(k_dfb_cls, dim3((unsigned)((nch + kBlock / 64 - 1) / (kBlock / 64)), tiles), dim3(kBlock), 0,
                           L->stream, L->m, nch, C, n_cls, grad_out, f, pc, pbc);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if (grad_w_cls && (e = rowsum::sum(L->stream, pc, nch, (int64_t)n_cls * C, tmp, grad_w_cls)) != hipSuccess)
            return e;
        if (grad_b_cls && (e = rowsum::sum(L->stream, pbc, nch, n_cls, tmp, grad_b_cls)) != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace

// Wavefronts of the point kernel and point chunks of the classifier kernel.
void deform_backward_shape(const lattice *L, int *nwaves, int *nch) {
    // four workgroups of four wavefronts per CU, as many as the point kernel's
    // registers let a CU hold at once (twice that left a tail of waiting
    // workgroups: four frames 181 against 178 us)
    *nwaves = L->cu_count * 4 * 4;
    const int64_t c = (L->m + kClsChunk - 1) / kClsChunk;  // classifier chunks
    *nch = (int)(c < 1 ? 1 : c);
}

int64_t deform_backward_scratch_bytes(const lattice *L, int C, int n_cls) {
    int nwaves, nch;
    deform_backward_shape(L, &nwaves, &nch);
    return dfb_layout(L->m, C, L->d + 1, n_cls, nwaves, nch, split_rows_max(L)).total;
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
