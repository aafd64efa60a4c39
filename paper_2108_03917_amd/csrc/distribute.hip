// Distribute + PointNet + per-vertex max, fused (Sec. "Proposed Operations":
// Distribute, Eq. distribute; the PointNet block of the network figure;
// Sec. "Performance" suggests fusing Distribute and the PointNet into one
// operation so that the distributed rows are never stored).
//
// Every pair (point p, simplex vertex v) of the last splat is one row:
//   h_0 = [g_p - mu_v ; f_p]          (D_G: position minus the local mean
//                                      mu_v of J_v; D_F: the features)
//   h_l = W_l relu(a_l * h_{l-1} + s_l) + b_l,   l = 1, 2, 3, widths 16, 32, 64
//   x_v = max over the rows of v of h_3, per channel.
// (a_l, s_l) is the normalisation as a per-channel affine: what a group
// normalisation reduces to once its statistics are known.
//
// The rows are the entries of the splat's pair lists, which are grouped by
// vertex, so the rows of one vertex are consecutive:
//   k_entry_vertex   entry -> vertex map (one thread per short list, one per
//                    32-entry part of a long list, as the splat's gather);
//                    also zeroes the vertex's fp64 position sum
//   k_local_mean     one lane per entry; each wavefront owns 64 consecutive
//                    entries and sums the positions of each run of equal
//                    vertex in fp64 (LDS, one lane per coordinate); a run
//                    that is the vertex's whole list writes mu_v, otherwise
//                    the run is added to the vertex's fp64 sum atomically
//   k_mean_finish    mu_v of the lists that cross a 64-entry chunk
//   k_pointnet_init  -inf in the output rows of those vertices
//   k_pointnet       one lane per entry runs the three blocks (parameters
//                    in LDS, read by all lanes at once); block 3's outputs go
//                    to LDS channel-major, 32 channels at a time; then lane c
//                    walks the wavefront's entries keeping the running max of
//                    channel c and stores it at the end of each run: a plain
//                    store (32 lanes, half a row) when the run is the
//                    vertex's whole list, else an atomic max.  The max is exact in any order, so the
//                    result does not depend on scheduling.
#include "internal.h"

namespace {

constexpr int kBlock = 256;
constexpr int kWaves = kBlock / 64;
constexpr int kW1 = 16, kW2 = 32, kW3 = 64;  // block widths (the paper's figure)
constexpr int kMaxK0 = 16;                   // d + f_d, zero-padded to 16
constexpr int kHalf = kW3 / 2;               // block 3's outputs are staged 32 channels at a time
constexpr int kYStride = 64 + 1;             // LDS row of one channel: 64 entries + 1 (bank offset)

// LDS copy of the parameters, zero-padded to kMaxK0 inputs in block 1.
struct PnLds {
    float a0[kMaxK0], s0[kMaxK0], w0[kW1][kMaxK0], b0[kW1];
    float a1[kW1], s1[kW1], w1[kW2][kW1], b1[kW2];
    float a2[kW2], s2[kW2], w2[kW3][kW2], b2[kW3];
};

__device__ __forceinline__ float relu(float x) { return x > 0.f ? x : 0.f; }

// Atomic max of a float in global memory (compare and swap on the bits).
__device__ __forceinline__ void atomic_max_f32(float *addr, float val) {
    unsigned int *a = reinterpret_cast<unsigned int *>(addr);
    unsigned int old = __atomic_load_n(a, __ATOMIC_RELAXED);
    while (val > __uint_as_float(old)) {
        const unsigned int prev = atomicCAS(a, old, __float_as_uint(val));
        if (prev == old) break;
        old = prev;
    }
}

__global__ __launch_bounds__(kBlock) void k_entry_vertex(const int32_t *__restrict__ vinfo,
                                                         const int32_t *__restrict__ split,
                                                         const int32_t *__restrict__ rowmap,
                                                         const int32_t *__restrict__ counters, int d,
                                                         int32_t *__restrict__ lvert, double *__restrict__ macc) {
    const int64_t V = counters[CNT_V];
    const int64_t nrows = counters[CNT_ROWS];
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t v = (int64_t)blockIdx.x * kBlock + threadIdx.x; v < V; v += stride) {
        for (int i = 0; i < d; ++i) macc[v * d + i] = 0.0;
        const int off = vinfo[2 * v], cnt = vinfo[2 * v + 1];
        if (cnt > kPart) continue;  // written by its parts below
        for (int e = off; e < off + cnt; ++e) lvert[e] = (int32_t)v;
    }
    for (int64_t u = (int64_t)blockIdx.x * kBlock + threadIdx.x; u < nrows; u += stride) {
        const int sp = rowmap[u];
        const int v = split[3 * sp], row0 = split[3 * sp + 1];
        const int off = vinfo[2 * v], cnt = vinfo[2 * v + 1];
        const int e0 = off + (int)(u - row0) * kPart;
        const int e1 = e0 + kPart < off + cnt ? e0 + kPart : off + cnt;
        for (int e = e0; e < e1; ++e) lvert[e] = v;
    }
}

// Whether entries [off, off + cnt) lie in one 64-entry chunk.
__device__ __forceinline__ bool in_one_chunk(int off, int cnt) { return (off >> 6) == ((off + cnt - 1) >> 6); }

__global__ __launch_bounds__(kBlock) void k_local_mean(const int32_t *__restrict__ list,
                                                       const int32_t *__restrict__ lvert,
                                                       const int32_t *__restrict__ vinfo,
                                                       const float *__restrict__ pos, int d,
                                                       const int32_t *__restrict__ counters,
                                                       double *__restrict__ macc, float *__restrict__ mu) {
    __shared__ double gsh[kWaves][64][LATTICE_MAX_D];
    __shared__ int32_t vsh[kWaves][64];
    const int64_t E = counters[CNT_E];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    for (int64_t base = (int64_t)blockIdx.x * kBlock; base < E; base += (int64_t)gridDim.x * kBlock) {
        const int64_t e = base + threadIdx.x;
        const bool valid = e < E;
        const int v = valid ? lvert[e] : -1;
        const int p = valid ? list[2 * e] : 0;
        vsh[w][lane] = v;
        for (int i = 0; i < d; ++i) gsh[w][lane][i] = valid ? (double)pos[(int64_t)p * d + i] : 0.0;
        __syncthreads();
        if (lane < d) {
            const int i = lane;
            const int64_t chunk0 = base + w * 64;
            double acc = 0.0;
            for (int j = 0; j < 64; ++j) {
                const int vj = vsh[w][j];
                if (vj < 0) break;
                acc = (j == 0 || vsh[w][j - 1] != vj) ? gsh[w][j][i] : acc + gsh[w][j][i];
                if (j == 63 || vsh[w][j + 1] != vj) {
                    const int off = vinfo[2 * vj], cnt = vinfo[2 * vj + 1];
                    if (off >= chunk0 && off + cnt <= chunk0 + 64)
                        mu[(int64_t)vj * d + i] = (float)(acc / cnt);
                    else
                        atomicAdd(&macc[(int64_t)vj * d + i], acc);
                }
            }
        }
        __syncthreads();
    }
}

__global__ __launch_bounds__(kBlock) void k_mean_finish(const int32_t *__restrict__ vinfo,
                                                        const double *__restrict__ macc, int d,
                                                        const int32_t *__restrict__ counters, float *__restrict__ mu) {
    const int64_t V = counters[CNT_V];
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t v = (int64_t)blockIdx.x * kBlock + threadIdx.x; v < V; v += stride) {
        const int off = vinfo[2 * v], cnt = vinfo[2 * v + 1];
        if (in_one_chunk(off, cnt)) continue;
        for (int i = 0; i < d; ++i) mu[v * d + i] = (float)(macc[v * d + i] / cnt);
    }
}

// -inf in the rows of the vertices whose list crosses a chunk boundary: the
// vertex of entry 64k (k >= 1) when its list starts before it.
__global__ __launch_bounds__(kBlock) void k_pointnet_init(const int32_t *__restrict__ lvert,
                                                          const int32_t *__restrict__ vinfo,
                                                          const int32_t *__restrict__ counters,
                                                          float *__restrict__ out) {
    const int64_t E = counters[CNT_E];
    const int64_t nb = E > 0 ? (E - 1) / 64 : 0;  // boundaries 64, 128, ... below E
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t q = (int64_t)blockIdx.x * kBlock + threadIdx.x; q < nb * kW3; q += stride) {
        const int64_t e0 = (q / kW3 + 1) * 64;
        const int c = (int)(q % kW3);
        const int v = lvert[e0];
        if (vinfo[2 * v] < e0) out[(int64_t)v * kW3 + c] = -__builtin_huge_valf();
    }
}

__global__ __launch_bounds__(kBlock) void k_pointnet(const int32_t *__restrict__ list,
                                                     const int32_t *__restrict__ lvert,
                                                     const int32_t *__restrict__ vinfo,
                                                     const float *__restrict__ pos, const float *__restrict__ feat,
                                                     int d, int f_d, const float *__restrict__ params,
                                                     const float *__restrict__ mu,
                                                     const int32_t *__restrict__ counters, float *__restrict__ out) {
    __shared__ PnLds P;
    __shared__ float ysh[kWaves][kHalf * kYStride];
    __shared__ int32_t vsh[kWaves][64];
    __shared__ int32_t fsh[kWaves][64];

    // parameters -> LDS, block 1 zero-padded to kMaxK0 inputs
    const int k0 = d + f_d;
    {
        float *flat = reinterpret_cast<float *>(&P);
        for (int i = threadIdx.x; i < (int)(sizeof(PnLds) / sizeof(float)); i += kBlock) flat[i] = 0.f;
        __syncthreads();
        int at = 0;
        for (int i = threadIdx.x; i < k0; i += kBlock) {
            P.a0[i] = params[at + i];
            P.s0[i] = params[at + k0 + i];
        }
        at += 2 * k0;
        for (int i = threadIdx.x; i < kW1 * k0; i += kBlock) P.w0[i / k0][i % k0] = params[at + i];
        at += kW1 * k0;
        for (int i = threadIdx.x; i < kW1; i += kBlock) P.b0[i] = params[at + i];
        at += kW1;
        float *rest = &P.a1[0];  // blocks 2 and 3 are stored unpadded, in the packed order
        const int nrest = 2 * kW1 + kW2 * kW1 + kW2 + 2 * kW2 + kW3 * kW2 + kW3;
        for (int i = threadIdx.x; i < nrest; i += kBlock) rest[i] = params[at + i];
        __syncthreads();
    }

    const int64_t E = counters[CNT_E];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    float *Y = ysh[w];
    for (int64_t base = (int64_t)blockIdx.x * kBlock; base < E; base += (int64_t)gridDim.x * kBlock) {
        const int64_t chunk0 = base + w * 64;
        const int64_t e = chunk0 + lane;
        const bool valid = e < E;
        const int v = valid ? lvert[e] : -1;
        const int p = valid ? list[2 * e] : 0;
        // run flags: 1 first entry of a run, 2 last, 4 the run is the vertex's whole list
        const int vprev = __shfl_up(v, 1);
        const int vnext = __shfl_down(v, 1);
        int flags = 0;
        if (valid) {
            if (lane == 0 || vprev != v) flags |= 1;
            if (lane == 63 || vnext != v) flags |= 2;
            const int off = vinfo[2 * v], cnt = vinfo[2 * v + 1];
            if (off >= chunk0 && off + cnt <= chunk0 + 64) flags |= 4;
        }
        vsh[w][lane] = v;
        fsh[w][lane] = flags;

        // h_0 = [g_p - mu_v ; f_p], zero-padded
        float h0[kMaxK0];
#pragma unroll
        for (int i = 0; i < kMaxK0; ++i) h0[i] = 0.f;
        if (valid) {
            for (int i = 0; i < d; ++i) h0[i] = pos[(int64_t)p * d + i] - mu[(int64_t)v * d + i];
            for (int i = 0; i < f_d; ++i) h0[d + i] = feat[(int64_t)p * f_d + i];
        }
        // block 1
        float r[kW2];
#pragma unroll
        for (int k = 0; k < kMaxK0; ++k) r[k] = relu(fmaf(P.a0[k], h0[k], P.s0[k]));
        float h1[kW1];
#pragma unroll
        for (int c = 0; c < kW1; ++c) {
            float acc = P.b0[c];
#pragma unroll
            for (int k = 0; k < kMaxK0; ++k) acc = fmaf(P.w0[c][k], r[k], acc);
            h1[c] = acc;
        }
        // block 2
#pragma unroll
        for (int k = 0; k < kW1; ++k) r[k] = relu(fmaf(P.a1[k], h1[k], P.s1[k]));
        float h2[kW2];
#pragma unroll
        for (int c = 0; c < kW2; ++c) {
            float acc = P.b1[c];
#pragma unroll
            for (int k = 0; k < kW1; ++k) acc = fmaf(P.w1[c][k], r[k], acc);
            h2[c] = acc;
        }
        // block 3, 32 output channels at a time into LDS (channel-major),
        // then lane c < 32 keeps the running max of channel h*32 + c over
        // each run of the wavefront's entries
#pragma unroll
        for (int k = 0; k < kW2; ++k) r[k] = relu(fmaf(P.a2[k], h2[k], P.s2[k]));
        for (int h = 0; h < kW3 / kHalf; ++h) {
#pragma unroll 4
            for (int c = 0; c < kHalf; ++c) {
                const int co = h * kHalf + c;
                float acc = P.b2[co];
#pragma unroll
                for (int k = 0; k < kW2; ++k) acc = fmaf(P.w2[co][k], r[k], acc);
                Y[c * kYStride + lane] = acc;
            }
            __syncthreads();
            if (lane < kHalf) {
                const int c = lane;
                float mx = 0.f;
#pragma unroll 8
                for (int j = 0; j < 64; ++j) {
                    const int vj = vsh[w][j];
                    const int fj = fsh[w][j];
                    const float y = Y[c * kYStride + j];
                    mx = (fj & 1) ? y : fmaxf(mx, y);
                    if (vj >= 0 && (fj & 2)) {
                        float *dst = out + (int64_t)vj * kW3 + h * kHalf + c;
                        if (fj & 4)
                            *dst = mx;
                        else
                            atomic_max_f32(dst, mx);
                    }
                }
            }
            __syncthreads();
        }
    }
}

}  // namespace

// Packed parameter count for d + f_d = k0 inputs: per block a [K], s [K],
// W [w][K], b [w] with K the block's input width.
int pointnet_param_count(int k0) {
    return 2 * k0 + kW1 * k0 + kW1 + 2 * kW1 + kW2 * kW1 + kW2 + 2 * kW2 + kW3 * kW2 + kW3;
}

hipError_t launch_distribute_pointnet(lattice *L, const float *pos, const float *feat, int f_d, const float *params,
                                      float *out, float *mean) {
    if (L->m == 0) return hipSuccess;
    const int d = L->d;
    float *mu = mean ? mean : L->mu;
    const int64_t E = L->m * (int64_t)(d + 1);
    const unsigned g_v = grid_for(L->max_vertices, kBlock, L->cu_count, 8);
    hipLaunchKernelGGL(k_entry_vertex, dim3(g_v), dim3(kBlock), 0, L->stream, L->vinfo, L->split, L->rowmap,
                       L->counters, d, L->lvert, L->macc);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const unsigned g_e = grid_for(E, kBlock, L->cu_count, 8);
    hipLaunchKernelGGL(k_local_mean, dim3(g_e), dim3(kBlock), 0, L->stream, L->list, L->lvert, L->vinfo, pos, d,
                       L->counters, L->macc, mu);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_mean_finish, dim3(g_v), dim3(kBlock), 0, L->stream, L->vinfo, L->macc, d, L->counters, mu);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const unsigned g_i = grid_for((E / 64 + 1) * kW3, kBlock, L->cu_count, 4);
    hipLaunchKernelGGL(k_pointnet_init, dim3(g_i), dim3(kBlock), 0, L->stream, L->lvert, L->vinfo, L->counters, out);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const unsigned g_p = grid_for(E, kBlock, L->cu_count, 3);  // 45 KB of LDS: three workgroups per CU
    hipLaunchKernelGGL(k_pointnet, dim3(g_p), dim3(kBlock), 0, L->stream, L->list, L->lvert, L->vinfo, pos, feat, d,
                       f_d, params, mu, L->counters, out);
    return hipGetLastError();
}
