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
//                    vertex in fp64 (a segmented scan over shuffles); a run
//                    that is the vertex's whole list writes mu_v, otherwise
//                    the run is added to the vertex's fp64 sum atomically
//   k_pointnet_prep  mu_v of the lists that cross a 64-entry chunk; the key
//                    of -inf in the key row of each vertex whose list crosses
//                    a chunk boundary; the parameters in the padded layout
//                    (three independent jobs in one launch)
//   k_pointnet       the three blocks as fp32 MFMA products over the
//                    wavefront's 64 entries (weight fragments held in
//                    registers); block 3's outputs go to LDS channel-major;
//                    then lane c walks the wavefront's entries keeping the
//                    running max of channel c and stores it at the end of
//                    each run: a plain store (64 lanes, one row, fp32 or bf16)
//                    when the run is the vertex's whole list, else an
//                    unsigned atomic max of an order-preserving key (no
//                    returned value to wait for) into the vertex's key row.
//                    A list that crosses a boundary starts in the chunk just
//                    before it, and only one list crosses each boundary, so
//                    key row j belongs to the list that starts in chunk j.
//                    The max is exact in any order, so the result does not
//                    depend on scheduling; a bf16 row is rounded once, from
//                    the fp32 max.
#include "internal.h"

namespace {

constexpr int kBlock = 256;
constexpr int kWaves = kBlock / 64;
constexpr int kW1 = 16, kW2 = 32, kW3 = 64;  // block widths (the paper's figure)
constexpr int kMaxK0 = 16;                   // d + f_d, zero-padded to 16
// LDS row of one output channel: 64 entries + 4 (16-byte aligned rows; the
// 16 lanes of a quarter-wave reading 16 bytes each then cover all 64 banks,
// and the MFMA output writes of the four lane quarters fall 16 banks apart)
constexpr int kYStride = 64 + 4;

__device__ __forceinline__ float relu(float x) { return x > 0.f ? x : 0.f; }

// Order-preserving map of a float to an unsigned integer (a > b exactly
// when key(a) > key(b), for non-NaN values), so that an unsigned atomic max,
// which needs no returned value, is a float max.
__device__ __forceinline__ unsigned int max_key(float f) {
    const unsigned int u = __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float key_value(unsigned int k) {
    return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

// Segment start of each lane: the highest lane at or below it whose entry
// starts a run of equal vertex (head).
__device__ __forceinline__ int run_start(bool head, int lane) {
    const unsigned long long hb = __ballot(head);
    const unsigned long long below = lane == 63 ? hb : (hb & ((2ull << lane) - 1ull));
    return 63 - __clzll(below);
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

// One lane per entry; the positions of each run of equal vertex within the
// wavefront's 64 entries are summed by a segmented scan in fp64 (shuffles),
// and the run's last lane writes mu_v or adds the run to the vertex's sum.
template <int D>
__global__ __launch_bounds__(kBlock) void k_local_mean(const int32_t *__restrict__ list,
                                                       const int32_t *__restrict__ lvert,
                                                       const int32_t *__restrict__ vinfo,
                                                       const float *__restrict__ pos,
                                                       const int32_t *__restrict__ counters,
                                                       double *__restrict__ macc, float *__restrict__ mu) {
    const int64_t E = counters[CNT_E];
    const int lane = threadIdx.x & 63;
    const int64_t nwaves = (int64_t)gridDim.x * kWaves;
    for (int64_t c = ((int64_t)blockIdx.x * kBlock + threadIdx.x) >> 6; c * 64 < E; c += nwaves) {
        const int64_t chunk0 = c * 64;
        const int64_t e = chunk0 + lane;
        const bool valid = e < E;
        const int v = valid ? lvert[e] : -1;
        const int p = valid ? list[2 * e] : 0;
        double acc[D];
#pragma unroll
        for (int i = 0; i < D; ++i) acc[i] = valid ? (double)pos[(int64_t)p * D + i] : 0.0;
        const int vprev = __shfl_up(v, 1), vnext = __shfl_down(v, 1);
        const int start = run_start(lane == 0 || vprev != v, lane);
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
#pragma unroll
            for (int i = 0; i < D; ++i) {
                const double t = __shfl_up(acc[i], off);
                if (lane - off >= start) acc[i] += t;
            }
        }
        if (valid && (lane == 63 || vnext != v)) {
            const int off = vinfo[2 * v], cnt = vinfo[2 * v + 1];
            if (off >= chunk0 && off + cnt <= chunk0 + 64) {
#pragma unroll
                for (int i = 0; i < D; ++i) mu[(int64_t)v * D + i] = (float)(acc[i] / cnt);
            } else {
#pragma unroll
                for (int i = 0; i < D; ++i) atomicAdd(&macc[(int64_t)v * D + i], acc[i]);
            }
        }
    }
}

// The bodies below take their block index and block count, so that one
// launch (k_pointnet_prep) can run several of them side by side.
__device__ __forceinline__ void mean_finish(int64_t bid, int64_t nblk, const int32_t *__restrict__ vinfo,
                                            const double *__restrict__ macc, int d,
                                            const int32_t *__restrict__ counters, float *__restrict__ mu) {
    const int64_t V = counters[CNT_V];
    const int64_t stride = nblk * kBlock;
    for (int64_t v = bid * kBlock + threadIdx.x; v < V; v += stride) {
        const int off = vinfo[2 * v], cnt = vinfo[2 * v + 1];
        if (in_one_chunk(off, cnt)) continue;
        for (int i = 0; i < d; ++i) mu[v * d + i] = (float)(macc[v * d + i] / cnt);
    }
}

// Store channel c of output row v as fp32 or, rounded to nearest even, bf16.
template <bool OUT_BF16>
__device__ __forceinline__ void store_out(void *out, int64_t v, int c, float x) {
    if (OUT_BF16)
        reinterpret_cast<uint16_t *>(out)[v * kW3 + c] = (uint16_t)bf16_bits(x);
    else
        reinterpret_cast<float *>(out)[v * kW3 + c] = x;
}

// Lists that cross a chunk boundary: the vertex of entry 64 (j + 1), j >= 0,
// when its list starts in chunk j.  Mode 0 sets key row j to the key of -inf;
// mode 1 decodes it into the vertex's output row.  A long list crosses
// several boundaries; only its first crossing does the work.
template <bool OUT_BF16>
__device__ __forceinline__ void pointnet_rows(int64_t bid, int64_t nblk, const int32_t *__restrict__ lvert,
                                              const int32_t *__restrict__ vinfo,
                                              const int32_t *__restrict__ counters, int mode,
                                              unsigned int *__restrict__ keys, void *__restrict__ out) {
    const int64_t E = counters[CNT_E];
    const int64_t nb = E > 0 ? (E - 1) / 64 : 0;  // boundaries 64, 128, ... below E
    const int64_t stride = nblk * kBlock;
    for (int64_t q = bid * kBlock + threadIdx.x; q < nb * kW3; q += stride) {
        const int64_t j = q / kW3;
        const int64_t e0 = (j + 1) * 64;
        const int c = (int)(q % kW3);
        const int v = lvert[e0];
        const int64_t off = vinfo[2 * v];
        if (off >= e0 || off < e0 - 64) continue;  // not crossing here, or crossed an earlier boundary
        if (mode == 0)
            keys[j * kW3 + c] = max_key(-__builtin_huge_valf());
        else
            store_out<OUT_BF16>(out, v, c, key_value(keys[j * kW3 + c]));
    }
}

// The parameters in a fixed layout: block 1 zero-padded to kMaxK0 inputs
// (a = s = W = 0 on the padding, so padded inputs contribute nothing), then
// blocks 2 and 3 as packed.  Every offset is a compile-time constant.
constexpr int kA0 = 0, kS0 = kA0 + kMaxK0, kWt0 = kS0 + kMaxK0, kB0 = kWt0 + kW1 * kMaxK0;
constexpr int kA1 = kB0 + kW1, kS1 = kA1 + kW1, kWt1 = kS1 + kW1, kB1 = kWt1 + kW2 * kW1;
constexpr int kA2 = kB1 + kW2, kS2 = kA2 + kW2, kWt2 = kS2 + kW2, kB2 = kWt2 + kW3 * kW2;
constexpr int kPadded = kB2 + kW3;

__device__ __forceinline__ void pack_pointnet(int64_t bid, int64_t nblk, const float *__restrict__ params, int k0,
                                              float *__restrict__ padded) {
    for (int64_t i = bid * kBlock + threadIdx.x; i < kPadded; i += nblk * kBlock) {
        float x = 0.f;
        if (i < kS0) {
            if (i - kA0 < k0) x = params[i - kA0];
        } else if (i < kWt0) {
            if (i - kS0 < k0) x = params[k0 + (i - kS0)];
        } else if (i < kB0) {
            const int c = (i - kWt0) / kMaxK0, k = (i - kWt0) % kMaxK0;
            if (k < k0) x = params[2 * k0 + c * k0 + k];
        } else {
            x = params[2 * k0 + kW1 * k0 + (i - kB0)];  // b0 and blocks 2, 3 as packed
        }
        padded[i] = x;
    }
}

// After the local means: mu_v of the crossing lists, the key rows set to
// -inf, and the parameters packed, in one launch (block ranges nb_mean,
// nb_rows, nb_pack).
__global__ __launch_bounds__(kBlock) void k_pointnet_prep(const int32_t *__restrict__ vinfo,
                                                          const double *__restrict__ macc, int d,
                                                          const int32_t *__restrict__ counters,
                                                          float *__restrict__ mu,
                                                          const int32_t *__restrict__ lvert,
                                                          unsigned int *__restrict__ keys,
                                                          const float *__restrict__ params, int k0,
                                                          float *__restrict__ padded, int nb_mean, int nb_rows,
                                                          int nb_pack) {
    const int b = blockIdx.x;
    if (b < nb_mean)
        mean_finish(b, nb_mean, vinfo, macc, d, counters, mu);
    else if (b < nb_mean + nb_rows)
        pointnet_rows<false>(b - nb_mean, nb_rows, lvert, vinfo, counters, 0, keys, nullptr);
    else
        pack_pointnet(b - nb_mean - nb_rows, nb_pack, params, k0, padded);
}

// After the PointNet: the crossing lists' keys decoded into their rows.
template <bool OUT_BF16>
__global__ __launch_bounds__(kBlock) void k_pointnet_rows(const int32_t *__restrict__ lvert,
                                                          const int32_t *__restrict__ vinfo,
                                                          const int32_t *__restrict__ counters,
                                                          unsigned int *__restrict__ keys, void *__restrict__ out) {
    pointnet_rows<OUT_BF16>(blockIdx.x, gridDim.x, lvert, vinfo, counters, 1, keys, out);
}

typedef float f32x4_t __attribute__((ext_vector_type(4)));

// v_mfma_f32_16x16x4f32: D[16 x 16] += A[16 x 4] B[4 x 16]; lane l supplies
// A[l % 16][l / 16] and B[l / 16][l % 16]; register r of lane l holds
// D[4 (l / 16) + r][l % 16].
__device__ __forceinline__ f32x4_t mfma16(float a, float b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// The three blocks on fp32 MFMA, with the entries as the columns:
// D_l [w_l x 16 entries] = W_l [w_l x K] R_{l-1}^T [K x 16 entries], one
// 16-entry column tile at a time (four per wavefront of 64 entries).
// Register r of lane l then holds output channel 4 (l / 16) + r (+16 per row
// tile) of entry l % 16, which is exactly the B operand the next block
// needs if its K index at step t, lane quarter q, is that channel: each
// lane's weight fragments are loaded once with that permutation, so no
// activation moves between blocks.  Block 1's input comes from LDS (each
// lane stages its own row).  The outputs go to LDS channel-major for the
// per-run max.  Each wavefront loops over its own chunks (wavefront-level
// synchronisation only).
template <bool OUT_BF16>
__global__ __launch_bounds__(kBlock) void k_pointnet(const int32_t *__restrict__ list,
                                                     const int32_t *__restrict__ lvert,
                                                     const int32_t *__restrict__ vinfo,
                                                     const float *__restrict__ pos, const float *__restrict__ feat,
                                                     int d, int f_d, const float *__restrict__ P,
                                                     const float *__restrict__ mu,
                                                     const int32_t *__restrict__ counters,
                                                     unsigned int *__restrict__ keys, void *__restrict__ out) {
    __shared__ __attribute__((aligned(16))) float ysh[kWaves][kW3 * kYStride];  // outputs [64 channels][64 entries]; first the staged inputs

    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int q = lane >> 4, j16 = lane & 15;
    float *Y = ysh[w];
    const int k0 = d + f_d;

    // weight fragments (A operands) and per-channel affines of this lane
    float wa1[4], na1[4], ns1[4];
    float wa2[2][4], na2[2][4], ns2[2][4];
    float wa3[4][8], bb3[4][4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        wa1[t] = P[kWt0 + j16 * kMaxK0 + 4 * t + q];  // block 1: K = 4 t + q (the staged input order)
        const int c = 4 * q + t;                       // block 1 output channel in register t
        na1[t] = P[kA1 + c];
        ns1[t] = fmaf(P[kA1 + c], P[kB0 + c], P[kS1 + c]);  // a (h + b) + s = a h + (a b + s)
    }
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            wa2[mt][t] = P[kWt1 + (16 * mt + j16) * kW1 + 4 * q + t];  // block 2: K = 4 q + t
            const int c = 16 * mt + 4 * q + t;
            na2[mt][t] = P[kA2 + c];
            ns2[mt][t] = fmaf(P[kA2 + c], P[kB1 + c], P[kS2 + c]);
        }
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
#pragma unroll
        for (int t = 0; t < 8; ++t)  // block 3: K = 16 (t / 4) + 4 q + t % 4
            wa3[mt][t] = P[kWt2 + (16 * mt + j16) * kW2 + 16 * (t / 4) + 4 * q + (t % 4)];
#pragma unroll
        for (int r = 0; r < 4; ++r) bb3[mt][r] = P[kB2 + 16 * mt + 4 * q + r];
    }

    const int64_t E = counters[CNT_E];
    const int64_t nwaves = (int64_t)gridDim.x * kWaves;
    // Software pipeline over this wavefront's chunks: the entry's vertex and
    // point (level 1) are loaded two chunks ahead, the vertex's list header,
    // the point's position and features and the vertex's mean (level 2, which
    // need level 1) one chunk ahead, so that a chunk's MFMAs never wait on
    // its own gathers.
    struct Rows {
        int v, p;             // level 1
        int off, cnt;         // level 2
        float x[kMaxK0];      // h_0 (level 2)
    };
    auto level1 = [&](int64_t chk, Rows &R) {
        const int64_t e = chk * 64 + lane;
        const bool valid = e < E;
        R.v = valid ? lvert[e] : -1;
        R.p = valid ? list[2 * e] : 0;
    };
    auto level2 = [&](Rows &R) {
        const bool valid = R.v >= 0;
        R.off = valid ? vinfo[2 * R.v] : 0;
        R.cnt = valid ? vinfo[2 * R.v + 1] : 0;
#pragma unroll
        for (int i = 0; i < kMaxK0; ++i) {
            float x = 0.f;
            if (valid && i < d) x = pos[(int64_t)R.p * d + i] - mu[(int64_t)R.v * d + i];
            else if (valid && i < k0) x = feat[(int64_t)R.p * f_d + (i - d)];
            R.x[i] = x;
        }
    };
    int64_t ch = ((int64_t)blockIdx.x * kBlock + threadIdx.x) >> 6;
    Rows cur, nxt;
    int v2 = -1, p2 = 0;
    if (ch * 64 < E) {
        level1(ch, cur);
        level2(cur);
        level1(ch + nwaves, nxt);
    }
    for (; ch * 64 < E; ch += nwaves) {
        // issue the next chunk's level 2 and the one after's level 1
        {
            Rows tmp;
            tmp.v = nxt.v;
            tmp.p = nxt.p;
            const int64_t e2 = (ch + 2 * nwaves) * 64 + lane;
            v2 = e2 < E ? lvert[e2] : -1;
            p2 = e2 < E ? list[2 * e2] : 0;
            level2(tmp);
            nxt = tmp;
        }
        const int64_t chunk0 = ch * 64;
        const int v = cur.v;
        const bool valid = v >= 0;
        // run flags: 1 first entry of a run, 2 last, 4 the run is the vertex's whole list
        const int vprev = __shfl_up(v, 1);
        const int vnext = __shfl_down(v, 1);
        int flags = 0;
        if (valid) {
            if (lane == 0 || vprev != v) flags |= 1;
            if (lane == 63 || vnext != v) flags |= 2;
            if (cur.off >= chunk0 && cur.off + cur.cnt <= chunk0 + 64) flags |= 4;
        }
        // destination of the run: the output row, or the key row of the
        // chunk where the vertex's list starts
        const int dest = (flags & 4) ? v : (valid ? (int)(cur.off >> 6) : -1);

        // r_0 = relu(a_0 h_0 + s_0), h_0 = [g_p - mu_v ; f_p] zero-padded, staged in LDS
#pragma unroll
        for (int i = 0; i < kMaxK0; ++i) Y[lane * (kMaxK0 + 1) + i] = relu(fmaf(P[kA0 + i], cur.x[i], P[kS0 + i]));
        wave_sync();
        float b1[4][4];  // B operands of block 1: entry 16 nt + j16, K = 4 t + q
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
#pragma unroll
            for (int t = 0; t < 4; ++t) b1[nt][t] = Y[(16 * nt + j16) * (kMaxK0 + 1) + 4 * t + q];
        wave_sync();

#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
            f32x4_t d1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int t = 0; t < 4; ++t) d1 = mfma16(wa1[t], b1[nt][t], d1);
            float r1[4];
#pragma unroll
            for (int t = 0; t < 4; ++t) r1[t] = relu(fmaf(na1[t], d1[t], ns1[t]));
            f32x4_t d2[2];
#pragma unroll
            for (int mt = 0; mt < 2; ++mt) {
                d2[mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int t = 0; t < 4; ++t) d2[mt] = mfma16(wa2[mt][t], r1[t], d2[mt]);
            }
            float r2[8];
#pragma unroll
            for (int t = 0; t < 8; ++t) r2[t] = relu(fmaf(na2[t / 4][t % 4], d2[t / 4][t % 4], ns2[t / 4][t % 4]));
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) {
                f32x4_t d3 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int t = 0; t < 8; ++t) d3 = mfma16(wa3[mt][t], r2[t], d3);
#pragma unroll
                for (int r = 0; r < 4; ++r) Y[(16 * mt + 4 * q + r) * kYStride + 16 * nt + j16] = d3[r] + bb3[mt][r];
            }
        }
        wave_sync();

        // lane c: running max of channel c over each run of the wavefront's
        // entries, four entries per LDS read; an entry's run flags and
        // destination come from its lane (readlane: scalar values, so the
        // store at a run's end is a uniform branch)
        {
            const int c = lane;
            float mx = 0.f;
#pragma unroll
            for (int j4 = 0; j4 < 16; ++j4) {
                const f32x4_t y4 = *reinterpret_cast<const f32x4_t *>(Y + c * kYStride + 4 * j4);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int jj = 4 * j4 + i;
                    const int fj = __builtin_amdgcn_readlane(flags, jj);
                    mx = (fj & 1) ? y4[i] : fmaxf(mx, y4[i]);
                    if (fj & 2) {
                        const int vj = __builtin_amdgcn_readlane(dest, jj);
                        if (fj & 4)
                            store_out<OUT_BF16>(out, vj, c, mx);
                        else
                            atomicMax(keys + (int64_t)vj * kW3 + c, max_key(mx));
                    }
                }
            }
        }
        wave_sync();
        cur = nxt;
        nxt.v = v2;
        nxt.p = p2;
    }
}

}  // namespace

// Packed parameter count for d + f_d = k0 inputs: per block a [K], s [K],
// W [w][K], b [w] with K the block's input width.
int pointnet_padded_count() { return kPadded; }

int pointnet_param_count(int k0) {
    return 2 * k0 + kW1 * k0 + kW1 + 2 * kW1 + kW2 * kW1 + kW2 + 2 * kW2 + kW3 * kW2 + kW3;
}

hipError_t launch_distribute_pointnet(lattice *L, const float *pos, const float *feat, int f_d, const float *params,
                                      void *out, bool out_bf16, float *mean) {
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
    switch (d) {
#define LM_CASE(DD)                                                                                              \
    case DD:                                                                                                     \
        hipLaunchKernelGGL(k_local_mean<DD>, dim3(g_e), dim3(kBlock), 0, L->stream, L->list, L->lvert, L->vinfo, \
                           pos, L->counters, L->macc, mu);                                                       \
        break;
        LM_CASE(1)
        LM_CASE(2)
        LM_CASE(3)
        LM_CASE(4)
#undef LM_CASE
        default:
            return hipErrorInvalidValue;
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const unsigned g_i = grid_for((E / 64 + 1) * kW3, kBlock, L->cu_count, 4);
    const unsigned g_k = (kPadded + kBlock - 1) / kBlock;
    hipLaunchKernelGGL(k_pointnet_prep, dim3(g_v + g_i + g_k), dim3(kBlock), 0, L->stream, L->vinfo, L->macc, d,
                       L->counters, mu, L->lvert, L->pn_keys, params, d + f_d, L->pn_params, (int)g_v, (int)g_i,
                       (int)g_k);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const unsigned g_p = grid_for(E, kBlock, L->cu_count, 2);  // 69 KB of LDS: two workgroups per CU
    hipLaunchKernelGGL((out_bf16 ? k_pointnet<true> : k_pointnet<false>), dim3(g_p), dim3(kBlock), 0, L->stream,
                       L->list, L->lvert, L->vinfo, pos, feat, d, f_d, L->pn_params, mu, L->counters, L->pn_keys,
                       out);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL((out_bf16 ? k_pointnet_rows<true> : k_pointnet_rows<false>), dim3(g_i), dim3(kBlock), 0,
                       L->stream, L->lvert, L->vinfo, L->counters, L->pn_keys, out);
    return hipGetLastError();
}
